"""xema_dit_block_fwd_static under HIP graph capture, the use it is meant
for: a warm-up call outside the capture (the first call on a device looks up
the static array's address), then the call captured into a graph on torch's
capture stream and replayed several times, with eager work and
synchronisation between the replays.  Every replay gives the bytes of
xema_dit_block_fwd with a caller workspace.  The single-stream block path
launches kernels only (no memset, allocation or event), so nothing else
enters the graph."""
import pytest
import torch

import paper_2607_11136_amd as X
import workloads as W

from gpu_util import Device, poison

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("chunk", [0, 64])
def test_static_entry_point_replays_in_a_graph(chunk):
    s = W.TINY
    dev = Device(W.make_inputs(s))
    want, _, _ = dev.run(chunk)
    out = poison(torch.empty_like(want))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up, eager
        X.xema_dit_block_fwd_static(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, chunk, out, side)
    torch.cuda.synchronize()
    assert torch.equal(out, want)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        X.xema_dit_block_fwd_static(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, chunk, out,
                                    torch.cuda.current_stream())
    for replay in range(3):
        poison(out)                      # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        print(f"graph replay {replay} (chunk {chunk})", flush=True)
        assert torch.equal(out, want), (chunk, replay)
    plan = X.xema_workspace_layout(dev.cfg, dev.req, chunk)
    assert X.xema_block_status(plan, None) == 0
    del graph
