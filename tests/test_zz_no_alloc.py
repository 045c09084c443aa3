"""xema_dit_block_fwd_static, the entry point that allocates nothing (its
arena is the library's static device array), against xema_dit_block_fwd
with a caller workspace: the same bytes on two calls in a row, the second
with a smaller request, unchunked and chunked; a request larger than the
static arena is refused before any launch."""
import pytest
import torch

import paper_2607_11136_amd as X
import workloads as W

from gpu_util import Device, poison

pytestmark = pytest.mark.gpu

# the tiny workload, then a smaller request of the same block (80 tokens)
FIRST = W.TINY
SECOND = W.TINY.with_(name="tiny_small", cfg_id=64, text_len=16, grid=(1, 8, 8))


@pytest.mark.parametrize("chunks", [(0, 0), (64, 32)])
def test_static_arena_matches_the_workspace_entry_point(chunks):
    for s, chunk in zip((FIRST, SECOND), chunks):
        print(f"static arena: {s.name} L={s.seq_len} chunk={chunk}", flush=True)
        dev = Device(W.make_inputs(s))
        want, _, _ = dev.run(chunk)
        plan = X.xema_workspace_layout(dev.cfg, dev.req, chunk)
        assert plan.workspace_bytes <= X.XEMA_STATIC_ARENA_BYTES
        out = poison(torch.empty_like(want))
        X.xema_dit_block_fwd_static(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, chunk, out)
        torch.cuda.synchronize()
        assert torch.equal(out, want), (s.name, chunk)
        assert X.xema_block_status(plan, None) == 0


def test_static_arena_refuses_a_request_beyond_its_size():
    s = W.VIDEO
    cfg = X.block_cfg(s.hidden, s.heads, s.head_dim, s.mlp_hidden, s.cond_dim, s.rope_dims)
    req = X.request(s.batch, s.text_len, *s.grid)
    assert X.xema_workspace_bytes(cfg, req, 0) > X.XEMA_STATIC_ARENA_BYTES
    w = X.block_weights({n: 1 << 20 for n in X.WEIGHT_FIELDS})   # never dereferenced: refused first
    with pytest.raises(X.XemaError) as e:
        X.xema_dit_block_fwd_static(cfg, req, 1 << 21, w, 1 << 22, 0, 1 << 23)
    assert e.value.status == X.XEMA_ERR_WORKSPACE_TOO_SMALL
