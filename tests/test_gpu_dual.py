"""Dual-stream modulation (a second AdaLN map for the text tokens) on the GPU,
through the C ABI: parity with the fp64 oracle, bit-identical output for
every chunk size (chunks that cut through the text tokens included), for
serialized batch groups and for offloaded N-block steps; with the two maps
equal it reproduces the single-stream block bit for bit, and zero gates of
one stream pass exactly that stream's tokens through."""
import numpy as np
import pytest
import torch

import paper_2607_11136_amd as X
import workloads as W
from oracle import block as O

from gpu_util import DEV, Device, assert_parity, bf16_dev, slot_view

pytestmark = pytest.mark.gpu

DUAL = {
    "d64_b2": W.tiny_shape(name="dual_d64_b2", cfg_id=60, batch=2, text_len=45, grid=(3, 9, 23),
                           hidden=512, heads=8, head_dim=64, mlp_hidden=2048, cond_dim=512,
                           rope_dims=(16, 24, 24), modulation_streams=2),
    "d128": W.tiny_shape(name="dual_d128", cfg_id=61, batch=1, text_len=130, grid=(2, 10, 13),
                         hidden=768, heads=6, head_dim=128, mlp_hidden=1024, cond_dim=256,
                         rope_dims=(32, 48, 48), modulation_streams=2),
}

_cache = {}


def _device(name):
    if name not in _cache:
        _cache.clear()
        _cache[name] = Device(W.make_inputs(DUAL[name]))
    return _cache[name]


def _single_inputs(inp: W.Inputs) -> W.Inputs:
    """The same tensors as a single-stream block (text map dropped)."""
    w = {k: v for k, v in inp.weights.items() if k not in W.TEXT_MOD_NAMES}
    return W.Inputs(inp.shape.with_(modulation_streams=1), inp.x, inp.cond, w)


@pytest.mark.parametrize("name", sorted(DUAL))
def test_dual_block_matches_oracle(name):
    s = DUAL[name]
    dev = _device(name)
    print(f"dual block {name}: B={s.batch} L={s.seq_len} L_t={s.text_len} D={s.hidden}", flush=True)
    out, _, _ = dev.run(0)
    ref = O.block_forward_shape(dev.inputs)
    assert_parity(out.cpu().numpy(), ref, f"dual block {name}")
    # the text map matters: the single-stream oracle is far from this output
    single = O.block_forward_shape(_single_inputs(dev.inputs))
    assert np.max(np.abs(out.cpu().numpy()[:, :s.text_len] - single[:, :s.text_len])) > 0.05


@pytest.mark.parametrize("name", sorted(DUAL))
def test_dual_chunked_runs_are_bit_identical(name):
    s = DUAL[name]
    dev = _device(name)
    base, _, _ = dev.run(0)
    T = s.text_len
    for chunk in sorted({T - 1, T, T + 1, 64, 100, 1 + s.seq_len // 3}):
        out, _, plan = dev.run(chunk)
        assert plan.chunk_tokens == chunk
        assert torch.equal(out, base), (name, chunk)


@pytest.mark.parametrize("name", sorted(DUAL))
def test_dual_pipelined_chunks_are_bit_identical(name):
    """The two-stream chunked driver picks each row's modulation by its sequence
    position like the one-stream one, for chunks that end just before, at and
    just after the text tokens."""
    s = DUAL[name]
    dev = _device(name)
    base, _, _ = dev.run(0)
    aux = torch.cuda.Stream()
    T = s.text_len
    for chunk in sorted({T - 1, T, T + 1, 100}):
        if chunk <= 0 or chunk >= s.seq_len:
            continue
        plan = X.xema_workspace_layout(dev.cfg, dev.req, chunk)
        ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
        out = torch.empty_like(base)
        X.xema_dit_block_fwd_pipelined(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, s.batch, chunk, ws,
                                       ws.numel(), out, None, aux)
        torch.cuda.synchronize()
        assert torch.equal(out, base), (name, chunk)


def test_dual_modulation_slot_holds_both_maps():
    s = DUAL["d64_b2"]
    dev = _device("d64_b2")
    _, ws, plan = dev.run(0)
    B, D = s.batch, s.hidden
    c, w = dev.inputs.f64("cond"), dev.inputs.weights_f64()
    mod = slot_view(ws, plan, "mod", torch.float32, (2, B, 6 * D)).cpu().numpy()
    np.testing.assert_allclose(mod[0], O.adaln_modulation(c, w["ada_w"], w["ada_b"]), rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(mod[1], O.adaln_modulation(c, w["ada_txt_w"], w["ada_txt_b"]),
                               rtol=1e-5, atol=1e-5)


def test_equal_maps_reproduce_the_single_stream_block():
    inp = W.make_inputs(DUAL["d64_b2"])
    inp.weights["ada_txt_w"] = inp.weights["ada_w"].copy()
    inp.weights["ada_txt_b"] = inp.weights["ada_b"].copy()
    dual, _, _ = Device(inp).run(0)
    single, _, _ = Device(_single_inputs(inp)).run(0)
    assert torch.equal(dual, single)


@pytest.mark.parametrize("stream", ["text", "visual"])
def test_zero_gates_of_one_stream_pass_its_tokens_through(stream):
    s = DUAL["d64_b2"]
    inp = W.make_inputs(s)
    D, T = s.hidden, s.text_len
    wk, bk = ("ada_txt_w", "ada_txt_b") if stream == "text" else ("ada_w", "ada_b")
    for blk in (2, 5):
        inp.weights[wk][blk * D:(blk + 1) * D] = 0
        inp.weights[bk][blk * D:(blk + 1) * D] = 0
    dev = Device(inp)
    x = dev.x.float()
    same, moved = (slice(0, T), slice(T, None)) if stream == "text" else (slice(T, None), slice(0, T))
    for chunk in (0, T, 64):
        out, _, _ = dev.run(chunk)
        assert torch.equal(out[:, same], x[:, same]), chunk
        assert torch.amin(torch.amax(torch.abs(out[:, moved] - x[:, moved]), dim=-1)) > 1e-3


def test_dual_serialized_groups_are_bit_identical():
    s = DUAL["d64_b2"]
    dev = _device("d64_b2")
    base, _, _ = dev.run(0)
    for chunk in (0, 100):
        plan = X.xema_workspace_layout(dev.cfg, X.request(1, s.text_len, *s.grid), chunk)
        ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
        out = torch.empty_like(base)
        X.xema_dit_block_fwd_serial(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, 1, chunk, ws,
                                    ws.numel(), out)
        torch.cuda.synchronize()
        assert torch.equal(out, base), chunk


def test_dual_step_with_offloading_is_bit_identical():
    s = DUAL["d64_b2"]
    n = 3
    inputs = W.make_inputs(s)
    bits = W.step_weights(s, n)
    assert all("ada_txt_w" in b for b in bits)
    x, cond = bf16_dev(inputs.x), bf16_dev(inputs.cond)
    dev_w = [{k: bf16_dev(v) for k, v in b.items()} for b in bits]
    host_w = []
    for b in bits:
        hw = {}
        for k, v in b.items():
            t = torch.empty(v.shape, dtype=torch.bfloat16, pin_memory=True)
            t.copy_(torch.from_numpy(np.ascontiguousarray(v).view(np.int16)).view(torch.bfloat16))
            hw[k] = t
        host_w.append(hw)
    dev = Device(inputs)
    outs = []
    for k, staging in ((0, 1), (2, 1), (3, 2)):
        plan = X.xema_offload_plan_k(dev.cfg, n, k, staging)
        off = set(plan.offloaded_blocks())
        ws_list = [X.block_weights(host_w[i] if i in off else dev_w[i]) for i in range(n)]
        nbytes = X.xema_step_workspace_bytes(dev.cfg, dev.req, 0, plan)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
        out = torch.empty((s.batch, s.seq_len, s.hidden), dtype=torch.float32, device=DEV)
        X.xema_dit_step_fwd(dev.cfg, dev.req, x, ws_list, plan, cond, 0, ws, nbytes, out,
                            copy_stream=torch.cuda.Stream())
        torch.cuda.synchronize()
        outs.append(out)
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    # block 0 of the step is the block API's output, carried on by blocks 1, 2
    one = X.xema_offload_plan_k(dev.cfg, 1, 1, 1)
    nbytes = X.xema_step_workspace_bytes(dev.cfg, dev.req, 0, one)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    out1 = torch.empty_like(outs[0])
    X.xema_dit_step_fwd(dev.cfg, dev.req, x, [X.block_weights(host_w[0])], one, cond, 0, ws, nbytes, out1,
                        copy_stream=torch.cuda.Stream())
    ref1, _, _ = dev.run(0)
    torch.cuda.synchronize()
    assert torch.equal(out1, ref1)
