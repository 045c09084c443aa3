"""Block-level GPU parity through xema_dit_block_fwd (C ABI) against the fp64
oracle, plus the properties that hold at any size: bit-identical output for
every chunk size and across runs, zero gates pass tokens through exactly,
batch rows are independent runs.  The five workloads are checked at their
full sizes on seeded row samples (the oracle forms K and V from every token
and the outputs of the sampled rows only)."""
import numpy as np
import pytest
import torch

import paper_2607_11136_amd as X
import workloads as W
from oracle import block as O

from gpu_util import DEV, Device, assert_parity, slot_view

pytestmark = pytest.mark.gpu

# Small shapes the oracle finishes in seconds, spanning several GEMM and
# attention tiles with ragged tails (L not a multiple of 64/128/256).
SMALL = {
    "tiny": W.TINY,
    "d64_b2": W.tiny_shape(name="d64_b2", cfg_id=50, batch=2, text_len=45, grid=(3, 9, 23), hidden=512,
                           heads=8, head_dim=64, mlp_hidden=2048, cond_dim=512, rope_dims=(16, 24, 24)),
    "d128_img": W.tiny_shape(name="d128_img", cfg_id=51, batch=1, text_len=64, grid=(1, 20, 31),
                             hidden=512, heads=4, head_dim=128, mlp_hidden=1536, cond_dim=256,
                             rope_dims=(0, 64, 64)),
    "d128_b3": W.tiny_shape(name="d128_b3", cfg_id=52, batch=3, text_len=7, grid=(5, 6, 11), hidden=768,
                            heads=6, head_dim=128, mlp_hidden=1024, cond_dim=768, rope_dims=(32, 48, 48)),
}

_cache = {}


def _device(s):
    if s.name not in _cache:
        _cache.clear()
        _cache[s.name] = Device(W.make_inputs(s))
    return _cache[s.name]


@pytest.mark.parametrize("name", sorted(SMALL))
def test_block_matches_oracle_full(name):
    s = SMALL[name]
    dev = _device(s)
    print(f"block {name}: B={s.batch} L={s.seq_len} D={s.hidden} H={s.heads}x{s.head_dim}", flush=True)
    out, ws, plan = dev.run(0)
    ref = O.block_forward_shape(dev.inputs)
    assert_parity(out.cpu().numpy(), ref, f"block {name}")


@pytest.mark.parametrize("name", sorted(SMALL))
def test_chunked_runs_are_bit_identical(name):
    s = SMALL[name]
    dev = _device(s)
    base, _, _ = dev.run(0)
    L = s.seq_len
    for chunk in sorted({64, 100, 256, L - 1, 1 + L // 3} | set(s.chunks[1:])):
        if chunk <= 0 or chunk >= L:
            continue
        out, _, plan = dev.run(chunk)
        assert plan.chunk_tokens == chunk
        assert torch.equal(out, base), (name, chunk)
    again, _, _ = dev.run(0)
    assert torch.equal(again, base)


def test_intermediates_in_arena_match_oracle_steps():
    """The arena keeps every slot at its planned offset: after an unchunked
    call, mod, Q, K and V^T hold the AdaLN map and the normalised/rotated
    heads of every token."""
    s = SMALL["d64_b2"]
    dev = _device(s)
    out, ws, plan = dev.run(0)
    B, L, D, H, d = s.batch, s.seq_len, s.hidden, s.heads, s.head_dim
    Lp = X.padded_len(L)
    x, c, w = dev.inputs.f64("x"), dev.inputs.f64("cond"), dev.inputs.weights_f64()
    m = O.adaln_modulation(c, w["ada_w"], w["ada_b"])
    mod = slot_view(ws, plan, "mod", torch.float32, (B, 6 * D)).cpu().numpy()
    np.testing.assert_allclose(mod, m, rtol=1e-5, atol=1e-5)
    q = slot_view(ws, plan, "q", torch.float16, (B, H, Lp, d)).float().cpu().numpy()
    k = slot_view(ws, plan, "k", torch.float16, (B, H, Lp, d)).float().cpu().numpy()
    vt = slot_view(ws, plan, "vt", torch.float16, (B, H, d, Lp)).float().cpu().numpy()
    coords = O.token_coords(s.text_len, s.grid)
    for b in range(B):
        h = O.modulate(O.layer_norm(x[b], s.ln_eps), m[b, :D], m[b, D:2 * D])
        qr, kr, vr = O.qkv_heads(h, w, H, d, coords, s.rope_dims, s.rope_theta, s.qk_eps)
        qr = qr * (np.log2(np.e) / np.sqrt(d))   # the softmax factor the stored queries carry
        # bf16 h and fp16 qkv / Q / K / V roundings on the GPU side
        for got, ref in ((q[b, :, :L].transpose(1, 0, 2), qr), (k[b, :, :L].transpose(1, 0, 2), kr),
                         (vt[b, :, :, :L].transpose(2, 0, 1), vr)):
            err = np.abs(got - ref)
            assert err.mean() < 5e-3 and err.max() < 6e-2, (err.mean(), err.max())
    assert np.all(q[:, :, L:] == 0) and np.all(vt[..., L:] == 0)


def test_zero_gates_pass_tokens_through_exactly():
    s = SMALL["d64_b2"]
    inp = W.make_inputs(s)
    D = s.hidden
    for blk in (2, 5):
        inp.weights["ada_w"][blk * D:(blk + 1) * D] = 0
        inp.weights["ada_b"][blk * D:(blk + 1) * D] = 0
    dev = Device(inp)
    out, _, _ = dev.run(0)
    assert torch.equal(out, dev.x.float())
    out64, _, _ = dev.run(64)
    assert torch.equal(out64, dev.x.float())


def test_batch_rows_are_independent_runs():
    s = SMALL["d128_b3"]
    dev = _device(s)
    full, _, _ = dev.run(0)
    for b in range(s.batch):
        one = W.Inputs(s.with_(batch=1), dev.inputs.x[b:b + 1].copy(), dev.inputs.cond[b:b + 1].copy(),
                       dev.inputs.weights)
        d1 = Device(one)
        o1, _, _ = d1.run(0)
        assert torch.equal(o1[0], full[b]), b


# Degenerate request shapes: text only (empty grid), visual only (no text),
# a sequence shorter than one 64-key tile, with extreme chunkings.
EDGE = {
    "text_only": W.tiny_shape(name="text_only", cfg_id=60, batch=2, text_len=100, grid=(0, 0, 0),
                              hidden=256, heads=4, head_dim=64, mlp_hidden=512, cond_dim=256,
                              rope_dims=(16, 24, 24)),
    "visual_only": W.tiny_shape(name="visual_only", cfg_id=61, batch=1, text_len=0, grid=(2, 5, 7),
                                hidden=256, heads=2, head_dim=128, mlp_hidden=256, cond_dim=256,
                                rope_dims=(32, 48, 48)),
    "short": W.tiny_shape(name="short", cfg_id=62, batch=2, text_len=5, grid=(1, 4, 8), hidden=512,
                          heads=8, head_dim=64, mlp_hidden=1024, cond_dim=512, rope_dims=(16, 24, 24)),
    # head_dim 64 takes the QKV GEMM's fused heads epilogue: every token rotated,
    # chunks of one token put each GEMM row in another batch element
    "visual_only_d64": W.tiny_shape(name="visual_only_d64", cfg_id=63, batch=2, text_len=0, grid=(3, 5, 7),
                                    hidden=256, heads=4, head_dim=64, mlp_hidden=512, cond_dim=256,
                                    rope_dims=(16, 24, 24)),
}


@pytest.mark.parametrize("name", sorted(EDGE))
def test_edge_shapes_match_oracle_and_chunk_exactly(name):
    s = EDGE[name]
    print(f"edge {name}: B={s.batch} L={s.seq_len} text={s.text_len} grid={s.grid}", flush=True)
    dev = Device(W.make_inputs(s))
    base, _, _ = dev.run(0)
    assert_parity(base.cpu().numpy(), O.block_forward_shape(dev.inputs), f"edge {name}")
    for chunk in (1, 7, s.seq_len - 1):
        out, _, _ = dev.run(chunk)
        assert torch.equal(out, base), (name, chunk)


def test_budget_plan_drives_the_call():
    """Plan a budget between the smallest and the unchunked arena, run with the
    planned chunk in an arena of exactly the planned size."""
    s = SMALL["d64_b2"]
    dev = _device(s)
    small = X.xema_workspace_bytes(dev.cfg, dev.req, 256)
    full = X.xema_workspace_bytes(dev.cfg, dev.req, 0)
    plan = X.xema_workspace_plan(dev.cfg, dev.req, (small + full) // 2)
    assert 0 < plan.chunk_tokens < s.seq_len and plan.workspace_bytes <= (small + full) // 2
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    out, _, _ = dev.run(plan.chunk_tokens, ws=ws)
    base, _, _ = dev.run(0)
    assert torch.equal(out, base)
    with pytest.raises(X.XemaError) as e:
        X.xema_dit_block_fwd(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, 0, ws, ws.numel(),
                             torch.empty_like(base))
    assert e.value.status == X.XEMA_ERR_WORKSPACE_TOO_SMALL


def test_temporary_serialization_is_bit_identical():
    """Sequences run through the block in groups (temporary serialization):
    every group size and chunk gives the unserialized output bit for bit."""
    s = SMALL["d128_b3"]
    dev = _device(s)
    base, _, _ = dev.run(0)
    for g, chunk in ((1, 0), (2, 0), (2, 100), (1, 37), (5, 64)):
        sub = X.request(min(g, s.batch), s.text_len, *s.grid)
        r_last = X.request(s.batch % g or min(g, s.batch), s.text_len, *s.grid)
        nbytes = max(X.xema_workspace_bytes(dev.cfg, sub, chunk), X.xema_workspace_bytes(dev.cfg, r_last, chunk))
        ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
        out = torch.empty_like(base)
        X.xema_dit_block_fwd_serial(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, g, chunk, ws, nbytes, out)
        torch.cuda.synchronize()
        assert torch.equal(out, base), (g, chunk)


def test_serial_plan_drives_the_call_below_the_batch_minimum():
    """A budget below the whole batch's smallest arena: the plan serializes,
    and the call with the planned group and chunk reproduces the output."""
    s = SMALL["d128_b3"]
    dev = _device(s)
    base, _, _ = dev.run(0)
    full_min = X.xema_workspace_layout(dev.cfg, dev.req, 0).min_workspace_bytes
    g, plan = X.xema_workspace_plan_serial(dev.cfg, dev.req, full_min - 1)
    assert g < s.batch and plan.workspace_bytes <= full_min - 1
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    out = torch.empty_like(base)
    X.xema_dit_block_fwd_serial(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, g, plan.chunk_tokens, ws,
                                ws.numel(), out)
    torch.cuda.synchronize()
    assert torch.equal(out, base)


# -- the five workloads at full size, on sampled rows ---------------------------------

FULL = [("tiny", 0, None), ("image", 0, 48), ("image_b4", 0, 24), ("video", 0, 48),
        ("long", 2048, 16), ("highres", 0, 16)]


@pytest.mark.parametrize("name,chunk,nrows", FULL)
def test_workload_parity_sampled_rows(name, chunk, nrows):
    s = W.CONFIGS[name]
    print(f"workload {name}: B={s.batch} L={s.seq_len} chunk={chunk} rows={nrows}", flush=True)
    dev = Device(W.make_inputs(s))
    out, _, plan = dev.run(chunk)
    rows = None if nrows is None else W.sample_rows(s, nrows)
    ref = O.block_forward_shape(dev.inputs, rows=rows)
    got = out.cpu().numpy() if rows is None else out[:, rows].cpu().numpy()
    assert_parity(got, ref, f"workload {name} chunk={chunk}")
    if name in ("long", "highres"):
        # bit-exact against the unchunked run / another chunking
        other, _, _ = dev.run(0 if chunk else 8192)
        assert torch.equal(other, out)
    del dev
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", sorted(SMALL))
def test_pipelined_chunks_are_bit_identical(name):
    """Each chunk's attention on a second stream (events between the
    streams) gives the one-stream bytes; back-to-back calls on one workspace
    stay ordered."""
    s = SMALL[name]
    dev = _device(s)
    base, _, _ = dev.run(0)
    aux = torch.cuda.Stream()
    L = s.seq_len
    for chunk in sorted({64, 100, 1 + L // 3}):
        if chunk >= L:
            continue
        plan = X.xema_workspace_layout(dev.cfg, dev.req, chunk)
        assert plan.slots()["attn"][3] == 10   # live through the MLP when chunked
        ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
        outs = [torch.empty_like(base) for _ in range(3)]
        for o in outs:   # no synchronisation between the calls
            X.xema_dit_block_fwd_pipelined(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, s.batch, chunk, ws,
                                           ws.numel(), o, None, aux)
        torch.cuda.synchronize()
        for o in outs:
            assert torch.equal(o, base), (name, chunk)


def test_pipelined_groups_are_bit_identical():
    s = SMALL["d128_b3"]
    dev = _device(s)
    base, _, _ = dev.run(0)
    aux = torch.cuda.Stream()
    chunk = 100
    plan = X.xema_workspace_layout(dev.cfg, X.request(1, s.text_len, *s.grid), chunk)
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    out = torch.empty_like(base)
    X.xema_dit_block_fwd_pipelined(dev.cfg, dev.req, dev.x, dev.weights, dev.cond, 1, chunk, ws, ws.numel(),
                                   out, None, aux)
    torch.cuda.synchronize()
    assert torch.equal(out, base)
