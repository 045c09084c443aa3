"""Per-step GPU parity: each entry point of xema_ops.h against the matching
oracle step, on identical input values (bf16/fp16 upcast exactly to fp64).
Shapes span several tiles and a ragged tail."""
import numpy as np
import pytest
import torch

import paper_2607_11136_amd as X
import workloads as W
from oracle import block as O

from gpu_util import DEV, bf16_dev, cfg_of, req_of

pytestmark = pytest.mark.gpu

LOG2E = 1.4426950408889634


def _rng(seed):
    return np.random.default_rng(seed)


def _bf16_bits(a):
    return W.to_bf16_bits(np.asarray(a, dtype=np.float32))


def _f16(a):
    return np.asarray(a, dtype=np.float16)


def _check_close(gpu, ref, rel, atol, what):
    gpu = np.asarray(gpu, dtype=np.float64)
    d = np.abs(gpu - ref)
    bound = rel * np.abs(ref) + atol
    bad = d > bound
    print(f"{what}: max|d|={d.max():.3e} mean|d|={d.mean():.3e} bad={int(bad.sum())}", flush=True)
    assert np.all(np.isfinite(gpu)), what
    assert not bad.any(), (what, float(d.max()), np.argwhere(bad)[:5])


def test_adaln_matches_oracle():
    for B, Dc, N in [(1, 256, 1536), (4, 3072, 6 * 512), (9, 520, 256)]:
        g = _rng(B + Dc)
        cond = _bf16_bits(g.standard_normal((B, Dc)))
        w = _bf16_bits(g.standard_normal((N, Dc)) / np.sqrt(Dc))
        b = _bf16_bits(g.standard_normal(N) / np.sqrt(Dc))
        mod = torch.empty((B, N), dtype=torch.float32, device=DEV)
        X.xema_op_adaln(bf16_dev(cond), bf16_dev(w), bf16_dev(b), B, Dc, N, mod)
        torch.cuda.synchronize()
        ref = O.adaln_modulation(W.bf16_bits_to_f64(cond), W.bf16_bits_to_f64(w), W.bf16_bits_to_f64(b))
        _check_close(mod.cpu().numpy(), ref, 1e-5, 1e-5, f"adaln B={B} Dc={Dc}")


@pytest.mark.parametrize("x_dtype,y_dtype", [(X.XEMA_BF16, X.XEMA_BF16), (X.XEMA_F32, X.XEMA_F16),
                                             (X.XEMA_BF16, X.XEMA_F16), (X.XEMA_F32, X.XEMA_BF16)])
@pytest.mark.parametrize("D", [768, 1024])    # 4 and 8 elements per lane
def test_ln_modulate_matches_oracle(x_dtype, y_dtype, D):
    g = _rng(3)
    B, L = 3, 77
    s0, cnt = 20, 45                       # a chunk of each sequence
    xs = g.standard_normal((B, L, D)) * 2.0 + 0.5
    mod = g.standard_normal((B, 6 * D)).astype(np.float32)
    if x_dtype == X.XEMA_BF16:
        bits = _bf16_bits(xs)
        x64 = W.bf16_bits_to_f64(bits)
        xd = bf16_dev(bits)
    else:
        x64 = xs.astype(np.float32).astype(np.float64)
        xd = torch.from_numpy(xs.astype(np.float32)).to(DEV)
    modd = torch.from_numpy(mod).to(DEV)
    ydt = torch.bfloat16 if y_dtype == X.XEMA_BF16 else torch.float16
    y = torch.empty((B * cnt, D), dtype=ydt, device=DEV)
    X.xema_op_ln_modulate(xd, x_dtype, X.rowmap(cnt, L, s0), B * cnt, D, modd[:, 3 * D:], modd[:, 4 * D:],
                          6 * D, 1e-6, y, y_dtype)
    torch.cuda.synchronize()
    m64 = mod.astype(np.float64)
    ref = np.concatenate([O.modulate(O.layer_norm(x64[b, s0:s0 + cnt], 1e-6), m64[b, 3 * D:4 * D],
                                     m64[b, 4 * D:5 * D]) for b in range(B)])
    rel = 2.0 ** -8 if y_dtype == X.XEMA_BF16 else 2.0 ** -10
    _check_close(y.float().cpu().numpy(), ref, rel, 1e-4, f"ln_modulate D={D}")


def _gemm_case(dtype, M, N, K, epi, seed, chunked=False):
    g = _rng(seed)
    np_t = np.float16 if dtype == X.XEMA_F16 else None
    a = g.standard_normal((M, K))
    b = g.standard_normal((N, K)) / np.sqrt(K)
    bias = _bf16_bits(g.standard_normal(N) * 0.1)
    if dtype == X.XEMA_F16:
        a16, b16 = _f16(a), _f16(b)
        A, Bm = torch.from_numpy(a16).to(DEV), torch.from_numpy(b16).to(DEV)
        a64, b64 = a16.astype(np.float64), b16.astype(np.float64)
    else:
        ab, bb = _bf16_bits(a), _bf16_bits(b)
        A, Bm = bf16_dev(ab), bf16_dev(bb)
        a64, b64 = W.bf16_bits_to_f64(ab), W.bf16_bits_to_f64(bb)
    bias64 = W.bf16_bits_to_f64(bias)
    acc = a64 @ b64.T + bias64
    if epi == X.XEMA_EPI_GATED_RESIDUAL:
        # rows of A belong to `nb` batches of `rpb` rows; C rows scattered into a
        # [nb, Ltot, N] buffer at offset s0 (the chunked layout of the block)
        rpb = M // 3 if chunked else M
        nb = M // rpb
        assert nb * rpb == M
        Ltot, s0 = rpb + 37, 11
        res = g.standard_normal((nb * Ltot, N)).astype(np.float32)
        gate = g.standard_normal((nb, 2 * N)).astype(np.float32)
        C = torch.full((nb * Ltot, N), float("nan"), dtype=torch.float32, device=DEV)
        args = X.gemm_args(dtype, A, M, K, Bm, N, bias_dev := bf16_dev(bias), epi, C, X.XEMA_F32, N,
                           c_map=X.rowmap(rpb, Ltot, s0),
                           resid=(resd := torch.from_numpy(res).to(DEV)), resid_dtype=X.XEMA_F32,
                           resid_map=X.rowmap(rpb, Ltot, s0), ld_resid=N,
                           gate=(gd := torch.from_numpy(gate).to(DEV))[:, N:], gate_stride=2 * N)
        X.xema_op_gemm(args)
        torch.cuda.synchronize()
        Cn = C.cpu().numpy().reshape(nb, Ltot, N)
        ref = np.empty((nb, rpb, N))
        for bi in range(nb):
            rows = slice(bi * rpb, (bi + 1) * rpb)
            r64 = res.reshape(nb, Ltot, N)[bi, s0:s0 + rpb].astype(np.float64)
            ref[bi] = r64 + gate[bi, N:].astype(np.float64) * acc[rows]
        # rows outside the mapped range stay untouched
        assert np.all(np.isnan(Cn[:, :s0])) and np.all(np.isnan(Cn[:, s0 + rpb:]))
        return Cn[:, s0:s0 + rpb].reshape(M, N), ref.reshape(M, N), 1e-6
    cdt = torch.float16 if dtype == X.XEMA_F16 else torch.bfloat16
    c_dtype = X.XEMA_F16 if dtype == X.XEMA_F16 else X.XEMA_BF16
    C = torch.empty((M, N), dtype=cdt, device=DEV)
    X.xema_op_gemm(X.gemm_args(dtype, A, M, K, Bm, N, bias_dev := bf16_dev(bias), epi, C, c_dtype, N))
    torch.cuda.synchronize()
    ref = O.gelu_tanh(acc) if epi == X.XEMA_EPI_BIAS_GELU else acc
    rel = 2.0 ** -10 if dtype == X.XEMA_F16 else 2.0 ** -8
    return C.float().cpu().numpy(), ref, rel


@pytest.mark.parametrize("dtype", [X.XEMA_BF16, X.XEMA_F16])
@pytest.mark.parametrize("epi", [X.XEMA_EPI_BIAS, X.XEMA_EPI_BIAS_GELU, X.XEMA_EPI_GATED_RESIDUAL])
@pytest.mark.parametrize("M,N,K", [(300, 768, 256), (1000, 256, 1024), (64, 512, 64), (513, 1024, 320)])
def test_gemm_matches_oracle(dtype, epi, M, N, K):
    gpu, ref, rel = _gemm_case(dtype, M, N, K, epi, seed=M + N + K + epi)
    # fp32 accumulation of K products of unit-scale terms plus output rounding
    _check_close(gpu, ref, rel, 2e-5 * np.sqrt(K), f"gemm dtype={dtype} epi={epi} {M}x{N}x{K}")


def test_gemm_gated_residual_row_maps():
    gpu, ref, rel = _gemm_case(X.XEMA_F16, 3 * 130, 512, 256, X.XEMA_EPI_GATED_RESIDUAL, 5, chunked=True)
    _check_close(gpu, ref, rel, 2e-5 * 16, "gemm gated residual, 3 batches")


def test_gemm_rows_independent_of_m():
    """Row r of C is bit-identical whether the call has M = 600 or only the
    first 100 rows (the chunked block relies on this)."""
    g = _rng(11)
    K, N = 512, 256
    a = torch.from_numpy(_f16(g.standard_normal((600, K)))).to(DEV)
    b = torch.from_numpy(_f16(g.standard_normal((N, K)) / 20)).to(DEV)
    bias = bf16_dev(_bf16_bits(g.standard_normal(N)))
    outs = []
    for M, off in ((600, 0), (100, 0), (77, 300)):
        C = torch.empty((M, N), dtype=torch.float16, device=DEV)
        X.xema_op_gemm(X.gemm_args(X.XEMA_F16, a[off:], M, K, b, N, bias, X.XEMA_EPI_BIAS, C, X.XEMA_F16, N))
        outs.append(C)
    torch.cuda.synchronize()
    assert torch.equal(outs[0][:100], outs[1])
    assert torch.equal(outs[0][300:377], outs[2])


@pytest.mark.parametrize("M,N,K,epi", [
    (16584, 3072, 12288, X.XEMA_EPI_GATED_RESIDUAL),   # 256-row tiles + a 128-row tail launch
    (17776, 12288, 3072, X.XEMA_EPI_BIAS_GELU),        # 256-row tiles only
])
def test_gemm_tile_heights_agree_at_full_size(M, N, K, epi):
    """Large calls run 256-row tiles (and, where that fills the CUs better, a
    second launch of 128-row tiles over the last rows); small calls run
    128-row tiles.  Rows around the split and elsewhere are bit-identical to
    the same rows computed by a small call, and sampled rows match fp64."""
    g = torch.Generator(device=DEV).manual_seed(M + N)
    a = torch.randn(M, K, device=DEV, generator=g).half()
    b = (torch.randn(N, K, device=DEV, generator=g) / np.sqrt(K)).half()
    bias = (torch.randn(N, device=DEV, generator=g) * 0.02).to(torch.bfloat16)
    gated = epi == X.XEMA_EPI_GATED_RESIDUAL
    cdt, c_dtype = (torch.float32, X.XEMA_F32) if gated else (torch.float16, X.XEMA_F16)
    res = torch.randn(M, N, device=DEV, generator=g) if gated else None
    gate = torch.randn(N, device=DEV, generator=g) if gated else None

    def run(r0, rows):
        C = torch.empty((rows, N), dtype=cdt, device=DEV)
        kw = dict(resid=res[r0:], resid_dtype=X.XEMA_F32, ld_resid=N, gate=gate, gate_stride=0) if gated else {}
        X.xema_op_gemm(X.gemm_args(X.XEMA_F16, a[r0:], rows, K, b, N, bias, epi, C, c_dtype, N, **kw))
        return C

    full = run(0, M)
    for r0, rows in ((16300, 200), (0, 96), (M - 150, 150)):
        part = run(r0, rows)
        torch.cuda.synchronize()
        assert torch.equal(full[r0:r0 + rows], part), (r0, rows)
    pick = np.array([0, 1, 16383, 16384, 16385, M // 2, M - 1])
    a64 = a[pick].double().cpu().numpy()
    acc = a64 @ b.double().cpu().numpy().T + bias.double().cpu().numpy()
    if gated:
        ref = res[pick].double().cpu().numpy() + gate.double().cpu().numpy() * acc
        rel = 1e-6
    else:
        ref, rel = O.gelu_tanh(acc), 2.0 ** -10
    _check_close(full[pick].float().cpu().numpy(), ref, rel, 2e-5 * np.sqrt(K), f"gemm {M}x{N}x{K}")


def test_convert_f16_matches_torch():
    g = _rng(12)
    vals = np.concatenate([g.standard_normal(4096) * s for s in (1e-7, 1e-4, 1.0, 1e3)])
    bits = _bf16_bits(vals)
    src = bf16_dev(bits)
    dst = torch.empty(bits.size, dtype=torch.float16, device=DEV)
    X.xema_op_convert_f16(src, dst, bits.size)
    torch.cuda.synchronize()
    assert torch.equal(dst.view(torch.int16), src.to(torch.float16).view(torch.int16))


@pytest.mark.parametrize("head_dim,rope_dims,grid,text_len", [
    (64, (16, 24, 24), (3, 5, 7), 19), (128, (0, 64, 64), (1, 12, 9), 40), (128, (32, 48, 48), (4, 3, 6), 8)])
def test_qk_norm_rope_matches_oracle(head_dim, rope_dims, grid, text_len):
    H, B = 512 // head_dim, 2
    s = W.tiny_shape(batch=B, text_len=text_len, grid=grid, hidden=H * head_dim, heads=H,
                     head_dim=head_dim, mlp_hidden=256, cond_dim=256, rope_dims=rope_dims)
    cfg, req = cfg_of(s), req_of(s)
    L, D = s.seq_len, s.hidden
    Lp = X.padded_len(L)
    g = _rng(head_dim + L)
    qkv = _f16(g.standard_normal((B, L, 3 * D)) * 1.5)
    gam = {n: _bf16_bits(1 + 0.1 * g.standard_normal(head_dim)) for n in ("q", "k")}
    table = torch.empty(max(1, sum(gr * d // 2 for gr, d in zip(grid, rope_dims))) * 2,
                        dtype=torch.float32, device=DEV)
    X.xema_op_rope_table(cfg, req, table)
    fill = torch.tensor(float("nan"), dtype=torch.float16)
    q = torch.full((B, H, Lp, head_dim), fill.item(), dtype=torch.float16, device=DEV)
    k = torch.full_like(q, fill.item())
    vt = torch.full((B, H, head_dim, Lp), fill.item(), dtype=torch.float16, device=DEV)
    # phase A in two uneven chunks (the second ends at L and zeroes the padding)
    cut = 37
    for t0, cnt in ((0, cut), (cut, L - cut)):
        part = torch.from_numpy(np.ascontiguousarray(qkv[:, t0:t0 + cnt])).to(DEV)
        X.xema_op_qk_norm_rope(cfg, req, part, t0, cnt, bf16_dev(gam["q"]), bf16_dev(gam["k"]), table,
                               q, k, vt)
    torch.cuda.synchronize()
    ang = O.rope_angles(O.token_coords(text_len, grid), rope_dims, head_dim, 10000.0)
    q64 = qkv.astype(np.float64)
    for which, out, gname in ((0, q, "q"), (1, k, "k")):
        z = q64[:, :, which * D:(which + 1) * D].reshape(B, L, H, head_dim)
        ref = np.stack([O.rope_rotate(O.rms_norm(z[b], W.bf16_bits_to_f64(gam[gname]), 1e-6), ang)
                        for b in range(B)])           # [B, L, H, d]
        if which == 0:   # stored queries carry the softmax factor log2(e)/sqrt(d)
            ref = ref * (LOG2E / np.sqrt(head_dim))
        got = out.float().cpu().numpy()
        _check_close(got[:, :, :L].transpose(0, 2, 1, 3), ref, 2.0 ** -10, 1e-4, f"qk_norm_rope {gname}")
        assert np.all(got[:, :, L:] == 0)
    vref = q64[:, :, 2 * D:].reshape(B, L, H, head_dim).transpose(0, 2, 3, 1)
    got = vt.float().cpu().numpy()
    assert np.array_equal(got[..., :L], vref)
    assert np.all(got[..., L:] == 0)


def _attention_case(qs, k, v, q0, qn, what, ref=None):
    """Run the attention op on queries pre-multiplied by log2(e)/sqrt(d)
    (weights 2^(qs . k)) and compare with `ref` ([B, qn, H, d]), by default
    the oracle's."""
    B, H, L, head_dim = qs.shape
    Lp = X.padded_len(L)
    q = qs.astype(np.float64) * (np.sqrt(head_dim) / LOG2E)
    qd = torch.zeros((B, H, Lp, head_dim), dtype=torch.float16, device=DEV)
    kd = torch.zeros_like(qd)
    vtd = torch.zeros((B, H, head_dim, Lp), dtype=torch.float16, device=DEV)
    qd[:, :, :L] = torch.from_numpy(qs).to(DEV)
    kd[:, :, :L] = torch.from_numpy(k).to(DEV)
    vtd[:, :, :, :L] = torch.from_numpy(np.ascontiguousarray(v.transpose(0, 1, 3, 2))).to(DEV)
    o = torch.empty((B * qn, H * head_dim), dtype=torch.float16, device=DEV)
    X.xema_op_attention(qd, kd, vtd, B, H, head_dim, L, Lp, q0, qn, o)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().reshape(B, qn, H, head_dim)
    if ref is None:
        ref = np.empty((B, qn, H, head_dim))
        for b in range(B):
            for h in range(H):
                ref[b, :, h] = O.attention(q[b, h, q0:q0 + qn], k[b, h].astype(np.float64),
                                           v[b, h].astype(np.float64))
    _check_close(got, ref, 2.0 ** -9, 2e-3, what)


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("L,q0,qn,scale", [(300, 0, 300, 1.0), (1000, 129, 700, 1.0), (1025, 0, 1025, 4.0),
                                             (64, 0, 64, 1.0), (1, 0, 1, 1.0)])
def test_attention_matches_oracle(head_dim, L, q0, qn, scale):
    B, H = 2, 3
    g = _rng(L + head_dim)
    qs = _f16(g.standard_normal((B, H, L, head_dim)) * (scale * LOG2E / np.sqrt(head_dim)))
    k = _f16(g.standard_normal((B, H, L, head_dim)) * scale)
    v = _f16(g.standard_normal((B, H, L, head_dim)))
    _attention_case(qs, k, v, q0, qn, f"attention d={head_dim} L={L} q=[{q0},{q0 + qn}) x{scale}")


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("profile", ["jump", "climb", "spike"])
def test_attention_rescaling(head_dim, profile):
    """Score profiles (log2 units, key index j) that drive the lazy reference
    max: "jump" lifts the last 129 keys by 7.5, so a tile's P sum crosses the
    trigger and the 896 earlier keys still carry a few percent of the weight
    (a wrong rescale factor shows); "climb" rises by 20 per 64-key tile, so
    the reference moves on every tile and the unshifted P of the common path
    overflows fp16 before the rescale recomputes it; "spike" puts one key 60
    above the rest.  Every query sees the same profile through its first
    coordinate; the others add a little noise."""
    B, H = 1, 2
    L = 1000 if profile == "climb" else 1025
    j = np.arange(L, dtype=np.float64)
    lift = {"jump": np.where(j >= 896, 7.5, 0.0),
            "climb": 20.0 * np.floor(j / 64),
            "spike": np.where(j == 700, 60.0, 0.0)}[profile]
    g = _rng({"jump": 301, "climb": 302, "spike": 303}[profile] + head_dim)
    qs = np.concatenate([np.ones((B, H, L, 1)), 0.02 * g.standard_normal((B, H, L, head_dim - 1))], axis=-1)
    k = g.standard_normal((B, H, L, head_dim))
    k[..., 0] = lift
    qs, k = _f16(qs), _f16(k)
    v = _f16(g.standard_normal((B, H, L, head_dim)))
    _attention_case(qs, k, v, 0, L, f"attention d={head_dim} rescaling profile {profile}")


@pytest.mark.parametrize("head_dim", [64, 128])
def test_attention_equal_keys_average_v(head_dim):
    """P10 on the GPU, against the closed form rather than the oracle: with
    every key of a head equal, all scores of a query are equal and its output
    is the mean of the head's V rows (1000 keys: fifteen full tiles and a
    ragged tail)."""
    B, H, L = 1, 2, 1000
    g = _rng(400 + head_dim)
    qs = _f16(g.standard_normal((B, H, L, head_dim)) * (LOG2E / np.sqrt(head_dim)))
    k = np.ascontiguousarray(np.repeat(_f16(g.standard_normal((B, H, 1, head_dim))), L, axis=2))
    v = _f16(g.standard_normal((B, H, L, head_dim)))
    mean_v = v.astype(np.float64).mean(axis=2)                      # [B, H, d]
    ref = np.broadcast_to(mean_v[:, None, :, :], (B, L, H, head_dim))
    _attention_case(qs, k, v, 0, L, f"attention d={head_dim}, equal keys", ref)


def test_attention_queries_independent_of_range():
    """A query's output is bit-identical whatever query range it is computed in."""
    B, H, L, hd = 1, 2, 777, 64
    Lp = X.padded_len(L)
    g = _rng(21)
    qd = torch.zeros((B, H, Lp, hd), dtype=torch.float16, device=DEV)
    kd = torch.zeros_like(qd)
    vtd = torch.zeros((B, H, hd, Lp), dtype=torch.float16, device=DEV)
    qd[:, :, :L] = torch.from_numpy(_f16(g.standard_normal((B, H, L, hd)))).to(DEV)
    kd[:, :, :L] = torch.from_numpy(_f16(g.standard_normal((B, H, L, hd)))).to(DEV)
    vtd[:, :, :, :L] = torch.from_numpy(_f16(g.standard_normal((B, H, hd, L)))).to(DEV)
    full = torch.empty((L, H * hd), dtype=torch.float16, device=DEV)
    X.xema_op_attention(qd, kd, vtd, B, H, hd, L, Lp, 0, L, full)
    for q0, qn in ((0, 100), (100, 33), (500, 277), (776, 1)):
        part = torch.empty((qn, H * hd), dtype=torch.float16, device=DEV)
        X.xema_op_attention(qd, kd, vtd, B, H, hd, L, Lp, q0, qn, part)
        torch.cuda.synchronize()
        assert torch.equal(part, full[q0:q0 + qn]), (q0, qn)
