"""C ABI checks that need no GPU: the library loads and exports every symbol
the headers declare; the C++ planner (Algorithm 1 + chunk plan) matches the
Python oracle byte for byte; host-side validation returns the documented
status codes before any device work."""
import ctypes
import os
import re

import pytest

import paper_2607_11136_amd as X
import workloads as W
from oracle import layout as OL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _cfg(s: W.BlockShape):
    return X.block_cfg(s.hidden, s.heads, s.head_dim, s.mlp_hidden, s.cond_dim, s.rope_dims,
                       s.rope_theta, s.ln_eps, s.qk_eps, s.modulation_streams)


def _req(s: W.BlockShape):
    return X.request(s.batch, s.text_len, *s.grid)


def _declared_symbols():
    names = set()
    for h in ("xema.h", "xema_ops.h", "xema_step.h", "xema_vae.h", "xema_static.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        names.update(re.findall(r"XEMA_API\s+[\w\s\*]+?\b(xema_\w+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    lib = X.lib()
    declared = _declared_symbols()
    assert len(declared) == 28, declared
    for name in declared:
        assert hasattr(lib, name), name
    assert declared == set(X.EXPORTED)


def test_status_strings():
    assert X.xema_status_str(0) == "ok"
    assert "budget" in X.xema_status_str(X.XEMA_ERR_BUDGET_TOO_SMALL)


@pytest.mark.parametrize("name", sorted(W.CONFIGS))
def test_layout_matches_oracle(name):
    s = W.CONFIGS[name]
    for chunk in sorted({0, 1, 64, 100, 256, 2048, 8192} | set(s.chunks)):
        p = X.xema_workspace_layout(_cfg(s), _req(s), chunk)
        ts = OL.block_tensors(s.batch, s.seq_len, s.hidden, s.mlp_hidden, s.grid, s.rope_dims, chunk,
                              s.modulation_streams)
        offs, peak = OL.static_layout(ts)
        assert p.n_slots == len(ts) == len(X.SLOT_NAMES)
        assert p.workspace_bytes == peak
        assert list(p.slot_offset[:p.n_slots]) == offs
        assert list(p.slot_bytes[:p.n_slots]) == [OL.round_up(t.size, OL.ALIGN) for t in ts]
        assert list(p.slot_begin[:p.n_slots]) == [t.begin for t in ts]
        assert list(p.slot_end[:p.n_slots]) == [t.end for t in ts]
        c = s.seq_len if chunk <= 0 or chunk >= s.seq_len else chunk
        assert p.chunk_tokens == c
        assert X.xema_workspace_bytes(_cfg(s), _req(s), chunk) == peak


@pytest.mark.parametrize("name", ["tiny", "video", "highres", "long"])
def test_plan_matches_oracle(name):
    s = W.CONFIGS[name]
    smallest = min(OL.workspace_bytes(s, c) for c in OL.chunk_candidates(s.seq_len))
    full = OL.workspace_bytes(s, 0)
    for budget in sorted({smallest, smallest + 12345, (smallest + full) // 2, full - 1, full,
                          32 * 10**9}):
        c, ws, small = OL.plan(s, budget)
        if c is None:   # a chunked arena can exceed the unchunked one on short sequences
            with pytest.raises(X.XemaError) as e:
                X.xema_workspace_plan(_cfg(s), _req(s), budget)
            assert e.value.status == X.XEMA_ERR_BUDGET_TOO_SMALL
            assert e.value.plan.min_workspace_bytes == small
            continue
        p = X.xema_workspace_plan(_cfg(s), _req(s), budget)
        assert (p.chunk_tokens, p.workspace_bytes, p.min_workspace_bytes) == (c, ws, small)


def test_plan_budget_too_small_reports_minimum():
    s = W.HIGHRES
    smallest = min(OL.workspace_bytes(s, c) for c in OL.chunk_candidates(s.seq_len))
    assert smallest == OL.workspace_bytes(s, 256)   # Q, K, V dominate: the smallest chunk is the smallest arena
    with pytest.raises(X.XemaError) as e:
        X.xema_workspace_plan(_cfg(s), _req(s), smallest - 1)
    assert e.value.status == X.XEMA_ERR_BUDGET_TOO_SMALL
    assert e.value.plan.min_workspace_bytes == smallest
    assert e.value.plan.chunk_tokens == 0


def test_highres_32gb_budget_runs_unchunked():
    s = W.HIGHRES
    p = X.xema_workspace_plan(_cfg(s), _req(s), 32 * 2**30)
    assert p.chunk_tokens == s.seq_len
    assert p.workspace_bytes <= 32 * 2**30


@pytest.mark.parametrize("name", ["image_b4", "long", "tiny"])
def test_serial_plan_matches_oracle(name):
    """Temporary serialization: per group size the largest chunk that fits,
    then the least modelled block time (oracle.layout.block_ms); the batch
    stays whole when chunking alone fits it at no modelled cost."""
    s = W.CONFIGS[name]
    cfg, req = _cfg(s), _req(s)
    cands = OL.chunk_candidates(s.seq_len)
    full_min = min(OL.workspace_bytes(s, c) for c in cands)
    one = s.with_(batch=1)
    one_min = min(OL.workspace_bytes(one, c) for c in cands)
    budgets = [OL.workspace_bytes(s, 0), full_min, full_min - 1, (full_min + one_min) // 2, one_min, one_min - 1]
    for budget in budgets:
        ref = OL.plan_serial(s, budget)
        if ref is None:
            with pytest.raises(X.XemaError) as e:
                X.xema_workspace_plan_serial(cfg, req, budget)
            assert e.value.status == X.XEMA_ERR_BUDGET_TOO_SMALL
            assert e.value.plan.min_workspace_bytes == one_min
            continue
        g, p = X.xema_workspace_plan_serial(cfg, req, budget)
        assert (g, p.chunk_tokens, p.workspace_bytes) == ref, (budget, ref)
        assert p.workspace_bytes <= budget
        if budget >= OL.workspace_bytes(s, 0):
            assert (g, p.chunk_tokens) == (s.batch, s.seq_len)   # no mitigation at all
        if budget < full_min:
            assert g < s.batch   # chunking alone cannot fit the whole batch


@pytest.mark.parametrize("hwt,grid", [((1024, 1024, 1), (1, 64, 64)), ((480, 720, 49), (13, 30, 45)),
                                      ((1080, 1920, 49), (13, 68, 120)), ((352, 608, 129), (33, 22, 38))])
def test_request_from_template(hwt, grid):
    r = X.xema_request_from_template(_cfg(W.VIDEO), *hwt, 1, 226)
    assert (r.grid_t, r.grid_h, r.grid_w) == grid
    assert (r.batch, r.text_len) == (1, 226)


def _bad_cfg(**kw):
    s = W.TINY
    c = _cfg(s)
    for k, v in kw.items():
        if k == "rope_dims":
            for i in range(3):
                c.rope_dims[i] = v[i]
        else:
            setattr(c, k, v)
    return c


@pytest.mark.parametrize("kw,status", [
    ({"head_dim": 32, "heads": 8, "rope_dims": (8, 12, 12)}, X.XEMA_ERR_UNSUPPORTED),
    ({"heads": 3}, X.XEMA_ERR_INVALID_ARG),
    ({"hidden": 320, "heads": 5}, X.XEMA_ERR_UNSUPPORTED),
    ({"mlp_hidden": 1000}, X.XEMA_ERR_UNSUPPORTED),
    ({"rope_dims": (16, 24, 25)}, X.XEMA_ERR_INVALID_ARG),
    ({"rope_dims": (32, 24, 24)}, X.XEMA_ERR_INVALID_ARG),
    ({"ln_eps": 0.0}, X.XEMA_ERR_INVALID_ARG),
    ({"cond_dim": 12}, X.XEMA_ERR_UNSUPPORTED),
])
def test_bad_shapes_rejected(kw, status):
    with pytest.raises(X.XemaError) as e:
        X.xema_workspace_layout(_bad_cfg(**kw), _req(W.TINY), 0)
    assert e.value.status == status


def test_bad_request_rejected():
    for r in (X.request(0, 32, 1, 16, 16), X.request(1, -1, 1, 16, 16), X.request(1, 0, 0, 0, 0)):
        with pytest.raises(X.XemaError) as e:
            X.xema_workspace_layout(_cfg(W.TINY), r, 0)
        assert e.value.status == X.XEMA_ERR_INVALID_ARG


# Host-side validation of the forward call.  The addresses below are never
# dereferenced: every case fails validation before any HIP call.
BASE = 1 << 40


def _fake_call(s, chunk=0, ws_bytes=None, ws_addr=None, out_addr=None, tok_addr=None, w_over=None):
    cfg, req = _cfg(s), _req(s)
    need = X.xema_workspace_bytes(cfg, req, chunk)
    ws_bytes = need if ws_bytes is None else ws_bytes
    addr = BASE
    tok = BASE + (1 << 34) if tok_addr is None else tok_addr
    out = BASE + (2 << 34) if out_addr is None else out_addr
    ws = BASE + (3 << 34) if ws_addr is None else ws_addr
    cond = BASE + (4 << 34)
    w = X.BlockWeights()
    for i, n in enumerate(X.WEIGHT_FIELDS):
        setattr(w, n, BASE + (5 << 34) + i * (1 << 30))
    for k, v in (w_over or {}).items():
        setattr(w, k, v)
    return X.lib().xema_dit_block_fwd(ctypes.byref(cfg), ctypes.byref(req), tok, ctypes.byref(w),
                                      cond, chunk, ws, ws_bytes, out, None)


def test_fwd_workspace_too_small():
    assert _fake_call(W.TINY, ws_bytes=1000) == X.XEMA_ERR_WORKSPACE_TOO_SMALL
    need64 = X.xema_workspace_bytes(_cfg(W.TINY), _req(W.TINY), 64)
    assert _fake_call(W.TINY, chunk=0, ws_bytes=need64) == X.XEMA_ERR_WORKSPACE_TOO_SMALL


def test_fwd_misaligned():
    assert _fake_call(W.TINY, ws_addr=BASE + (3 << 34) + 128) == X.XEMA_ERR_MISALIGNED
    assert _fake_call(W.TINY, out_addr=BASE + (2 << 34) + 8) == X.XEMA_ERR_MISALIGNED
    assert _fake_call(W.TINY, w_over={"qkv_w": BASE + (9 << 34) + 4}) == X.XEMA_ERR_MISALIGNED


def test_fwd_aliasing_rejected():
    # out overlapping tokens, or the workspace overlapping a weight
    assert _fake_call(W.TINY, out_addr=BASE + (1 << 34) + 4096) == X.XEMA_ERR_INVALID_ARG
    assert _fake_call(W.TINY, w_over={"o_w": BASE + (3 << 34) + 1024}) == X.XEMA_ERR_INVALID_ARG
    assert _fake_call(W.TINY, w_over={"down_b": None}) == X.XEMA_ERR_INVALID_ARG


def test_dual_stream_validation():
    s = W.TINY.with_(modulation_streams=2)
    txt = {"ada_txt_w": BASE + (6 << 34), "ada_txt_b": BASE + (6 << 34) + (1 << 30)}
    # a dual-stream block needs the text tokens' map (a single-stream one ignores it)
    assert _fake_call(s) == X.XEMA_ERR_INVALID_ARG
    assert _fake_call(s, w_over=dict(txt, ada_txt_b=None)) == X.XEMA_ERR_INVALID_ARG
    assert _fake_call(s, w_over=dict(txt, ada_txt_w=BASE + (6 << 34) + 8)) == X.XEMA_ERR_MISALIGNED
    assert _fake_call(s, w_over=dict(txt, ada_txt_w=BASE + (2 << 34))) == X.XEMA_ERR_INVALID_ARG  # in out
    assert _fake_call(s, w_over=dict(txt, ada_txt_b=BASE + (3 << 34) + 512)) == X.XEMA_ERR_INVALID_ARG  # in ws
    assert _fake_call(s, w_over=txt, ws_bytes=X.xema_workspace_bytes(_cfg(W.TINY), _req(W.TINY), 0)) == \
        X.XEMA_ERR_WORKSPACE_TOO_SMALL  # the mod slot doubles
    for streams, ok in ((0, True), (1, True), (2, True), (3, False), (-1, False)):
        c = _cfg(W.TINY)
        c.modulation_streams = streams
        if ok:
            X.xema_workspace_layout(c, _req(W.TINY), 0)
        else:
            with pytest.raises(X.XemaError) as e:
                X.xema_workspace_layout(c, _req(W.TINY), 0)
            assert e.value.status == X.XEMA_ERR_INVALID_ARG


def test_vae_upconv_validation():
    lib = X.lib()
    n = ctypes.c_int64()
    # 4 phases x co x 8 (hi and lo of 4 taps) x ci bf16
    assert lib.xema_vae_upconv_weight_bytes(256, 512, ctypes.byref(n)) == X.XEMA_OK and n.value == 64 * 256 * 512
    assert lib.xema_vae_upconv_weight_bytes(96, 256, ctypes.byref(n)) == X.XEMA_ERR_UNSUPPORTED
    assert lib.xema_vae_upconv_weight_bytes(64, 128, ctypes.byref(n)) == X.XEMA_ERR_UNSUPPORTED
    assert lib.xema_vae_upconv_weight_bytes(0, 256, ctypes.byref(n)) == X.XEMA_ERR_INVALID_ARG
    x, wp, b, y = BASE, BASE + (1 << 34), BASE + (2 << 34), BASE + (3 << 34)
    f = lib.xema_vae_upconv
    # every case fails validation before any launch
    assert f(None, 1, 4, 4, 64, wp, b, 256, 0, 4, y, None) == X.XEMA_ERR_INVALID_ARG
    assert f(x, 1, 4, 4, 64, wp, b, 256, 3, 2, y, None) == X.XEMA_ERR_INVALID_ARG      # rows past h
    assert f(x, 1, 4, 4, 64, wp, b, 256, -1, 2, y, None) == X.XEMA_ERR_INVALID_ARG
    assert f(x, 1, 4, 4, 64, wp, b, 256, 0, 0, y, None) == X.XEMA_ERR_INVALID_ARG
    assert f(x, 1, 4, 4, 80, wp, b, 256, 0, 4, y, None) == X.XEMA_ERR_UNSUPPORTED
    assert f(x, 64, 512, 512, 128, wp, b, 256, 0, 4, y, None) == X.XEMA_ERR_UNSUPPORTED  # input >= 2 GiB
    assert f(x + 8, 1, 4, 4, 64, wp, b, 256, 0, 4, y, None) == X.XEMA_ERR_MISALIGNED
    assert f(x, 1, 4, 4, 64, wp, b, 256, 0, 4, x + 256, None) == X.XEMA_ERR_INVALID_ARG  # y overlaps x
    assert lib.xema_vae_upconv_prepare(wp, 64, 256, wp + 1024, None) == X.XEMA_ERR_INVALID_ARG  # overlap
    assert lib.xema_vae_upconv_prepare(wp + 4, 64, 256, y, None) == X.XEMA_ERR_MISALIGNED


def test_op_validation():
    L = X.lib()
    f = BASE
    # attention: head_dim 96 unsupported; padded_len not a multiple of 128
    assert L.xema_op_attention(f, f, f, 1, 4, 96, 300, 384, 0, 300, f + (1 << 30), None) == X.XEMA_ERR_UNSUPPORTED
    assert L.xema_op_attention(f, f, f, 1, 4, 64, 300, 320, 0, 300, f + (1 << 30), None) == X.XEMA_ERR_UNSUPPORTED
    assert L.xema_op_attention(f, f, f, 1, 4, 64, 300, 384, 200, 200, f + (1 << 30), None) == X.XEMA_ERR_INVALID_ARG
    # gemm: N not a multiple of 256
    g = X.gemm_args(X.XEMA_BF16, f, 100, 256, f, 300, f, X.XEMA_EPI_BIAS, f + (1 << 30), X.XEMA_F16, 300)
    assert L.xema_op_gemm(ctypes.byref(g), None) == X.XEMA_ERR_UNSUPPORTED
    g = X.gemm_args(X.XEMA_BF16, f + 2, 100, 256, f, 256, f, X.XEMA_EPI_BIAS, f + (1 << 30), X.XEMA_F16, 256)
    assert L.xema_op_gemm(ctypes.byref(g), None) == X.XEMA_ERR_MISALIGNED
    # gated residual needs fp32 output
    g = X.gemm_args(X.XEMA_F16, f, 100, 256, f, 256, f, X.XEMA_EPI_GATED_RESIDUAL, f + (1 << 30),
                    X.XEMA_F16, 256, resid=f, ld_resid=256, gate=f)
    assert L.xema_op_gemm(ctypes.byref(g), None) == X.XEMA_ERR_UNSUPPORTED
    # the fused QKV-heads epilogues (codes 3 and 4, head dims 64 and 128) are
    # internal to the block forward
    for code in (3, 4):
        g = X.gemm_args(X.XEMA_BF16, f, 100, 256, f, 256, f, code, f + (1 << 30), X.XEMA_F16, 256)
        assert L.xema_op_gemm(ctypes.byref(g), None) == X.XEMA_ERR_INVALID_ARG, code
    # LN: dim not a multiple of 256
    assert L.xema_op_ln_modulate(f, X.XEMA_BF16, X.rowmap(4, 4, 0), 4, 300, f, f, 1800, 1e-6, f,
                                 X.XEMA_BF16, None) == X.XEMA_ERR_UNSUPPORTED
    # convert: overlapping buffers
    assert L.xema_op_convert_f16(f, f + 16, 1024, None) == X.XEMA_ERR_INVALID_ARG
