"""Pins of the fp64 oracle against what the definition and mathematics fix.

Each test checks the oracle against something other than itself: closed forms,
invariants, textbook/library special cases (torch fp64 CPU ops), and the
independent scalar brute force.  test_planted_mistakes_are_caught then plants
plausible mistakes in the oracle and checks that a pin fails for each.
"""
import math

import numpy as np
import pytest
import torch

import workloads as W
from oracle import block as O
from oracle import brute


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _weights(shape: W.BlockShape):
    inp = W.make_inputs(shape)
    return inp.f64("x"), inp.f64("cond"), inp.weights_f64()


def _kw(s: W.BlockShape, **over):
    kw = dict(heads=s.heads, head_dim=s.head_dim, text_len=s.text_len, grid=s.grid,
              rope_dims=s.rope_dims, rope_theta=s.rope_theta, ln_eps=s.ln_eps, qk_eps=s.qk_eps)
    kw.update(over)
    return kw


def _nested(a):
    return a.tolist()


def _brute(x, cond, w, s, **over):
    kw = _kw(s, **over)
    return np.array(brute.block_forward(_nested(x), _nested(cond), {k: _nested(v) for k, v in w.items()}, **kw))


# -- P1: softmax rows sum to one -------------------------------------------------------


def test_p1_softmax_rows_sum_to_one():
    s = _rand((64, 300), 1, scale=30.0)
    p = O.softmax_rows(s)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(axis=-1) - 1.0)) <= 1e-12
    # and the attention weights the block uses on real (q, k) pairs
    q = _rand((50, 16), 2)
    k = _rand((70, 16), 3)
    p = O.softmax_rows(q @ k.T / 4.0)
    assert np.max(np.abs(p.sum(axis=-1) - 1.0)) <= 1e-12


# -- P2: zero-angle RoPE is the identity -------------------------------------------------


def test_p2_zero_angle_rope_is_identity():
    z = _rand((10, 3, 12), 4)
    assert np.array_equal(O.rope_rotate(z, np.zeros((10, 6))), z)


def test_p2_rope_off_equals_all_positions_zero():
    s = W.tiny_shape()
    x, c, w = _weights(s)
    off = O.block_forward(x, c, w, **_kw(s, rope_dims=(0, 0, 0)))
    zero_coords = np.zeros((s.seq_len, 3), dtype=np.int64)
    at_zero = O.block_forward(x, c, w, **_kw(s), coords=zero_coords)
    np.testing.assert_allclose(at_zero, off, rtol=0, atol=1e-12)


def test_p2_single_cell_grid_rotates_nothing():
    s = W.tiny_shape(grid=(1, 1, 1), text_len=5)
    ang = O.rope_angles(O.token_coords(s.text_len, s.grid), s.rope_dims, s.head_dim, s.rope_theta)
    assert np.all(ang == 0.0)


def test_p2_time_segment_unrotated_for_single_frame():
    s = W.TINY  # G_t = 1
    ang = O.rope_angles(O.token_coords(s.text_len, s.grid), s.rope_dims, s.head_dim, s.rope_theta)
    assert np.all(ang[:, : s.rope_dims[0] // 2] == 0.0)
    assert np.any(ang[:, s.rope_dims[0] // 2:] != 0.0)


# -- P3: without RoPE, permuting tokens permutes outputs ------------------------------------


def test_p3_permutation_equivariance_without_rope():
    s = W.tiny_shape(text_len=4, grid=(2, 3, 4), hidden=32, heads=2, head_dim=16, mlp_hidden=64,
                     cond_dim=32)
    x, c, w = _weights(s)
    perm = np.random.default_rng(5).permutation(s.seq_len)
    kw = _kw(s, rope_dims=(0, 0, 0))
    a = O.block_forward(x, c, w, **kw)
    b = O.block_forward(x[:, perm], c, w, **kw)
    np.testing.assert_allclose(b, a[:, perm], rtol=0, atol=1e-12)
    # with RoPE on, the same permutation must change the result
    kw_on = _kw(s, rope_dims=(4, 6, 6))
    a_on = O.block_forward(x, c, w, **kw_on)
    b_on = O.block_forward(x[:, perm], c, w, **kw_on)
    assert np.max(np.abs(b_on - a_on[:, perm])) > 1e-6


# -- P4: one token => attention returns v ---------------------------------------------------


def test_p4_single_key_returns_v():
    q = _rand((5, 8), 6)
    k = _rand((1, 8), 7)
    v = _rand((1, 8), 8)
    np.testing.assert_array_equal(O.attention(q, k, v), np.repeat(v, 5, axis=0))


def test_p4_one_token_block_branch_is_projected_v():
    s = W.tiny_shape(text_len=1, grid=(0, 1, 1))
    assert s.seq_len == 1
    x, c, w = _weights(s)
    out = O.block_forward(x, c, w, **_kw(s))
    D = s.hidden
    # closed form: attention output = v, so x1 = x + gate1 * (W_o v + b_o)
    m = c @ w["ada_w"].T + w["ada_b"]
    xb = x[0, 0]
    mu, var = xb.mean(), xb.var()
    h = (xb - mu) / math.sqrt(var + s.ln_eps) * (1 + m[0, D:2 * D]) + m[0, :D]
    v = w["qkv_w"][2 * D:] @ h + w["qkv_b"][2 * D:]
    x1 = xb + m[0, 2 * D:3 * D] * (w["o_w"] @ v + w["o_b"])
    mu2, var2 = x1.mean(), x1.var()
    h2 = (x1 - mu2) / math.sqrt(var2 + s.ln_eps) * (1 + m[0, 4 * D:5 * D]) + m[0, 3 * D:4 * D]
    u = w["up_w"] @ h2 + w["up_b"]
    g = np.array([0.5 * t * (1 + math.tanh(math.sqrt(2 / math.pi) * (t + 0.044715 * t ** 3))) for t in u])
    ref = x1 + m[0, 5 * D:] * (w["down_w"] @ g + w["down_b"])
    np.testing.assert_allclose(out[0, 0], ref, rtol=1e-12, atol=1e-12)


# -- P5: scalar brute force ------------------------------------------------------------------


@pytest.mark.parametrize("over", [
    {},
    {"batch": 2},
    {"text_len": 0, "grid": (2, 3, 2), "rope_dims": (4, 4, 2)},
    {"grid": (1, 3, 4), "rope_dims": (0, 6, 6)},
])
def test_p5_brute_force_matches(over):
    s = W.tiny_shape(**over)
    x, c, w = _weights(s)
    a = O.block_forward(x, c, w, **_kw(s))
    b = _brute(x, c, w, s)
    rel = np.max(np.abs(a - b)) / np.max(np.abs(b))
    assert rel <= 1e-12, rel


# -- P6: zero gates give out == x exactly -----------------------------------------------------


def test_p6_zero_gates_pass_tokens_through():
    s = W.tiny_shape()
    x, c, w = _weights(s)
    D = s.hidden
    w = dict(w)
    w["ada_w"] = w["ada_w"].copy()
    w["ada_b"] = w["ada_b"].copy()
    for blk in (2, 5):
        w["ada_w"][blk * D:(blk + 1) * D] = 0.0
        w["ada_b"][blk * D:(blk + 1) * D] = 0.0
    out = O.block_forward(x, c, w, **_kw(s))
    assert np.array_equal(out, x)


# -- P7: library special cases (torch fp64 CPU) -------------------------------------------------


def test_p7_layer_norm_matches_torch():
    x = _rand((7, 40), 9, scale=3.0) + 2.0
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (40,), eps=1e-6).numpy()
    np.testing.assert_allclose(O.layer_norm(x, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_p7_rms_norm_matches_torch():
    z = _rand((7, 3, 16), 10)
    g = 1 + 0.1 * _rand((16,), 11)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(z), (16,), weight=torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(O.rms_norm(z, g, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_p7_attention_matches_torch_sdpa():
    q, k, v = _rand((33, 16), 12), _rand((57, 16), 13), _rand((57, 16), 14)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None])[0].numpy()
    np.testing.assert_allclose(O.attention(q, k, v, row_group=8), ref, rtol=1e-11, atol=1e-12)


def test_p7_gelu_matches_torch():
    u = np.linspace(-12, 12, 2001)
    ref = torch.nn.functional.gelu(torch.from_numpy(u), approximate="tanh").numpy()
    np.testing.assert_allclose(O.gelu_tanh(u), ref, rtol=1e-12, atol=1e-14)


def test_p7_linear_matches_torch():
    x, wt, b = _rand((5, 12), 15), _rand((9, 12), 16), _rand((9,), 17)
    ref = torch.nn.functional.linear(torch.from_numpy(x), torch.from_numpy(wt), torch.from_numpy(b)).numpy()
    np.testing.assert_allclose(O.linear(x, wt, b), ref, rtol=1e-12, atol=1e-12)


# -- P8: GELU closed forms -------------------------------------------------------------------


def test_p8_gelu_odd_part_and_zero():
    u = np.linspace(-9, 9, 1001)
    np.testing.assert_allclose(O.gelu_tanh(u) - O.gelu_tanh(-u), u, rtol=0, atol=1e-13)
    assert O.gelu_tanh(np.array([0.0]))[0] == 0.0


# -- P9: RoPE is a rotation, and attention sees relative positions -----------------------------


def test_p9_rope_is_complex_rotation_and_preserves_pair_norms():
    L, H, d = 9, 2, 12
    z = _rand((L, H, d), 18)
    ang = _rand((L, d // 2), 19, scale=5.0)
    r = O.rope_rotate(z, ang)
    # as complex multiplication (u0 + i u1) * exp(i phi)
    zc = (z[..., 0::2] + 1j * z[..., 1::2]) * np.exp(1j * ang)[:, None, :]
    np.testing.assert_allclose(r[..., 0::2], zc.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(r[..., 1::2], zc.imag, rtol=0, atol=1e-12)
    n0 = z[..., 0::2] ** 2 + z[..., 1::2] ** 2
    n1 = r[..., 0::2] ** 2 + r[..., 1::2] ** 2
    np.testing.assert_allclose(n1, n0, rtol=1e-12)


def test_p9_rope_frequencies_closed_form():
    # pair j of a segment of width d_a turns by p * theta^(-2j/d_a)
    coords = np.array([[-1, -1, -1], [3, 1, 2]])
    ang = O.rope_angles(coords, (4, 4, 2), 12, 10000.0)
    assert np.all(ang[0] == 0.0)
    # t segment: pairs 0,1 -> 3*1, 3*10000^-0.5 ; y segment: 1, 1e-2 ; w: 2
    np.testing.assert_allclose(ang[1], [3.0, 0.03, 1.0, 0.01, 2.0, 0.0], rtol=1e-15)


def test_p9_grid_shift_leaves_block_unchanged():
    s = W.tiny_shape(text_len=0, grid=(2, 2, 3))
    x, c, w = _weights(s)
    coords = O.token_coords(0, s.grid)
    a = O.block_forward(x, c, w, **_kw(s), coords=coords)
    b = O.block_forward(x, c, w, **_kw(s), coords=coords + np.array([5, 7, 11]))
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-11)
    # a shift along one axis only changes nothing either; a scaling does
    b2 = O.block_forward(x, c, w, **_kw(s), coords=coords * 2)
    assert np.max(np.abs(b2 - a)) > 1e-6


# -- P10: closed forms of attention and LayerNorm ---------------------------------------------


def test_p10_equal_keys_average_values():
    q = _rand((6, 8), 20)
    k = np.repeat(_rand((1, 8), 21), 40, axis=0)
    v = _rand((40, 8), 22)
    np.testing.assert_allclose(O.attention(q, k, v), np.repeat(v.mean(0, keepdims=True), 6, 0),
                               rtol=0, atol=1e-13)


def test_p10_constant_row_layer_norm_gives_shift():
    x = np.full((3, 16), 2.5)
    shift, scale = _rand((16,), 23), _rand((16,), 24)
    np.testing.assert_array_equal(O.modulate(O.layer_norm(x, 1e-6), shift, scale), np.broadcast_to(shift, (3, 16)))


# -- P11: batch independence, row subsets -------------------------------------------------------


def test_p11_batch_rows_are_independent_runs():
    s = W.tiny_shape(batch=3)
    x, c, w = _weights(s)
    full = O.block_forward(x, c, w, **_kw(s))
    for b in range(3):
        one = O.block_forward(x[b:b + 1], c[b:b + 1], w, **_kw(s))
        np.testing.assert_allclose(full[b:b + 1], one, rtol=0, atol=1e-13)


def test_p11_row_subset_equals_full_rows():
    s = W.TINY
    x, c, w = _weights(s)
    full = O.block_forward(x, c, w, **_kw(s))
    rows = [0, 5, 31, 32, 100, 287]
    sub = O.block_forward(x, c, w, **_kw(s), rows=rows)
    np.testing.assert_allclose(sub, full[:, rows], rtol=0, atol=1e-12)


# -- planted mistakes: every one must break a pin ---------------------------------------------


def _mut_modulate_no_one(xhat, shift, scale):
    return xhat * scale + shift


def _mut_rope_sign(z, angles):
    c = np.cos(angles)[:, None, :]
    s = np.sin(angles)[:, None, :]
    out = np.empty_like(z)
    out[..., 0::2] = z[..., 0::2] * c + z[..., 1::2] * s
    out[..., 1::2] = -z[..., 0::2] * s + z[..., 1::2] * c
    return out


def _mut_rope_half_split(z, angles):
    h = z.shape[-1] // 2
    c = np.cos(angles)[:, None, :]
    s = np.sin(angles)[:, None, :]
    out = np.empty_like(z)
    out[..., :h] = z[..., :h] * c - z[..., h:] * s
    out[..., h:] = z[..., :h] * s + z[..., h:] * c
    return out


def _mut_attention_no_scale(q, k, v, row_group=1024):
    return O.softmax_rows(q @ k.T) @ v


def _mut_ln_unbiased(x, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)
    return (x - mu) / np.sqrt(var + eps)


def _mut_gelu_erf(u):
    return np.array([0.5 * t * (1 + math.erf(t / math.sqrt(2))) for t in np.ravel(u)]).reshape(np.shape(u))


def _mut_split_order(m):
    a = np.split(m, 6, axis=-1)
    return (a[0], a[2], a[1], a[3], a[4], a[5])


def _mut_rms_no_gamma(z, gamma, eps):
    return z / np.sqrt((z * z).mean(axis=-1, keepdims=True) + eps)


def _mut_coords_swap(text_len, grid):
    gt, gh, gw = grid
    n = gt * gh * gw
    out = -np.ones((text_len + n, 3), dtype=np.int64)
    v = np.arange(n)
    out[text_len:, 0] = v // (gh * gw)
    out[text_len:, 1] = v % gw          # row and column swapped
    out[text_len:, 2] = (v // gw) % gh
    return out


def _mut_softmax_no_max(s):
    e = np.exp(s)
    return e / e.sum(axis=-1, keepdims=True) * (1 + 1e-3)


_MUTATIONS = {
    "modulate_without_one": ("modulate", _mut_modulate_no_one),
    "rope_sign": ("rope_rotate", _mut_rope_sign),
    "rope_half_split_pairs": ("rope_rotate", _mut_rope_half_split),
    "attention_without_scale": ("attention", _mut_attention_no_scale),
    "layer_norm_unbiased_var": ("layer_norm", _mut_ln_unbiased),
    "gelu_erf_form": ("gelu_tanh", _mut_gelu_erf),
    "modulation_split_order": ("split_modulation", _mut_split_order),
    "rms_norm_without_gain": ("rms_norm", _mut_rms_no_gamma),
    "grid_axes_swapped": ("token_coords", _mut_coords_swap),
    "softmax_off_by_scale": ("softmax_rows", _mut_softmax_no_max),
}


@pytest.mark.parametrize("name", sorted(_MUTATIONS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, fn = _MUTATIONS[name]
    s = W.tiny_shape(grid=(2, 3, 2), rope_dims=(4, 4, 4))
    x, c, w = _weights(s)
    ref = _brute(x, c, w, s)
    monkeypatch.setattr(O, attr, fn)
    bad = O.block_forward(x, c, w, **_kw(s))
    assert np.max(np.abs(bad - ref)) / np.max(np.abs(ref)) > 1e-9, f"mistake {name} not caught"


# -- P13: dual-stream modulation (reading R24) ---------------------------------------------------


def _dual(**over):
    s = W.tiny_shape(modulation_streams=2, **over)
    return (s,) + _weights(s)


def _single(w):
    return {k: v for k, v in w.items() if k not in W.TEXT_MOD_NAMES}


@pytest.mark.parametrize("over", [{}, {"batch": 2}, {"text_len": 1}])
def test_p13_dual_brute_force_matches(over):
    s, x, c, w = _dual(**over)
    a = O.block_forward(x, c, w, **_kw(s))
    b = _brute(x, c, w, s)
    rel = np.max(np.abs(a - b)) / np.max(np.abs(b))
    assert rel <= 1e-12, rel
    # and the text map does matter
    assert np.max(np.abs(a - O.block_forward(x, c, _single(w), **_kw(s)))) > 1e-3


def test_p13_equal_maps_equal_single_stream():
    s, x, c, w = _dual()
    same = dict(w, ada_txt_w=w["ada_w"], ada_txt_b=w["ada_b"])
    assert np.array_equal(O.block_forward(x, c, same, **_kw(s)),
                          O.block_forward(x, c, _single(w), **_kw(s)))


def test_p13_no_text_tokens_ignores_the_text_map():
    s, x, c, w = _dual(text_len=0, grid=(2, 3, 2), rope_dims=(4, 4, 2))
    assert np.array_equal(O.block_forward(x, c, w, **_kw(s)),
                          O.block_forward(x, c, _single(w), **_kw(s)))


@pytest.mark.parametrize("stream", ["text", "visual"])
def test_p13_zero_gates_of_one_stream_pass_its_tokens_through(stream):
    s, x, c, w = _dual()
    D, T = s.hidden, s.text_len
    w = dict(w)
    wk, bk = ("ada_txt_w", "ada_txt_b") if stream == "text" else ("ada_w", "ada_b")
    w[wk], w[bk] = w[wk].copy(), w[bk].copy()
    for blk in (2, 5):
        w[wk][blk * D:(blk + 1) * D] = 0.0
        w[bk][blk * D:(blk + 1) * D] = 0.0
    out = O.block_forward(x, c, w, **_kw(s))
    same, moved = (slice(0, T), slice(T, None)) if stream == "text" else (slice(T, None), slice(0, T))
    assert np.array_equal(out[:, same], x[:, same])
    assert np.min(np.max(np.abs(out[:, moved] - x[:, moved]), axis=-1)) > 1e-3


def _sel(L, rows):
    return np.arange(L) if rows is None else np.asarray(rows)


def _mut_rows_swapped(cond, w, text_len, L, rows=None):
    m = O.adaln_modulation(cond, w["ada_w"], w["ada_b"])
    t = O.adaln_modulation(cond, w["ada_txt_w"], w["ada_txt_b"])
    sel = _sel(L, rows)
    out = np.repeat(t[:, None, :], sel.size, axis=1)
    out[:, sel < text_len, :] = m[:, None, :]
    return out


def _mut_rows_boundary(cond, w, text_len, L, rows=None):
    m = O.adaln_modulation(cond, w["ada_w"], w["ada_b"])
    t = O.adaln_modulation(cond, w["ada_txt_w"], w["ada_txt_b"])
    sel = _sel(L, rows)
    out = np.repeat(m[:, None, :], sel.size, axis=1)
    out[:, sel < text_len + 1, :] = t[:, None, :]
    return out


def _mut_rows_text_ignored(cond, w, text_len, L, rows=None):
    m = O.adaln_modulation(cond, w["ada_w"], w["ada_b"])
    return np.repeat(m[:, None, :], _sel(L, rows).size, axis=1)


@pytest.mark.parametrize("fn", [_mut_rows_swapped, _mut_rows_boundary, _mut_rows_text_ignored])
def test_planted_dual_stream_mistakes_are_caught(fn, monkeypatch):
    s, x, c, w = _dual()
    ref = _brute(x, c, w, s)
    monkeypatch.setattr(O, "row_modulation", fn)
    bad = O.block_forward(x, c, w, **_kw(s))
    assert np.max(np.abs(bad - ref)) / np.max(np.abs(ref)) > 1e-9
