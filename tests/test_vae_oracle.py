"""Pins of the VAE upsampling-stage oracle (reading R25) against what the
definition and mathematics fix: torch fp64 CPU ops (nearest interpolation and
conv2d), the scalar brute force, closed forms for a delta and a constant
input, the phase form of the fused computation, and planted mistakes."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import vae as V


def _inputs(shape):
    inp = W.make_vae_inputs(shape)
    return inp.f64("x"), inp.f64("weight"), inp.f64("bias")


def _torch_ref(x, w, b):
    xt = torch.from_numpy(x).permute(0, 3, 1, 2)                    # NCHW
    up = torch.nn.functional.interpolate(xt, scale_factor=2, mode="nearest")
    wt = torch.from_numpy(w).permute(0, 3, 1, 2)                    # [co, ci, 3, 3]
    y = torch.nn.functional.conv2d(up, wt, torch.from_numpy(b), padding=1)
    return y.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("shape", [W.VAE_TINY, W.VAE_TINY.with_(n=1, h=1, w=1, ci=8, co=4),
                                   W.VAE_TINY.with_(n=3, h=4, w=2, ci=16, co=8)])
def test_matches_torch_interpolate_and_conv2d(shape):
    x, w, b = _inputs(shape)
    got = V.upsample_conv(x, w, b)
    ref = _torch_ref(x, w, b)
    assert got.shape == (shape.n, 2 * shape.h, 2 * shape.w, shape.co)
    assert np.max(np.abs(got - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def _brute(x, w, b):
    n, h, wd, ci = x.shape
    co = w.shape[0]
    out = np.zeros((n, 2 * h, 2 * wd, co))
    for f in range(n):
        for u in range(2 * h):
            for v in range(2 * wd):
                for o in range(co):
                    acc = b[o]
                    for dy in (-1, 0, 1):
                        for dx in (-1, 0, 1):
                            uu, vv = u + dy, v + dx
                            if 0 <= uu < 2 * h and 0 <= vv < 2 * wd:
                                acc += sum(w[o, dy + 1, dx + 1, c] * x[f, uu // 2, vv // 2, c] for c in range(ci))
                    out[f, u, v, o] = acc
    return out


def test_matches_scalar_brute_force():
    s = W.VAE_TINY.with_(n=2, h=3, w=2, ci=5, co=3)
    x, w, b = _inputs(s)
    assert np.max(np.abs(V.upsample_conv(x, w, b) - _brute(x, w, b))) <= 1e-12


def test_delta_input_closed_form():
    s = W.VAE_TINY.with_(n=1, h=4, w=5, ci=6, co=3)
    _, w, b = _inputs(s)
    i, j, c = 2, 1, 4
    x = np.zeros((1, s.h, s.w, s.ci))
    x[0, i, j, c] = 1.0
    y = V.upsample_conv(x, w, b)
    for u in range(2 * s.h):
        for v in range(2 * s.w):
            want = b.copy()
            for dy in (-1, 0, 1):
                for dx in (-1, 0, 1):
                    if (u + dy) // 2 == i and (v + dx) // 2 == j and 0 <= u + dy and 0 <= v + dx:
                        want = want + w[:, dy + 1, dx + 1, c]
            assert np.array_equal(y[0, u, v], want), (u, v)


def test_constant_input_interior_and_corner():
    s = W.VAE_TINY.with_(n=1, h=3, w=3, ci=4, co=2)
    _, w, b = _inputs(s)
    x = np.full((1, s.h, s.w, s.ci), 0.75)
    y = V.upsample_conv(x, w, b)
    full = b + 0.75 * w.sum(axis=(1, 2, 3))
    corner = b + 0.75 * w[:, 1:, 1:, :].sum(axis=(1, 2, 3))   # top-left: taps dy, dx >= 0
    np.testing.assert_allclose(y[0, 2, 3], full, rtol=0, atol=1e-14)
    np.testing.assert_allclose(y[0, 0, 0], corner, rtol=0, atol=1e-14)


def test_phase_form_equals_the_definition():
    """The fused method: output pixel (2i+py, 2j+px) is a 2x2 convolution of
    x (zero-padded) with weights summed over the 3x3 taps that land on the
    same source pixel.  Written here independently of the oracle."""
    s = W.VAE_TINY.with_(n=2, h=4, w=5, ci=6, co=3)
    x, w, b = _inputs(s)
    taps = {0: [[0], [1, 2]], 1: [[0, 1], [2]]}   # phase -> source offset a -> kernel rows
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    y = np.zeros((s.n, 2 * s.h, 2 * s.w, s.co))
    for py in (0, 1):
        for px in (0, 1):
            acc = np.broadcast_to(b, (s.n, s.h, s.w, s.co)).copy()
            for a in (0, 1):
                for c in (0, 1):
                    wc = sum(w[:, ky, kx, :] for ky in taps[py][a] for kx in taps[px][c])
                    r0, c0 = py + a, px + c            # padded source row/col of pixel (0, 0)
                    acc += xp[:, r0:r0 + s.h, c0:c0 + s.w, :] @ wc.T
            y[:, py::2, px::2, :] = acc
    ref = V.upsample_conv(x, w, b)
    assert np.max(np.abs(y - ref)) <= 1e-12


_conv = V.conv3x3_same


def _mut_up_shift(x):
    u = np.repeat(np.repeat(x, 2, axis=1), 2, axis=2)
    return np.roll(u, 1, axis=1)


def _mut_conv_flipped(u, w, b):
    return _conv(u, w[:, ::-1, ::-1, :], b)


def _mut_conv_no_bias(u, w, b):
    return _conv(u, w, np.zeros_like(b))


def _mut_conv_transposed_taps(u, w, b):
    return _conv(u, w.transpose(0, 2, 1, 3), b)


@pytest.mark.parametrize("attr,fn", [("upsample_nearest2x", _mut_up_shift),
                                     ("conv3x3_same", _mut_conv_flipped),
                                     ("conv3x3_same", _mut_conv_no_bias),
                                     ("conv3x3_same", _mut_conv_transposed_taps)])
def test_planted_mistakes_are_caught(attr, fn, monkeypatch):
    s = W.VAE_TINY.with_(n=1, h=3, w=4, ci=8, co=4)
    x, w, b = _inputs(s)
    ref = _torch_ref(x, w, b)
    monkeypatch.setattr(V, attr, fn)
    bad = V.upsample_conv(x, w, b)
    assert np.max(np.abs(bad - ref)) > 1e-6
