"""The VAE decoder's fused upsampling stage on the GPU (xema_vae_upconv, C
ABI) against the fp64 oracle (nearest 2x, then 3x3 convolution): the summed
weights byte for byte, parity on small stages spanning several tiles with
ragged tails, bit-identical output for every row banding, and the full-size
stages on sampled output pixels."""
import numpy as np
import pytest
import torch

import paper_2607_11136_amd as X
import workloads as W
from oracle import vae as V

from gpu_util import DEV, bf16_dev, errors

pytestmark = pytest.mark.gpu


def assert_vae_parity(got: np.ndarray, ref: np.ndarray, what: str):
    """The bar, from the arithmetic (reading R26).  One bf16 rounding
    separates the GPU from the exact definition: the output's own, whose mean
    cost is the 'bf16 floor' MAE(bf16_RNE(ref), ref).  The phase-summed
    weights enter as hi + lo bf16 pairs (about 2^-17 of each weight) and the
    products accumulate in fp32, so MAE <= floor + 4e-4, and |g - o| <= 2e-2
    max(|o|, 1) elementwise."""
    e = errors(got, ref)
    floor = float(np.mean(np.abs(W.bf16_bits_to_f64(W.to_bf16_bits(ref.astype(np.float32))) - ref)))
    print(f"{what}: {e} bf16 floor {floor:.3g}", flush=True)
    assert np.all(np.isfinite(got)), what
    assert e["max_rel"] <= 2e-2 and e["mae"] <= floor + 4e-4, (what, e, floor)

SMALL = {
    "tiny": W.VAE_TINY,
    "wide": W.VaeShape("vae_wide", 23, 1, 9, 33, 128, 512),
    "tall": W.VaeShape("vae_tall", 24, 3, 17, 6, 192, 256),
}


class Stage:
    def __init__(self, s: W.VaeShape):
        self.s = s
        self.inp = W.make_vae_inputs(s)
        self.x, self.w, self.b = bf16_dev(self.inp.x), bf16_dev(self.inp.weight), bf16_dev(self.inp.bias)
        self.wp = torch.empty(X.xema_vae_upconv_weight_bytes(s.ci, s.co) // 2, dtype=torch.bfloat16, device=DEV)
        X.xema_vae_upconv_prepare(self.w, s.ci, s.co, self.wp)

    def run(self, bands=None):
        s = self.s
        y = torch.full((s.n, 2 * s.h, 2 * s.w, s.co), float("nan"), dtype=torch.bfloat16, device=DEV)
        for r0, rc in (bands or [(0, s.h)]):
            X.xema_vae_upconv(self.x, s.n, s.h, s.w, s.ci, self.wp, self.b, s.co, r0, rc, y)
        torch.cuda.synchronize()
        return y


def _bf16_rne(a32: np.ndarray) -> np.ndarray:
    return W.bf16_bits_to_f64(W.to_bf16_bits(a32.astype(np.float32)))


def test_summed_weights_byte_exact():
    s = SMALL["wide"]
    st = Stage(s)
    w = W.bf16_bits_to_f64(st.inp.weight).astype(np.float32)      # [co, 3, 3, ci]
    rows = {0: [[0], [1, 2]], 1: [[0, 1], [2]]}
    want = np.empty((4, s.co, 8, s.ci), dtype=np.float64)
    for p in range(4):
        py, px = p >> 1, p & 1
        for t in range(4):
            a, b = t >> 1, t & 1
            acc = np.zeros((s.co, s.ci), dtype=np.float32)
            for ky in rows[py][a]:
                for kx in rows[px][b]:
                    acc = acc + w[:, ky, kx, :]
            hi = _bf16_rne(acc)
            want[p, :, t, :] = hi
            want[p, :, 4 + t, :] = _bf16_rne(acc - hi.astype(np.float32))   # the remainder is exact in fp32
    got = st.wp.float().cpu().numpy().astype(np.float64).reshape(4, s.co, 8, s.ci)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_upconv_matches_oracle(name):
    s = SMALL[name]
    st = Stage(s)
    print(f"vae {name}: n={s.n} {s.h}x{s.w} ci={s.ci} co={s.co}", flush=True)
    y = st.run().float().cpu().numpy()
    ref = V.upsample_conv(st.inp.f64("x"), st.inp.f64("weight"), st.inp.f64("bias"))
    assert_vae_parity(y, ref, f"vae {name}")


@pytest.mark.parametrize("name", sorted(SMALL))
def test_row_bands_are_bit_identical(name):
    s = SMALL[name]
    st = Stage(s)
    base = st.run()
    h = s.h
    for bands in ([(r, 1) for r in range(h)], [(0, h // 2), (h // 2, h - h // 2)],
                  [(0, 1), (1, max(h - 2, 1))] + ([(h - 1, 1)] if h > 2 else [])):
        if sum(rc for _, rc in bands) != h:
            continue
        assert torch.equal(st.run(bands), base), bands
    # a band writes only its own output rows
    y = torch.zeros_like(base)
    X.xema_vae_upconv(st.x, s.n, s.h, s.w, s.ci, st.wp, st.b, s.co, 1, 1, y)
    torch.cuda.synchronize()
    assert torch.equal(y[:, 2:4], base[:, 2:4])
    assert not torch.any(y[:, :2] != 0) and not torch.any(y[:, 4:] != 0)


def _sampled_reference(inp: W.VaeInputs, picks):
    """The definition at single output pixels: 9 taps of the upsampled image."""
    x, w, b = inp.f64("x"), inp.f64("weight"), inp.f64("bias")
    n, h, wd, _ = x.shape
    out = []
    for f, u, v in picks:
        acc = b.copy()
        for dy in (-1, 0, 1):
            for dx in (-1, 0, 1):
                uu, vv = u + dy, v + dx
                if 0 <= uu < 2 * h and 0 <= vv < 2 * wd:
                    acc = acc + w[:, dy + 1, dx + 1, :] @ x[f, uu // 2, vv // 2, :]
        out.append(acc)
    return np.array(out)


@pytest.mark.parametrize("name", ["vae_video", "vae_1080p"])
def test_full_size_stage_on_sampled_pixels(name):
    s = W.VAE_CONFIGS[name]
    st = Stage(s)
    print(f"vae {name}: n={s.n} {s.h}x{s.w} ci={s.ci} co={s.co}", flush=True)
    y = st.run()
    g = np.random.default_rng(np.random.SeedSequence([2607, 77, s.cfg_id]))
    picks = {(int(g.integers(s.n)), int(g.integers(2 * s.h)), int(g.integers(2 * s.w))) for _ in range(400)}
    for f in (0, s.n - 1):
        for u in (0, 1, 2 * s.h - 2, 2 * s.h - 1):
            for v in (0, 1, 2 * s.w - 2, 2 * s.w - 1):
                picks.add((f, u, v))
    picks = sorted(picks)
    idx = torch.tensor(picks, device=DEV)
    got = y[idx[:, 0], idx[:, 1], idx[:, 2]].float().cpu().numpy()
    assert_vae_parity(got, _sampled_reference(st.inp, picks), f"vae {name} sampled")
    assert not torch.isnan(y).any()
