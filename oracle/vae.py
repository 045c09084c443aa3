"""fp64 CPU oracle of a VAE decoder upsampling stage (test infrastructure only).

ONLY tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this module.  It shares no code with the HIP path.

What it computes.  The VAE decoder runs once per request near the output
resolution and is built from convolution, normalization, residual and
upsampling modules (Sec. 2.1); its upsampling creates large short-lived
activation peaks, so the paper chunks or fuses the operators around it
(Sec. 5.2, "Localized chunking and fusion"; Sec. 8, memory mitigation
primitives).  The paper prints no arithmetic for the stage; reading R25 takes
the upsampler of latent-diffusion VAE decoders: nearest-neighbour 2x
upsampling followed by a 3x3 convolution with zero padding 1 and a bias,

    U[n, u, v, c]  = x[n, u // 2, v // 2, c]                 (0 <= u < 2H, 0 <= v < 2W)
    y[n, u, v, o]  = b[o] + sum_{dy, dx in {-1, 0, 1}} sum_c w[o, dy+1, dx+1, c] * U[n, u+dy, v+dx, c]

with U taken as zero outside the image.  Layout NHWC (channels last); the
weight is [C_out, 3, 3, C_in].  The oracle materialises U and runs the
convolution as nine shifted matrix products: the plain definition.
"""
from __future__ import annotations

import numpy as np


def upsample_nearest2x(x: np.ndarray) -> np.ndarray:
    """[N, H, W, C] -> [N, 2H, 2W, C]: every pixel repeated into a 2x2 block."""
    return np.repeat(np.repeat(x, 2, axis=1), 2, axis=2)


def conv3x3_same(u: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """3x3 convolution with zero padding 1 and bias: u [N, H, W, C_in],
    w [C_out, 3, 3, C_in], b [C_out] -> [N, H, W, C_out]."""
    n, h, wd, _ = u.shape
    pad = np.pad(u, ((0, 0), (1, 1), (1, 1), (0, 0)))
    out = np.broadcast_to(b, (n, h, wd, w.shape[0])).astype(np.float64).copy()
    for ky in range(3):
        for kx in range(3):
            out += pad[:, ky:ky + h, kx:kx + wd, :] @ w[:, ky, kx, :].T
    return out


def upsample_conv(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """The upsampling stage: conv3x3_same(upsample_nearest2x(x))."""
    return conv3x3_same(upsample_nearest2x(x), w, b)
