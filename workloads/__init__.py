"""Seeded synthetic workloads for the DiT block forward.

This module is shared by the fp64 oracle tests and by the HIP path's tests and
benchmark. It holds shapes and seeded random draws only: none of the block's
arithmetic lives here.

Shapes follow the request templates the paper serves (Sec. 2.1 defines a
template as model, output height, width and frame count; Sec. 9 lists the
Flux.2 / CogVideoX-5B / LTX-2 templates).  The widths (hidden size, heads, MLP
width) are those of DiT denoisers of that family.  No trained weights or real
activations exist here, so every tensor is a seeded draw:

* tokens x and conditioning vector c ~ N(0, 1)
* every Linear weight and bias ~ N(0, 1/fan_in)
* the QK-RMSNorm gains gamma = 1 + 0.1 * N(0, 1)

Each tensor is drawn in fp32 from PCG64 seeded by SeedSequence([2607, cfg_id,
tensor_id]) and then rounded to bfloat16 with round-to-nearest-even.  Both the
oracle (after an exact upcast to fp64) and the GPU consume the same bf16 values.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED_ROOT = 2607

# Order of the twelve weight tensors; the C ABI's weight struct uses this order.
WEIGHT_NAMES: Tuple[str, ...] = (
    "ada_w", "ada_b", "qkv_w", "qkv_b", "q_gamma", "k_gamma",
    "o_w", "o_b", "up_w", "up_b", "down_w", "down_b",
)
# The text tokens' own AdaLN map of a dual-stream block (tensor ids 14, 15).
TEXT_MOD_NAMES: Tuple[str, ...] = ("ada_txt_w", "ada_txt_b")


@dataclasses.dataclass(frozen=True)
class BlockShape:
    """Hyper-parameters of one DiT block plus one request (batch and grid)."""
    name: str
    cfg_id: int
    batch: int
    text_len: int
    grid: Tuple[int, int, int]          # (G_t, G_h, G_w) latent patch grid
    hidden: int                         # D
    heads: int                          # H
    head_dim: int                       # d
    mlp_hidden: int                     # F
    cond_dim: int                       # D_c
    rope_dims: Tuple[int, int, int]     # (d_t, d_h, d_w), even, sum <= d
    rope_theta: float = 10000.0
    ln_eps: float = 1e-6
    qk_eps: float = 1e-6
    chunks: Tuple[int, ...] = (0,)      # chunk_tokens values exercised; 0 = all
    modulation_streams: int = 1         # 2: text tokens have their own AdaLN map
    weights_f16: int = 0                # 1: W_o, W_up, W_down handed over in fp16

    @property
    def n_visual(self) -> int:
        t, h, w = self.grid
        return t * h * w

    @property
    def seq_len(self) -> int:
        return self.text_len + self.n_visual

    def with_(self, **kw) -> "BlockShape":
        return dataclasses.replace(self, **kw)

    def weight_shapes(self) -> Dict[str, Tuple[int, ...]]:
        D, F, Dc, d = self.hidden, self.mlp_hidden, self.cond_dim, self.head_dim
        return {
            "ada_w": (6 * D, Dc), "ada_b": (6 * D,),
            "qkv_w": (3 * D, D), "qkv_b": (3 * D,),
            "q_gamma": (d,), "k_gamma": (d,),
            "o_w": (D, D), "o_b": (D,),
            "up_w": (F, D), "up_b": (F,),
            "down_w": (D, F), "down_b": (D,),
            **({"ada_txt_w": (6 * D, Dc), "ada_txt_b": (6 * D,)} if self.modulation_streams == 2 else {}),
        }

    def fan_in(self, name: str) -> Optional[int]:
        D, F, Dc = self.hidden, self.mlp_hidden, self.cond_dim
        return {"ada_w": Dc, "ada_b": Dc, "ada_txt_w": Dc, "ada_txt_b": Dc, "qkv_w": D, "qkv_b": D,
                "o_w": D, "o_b": D, "up_w": D, "up_b": D,
                "down_w": F, "down_b": F}.get(name)

    def flops(self) -> int:
        """Algorithmic FLOPs of one block step: the five contractions plus the
        AdaLN map(s) (elementwise work is not counted)."""
        B, L, D, F, Dc = self.batch, self.seq_len, self.hidden, self.mlp_hidden, self.cond_dim
        return (2 * B * Dc * 6 * D * self.modulation_streams + 6 * B * L * D * D + 2 * B * L * D * D
                + 4 * B * L * D * F + 4 * B * L * L * D)


# The five workloads.  cfg_id fixes the seeds.
TINY = BlockShape("tiny", 0, 1, 32, (1, 16, 16), 256, 4, 64, 1024, 256, (16, 24, 24),
                  chunks=(0, 64))
IMAGE = BlockShape("image", 1, 1, 512, (1, 64, 64), 3072, 24, 128, 12288, 3072, (0, 64, 64))
IMAGE_B4 = IMAGE.with_(name="image_b4", batch=4)
VIDEO = BlockShape("video", 2, 1, 226, (13, 30, 45), 3072, 48, 64, 12288, 3072, (16, 24, 24))
HIGHRES = BlockShape("highres", 3, 1, 226, (13, 68, 120), 3072, 48, 64, 12288, 3072, (16, 24, 24))
LONG = BlockShape("long", 4, 2, 1024, (33, 22, 38), 4096, 32, 128, 16384, 4096, (32, 48, 48),
                  chunks=(0, 8192, 2048))
# The video block with dual-stream modulation: the same tensors as VIDEO plus
# the text tokens' AdaLN map.
VIDEO_DUAL = VIDEO.with_(name="video_dual", modulation_streams=2)

CONFIGS: Dict[str, BlockShape] = {c.name: c for c in (TINY, IMAGE, IMAGE_B4, VIDEO, HIGHRES, LONG,
                                                      VIDEO_DUAL)}


def _rng(cfg_id: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, cfg_id, tensor_id])))


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> exact fp64 values."""
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _draw(shape, cfg_id: int, tensor_id: int, std: float, mean: float = 0.0) -> np.ndarray:
    g = _rng(cfg_id, tensor_id)
    a = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if mean != 0.0:
        a += np.float32(mean)
    return to_bf16_bits(a)


@dataclasses.dataclass
class Inputs:
    """bf16 bit patterns (uint16) of every input of one block call."""
    shape: BlockShape
    x: np.ndarray                       # [B, L, D]
    cond: np.ndarray                    # [B, D_c]
    weights: Dict[str, np.ndarray]      # WEIGHT_NAMES (+ TEXT_MOD_NAMES) -> array

    def f64(self, name: str) -> np.ndarray:
        if name == "x":
            return bf16_bits_to_f64(self.x)
        if name == "cond":
            return bf16_bits_to_f64(self.cond)
        return bf16_bits_to_f64(self.weights[name])

    def weights_f64(self) -> Dict[str, np.ndarray]:
        return {k: bf16_bits_to_f64(v) for k, v in self.weights.items()}


def make_inputs(shape: BlockShape, seed_id: Optional[int] = None) -> Inputs:
    """Seeded inputs for `shape`.  `seed_id` overrides cfg_id (ad-hoc shapes)."""
    cid = shape.cfg_id if seed_id is None else seed_id
    B, L, D, Dc = shape.batch, shape.seq_len, shape.hidden, shape.cond_dim
    x = _draw((B, L, D), cid, 0, 1.0)
    cond = _draw((B, Dc), cid, 1, 1.0)
    w = {}
    for i, (name, shp) in enumerate(shape.weight_shapes().items()):
        if name in ("q_gamma", "k_gamma"):
            w[name] = _draw(shp, cid, 2 + i, 0.1, mean=1.0)
        else:
            w[name] = _draw(shp, cid, 2 + i, float(1.0 / np.sqrt(shape.fan_in(name))))
    return Inputs(shape, x, cond, w)


def tiny_shape(**kw) -> BlockShape:
    """A very small block for brute-force checks (defaults: L_t=3, grid 2x2x3,
    D=24, 2 heads x 12, F=48, RoPE (4,4,4))."""
    base = BlockShape("brute", 90, 1, 3, (2, 2, 3), 24, 2, 12, 48, 24, (4, 4, 4))
    return base.with_(**kw)


def sample_rows(shape: BlockShape, n: int, seed: int = 7) -> List[int]:
    """A seeded sample of token rows of one sequence that always contains the
    first and last rows and the text/visual boundary."""
    L = shape.seq_len
    g = np.random.default_rng(np.random.SeedSequence([SEED_ROOT, 99, seed]))
    pick = set(int(i) for i in g.choice(L, size=min(n, L), replace=False))
    pick.update({0, L - 1, max(shape.text_len - 1, 0), min(shape.text_len, L - 1)})
    return sorted(pick)


def step_weights(shape: BlockShape, n_blocks: int) -> List[Dict[str, np.ndarray]]:
    """Distinct seeded weights (bf16 bit patterns) for the blocks of an
    n-block step: block 0 has the shape's own weights, block i > 0 those of
    seed id 1000 + 64 * cfg_id + i."""
    out = [make_inputs(shape).weights]
    for i in range(1, n_blocks):
        out.append(make_inputs(shape, seed_id=1000 + 64 * shape.cfg_id + i).weights)
    return out


# -- the VAE decoder's upsampling stage -------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class VaeShape:
    """A VAE decoder upsampling stage: nearest 2x then a 3x3 convolution,
    NHWC activations of n frames (the decoder runs frame by frame here)."""
    name: str
    cfg_id: int
    n: int            # frames
    h: int            # input rows
    w: int            # input columns
    ci: int           # input channels
    co: int           # output channels

    def with_(self, **kw) -> "VaeShape":
        return dataclasses.replace(self, **kw)

    def flops(self) -> int:
        """Algorithmic FLOPs of the definition: a 3x3 convolution over the
        2H x 2W upsampled image."""
        return 2 * self.n * (2 * self.h) * (2 * self.w) * 9 * self.ci * self.co


@dataclasses.dataclass
class VaeInputs:
    """bf16 bit patterns: x [n, h, w, ci], weight [co, 3, 3, ci], bias [co]."""
    shape: VaeShape
    x: np.ndarray
    weight: np.ndarray
    bias: np.ndarray

    def f64(self, name: str) -> np.ndarray:
        return bf16_bits_to_f64(getattr(self, name))


def make_vae_inputs(shape: VaeShape) -> VaeInputs:
    """x ~ N(0, 1); weight and bias ~ N(0, 1 / (9 ci)), the convolution's fan-in."""
    s = shape
    std = float(1.0 / np.sqrt(9 * s.ci))
    return VaeInputs(s, _draw((s.n, s.h, s.w, s.ci), s.cfg_id, 0, 1.0),
                     _draw((s.co, 3, 3, s.ci), s.cfg_id, 1, std), _draw((s.co,), s.cfg_id, 2, std))


# The last upsampler of a 480x720 video decoder (256 channels, 240x360 ->
# 480x720), over 8 frames, and of a 1080p decoder (540x960 -> 1080x1920) over
# 2 frames; a small stage for parity tests.
VAE_TINY = VaeShape("vae_tiny", 20, 2, 5, 7, 64, 256)
VAE_VIDEO = VaeShape("vae_video", 21, 8, 240, 360, 256, 256)
VAE_1080P = VaeShape("vae_1080p", 22, 2, 540, 960, 256, 256)
VAE_CONFIGS: Dict[str, VaeShape] = {c.name: c for c in (VAE_TINY, VAE_VIDEO, VAE_1080P)}
