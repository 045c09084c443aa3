"""fp64 CPU oracle of one DiT block forward (test infrastructure only).

ONLY tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this module.  The HIP path never calls it, and it shares no code with the HIP
path: it reads fp64 arrays and returns fp64 arrays.

What it computes.  The paper's denoiser is a stack of repeated transformer
blocks (Sec. 2.1) whose activations grow with the latent sequence length, which
scales with H x W x T (Sec. 2.2); DiT attention is the operator the paper
chunks to fit a memory budget (Sec. 5.2, "Localized chunking and fusion"; Sec.
8, memory mitigation primitives).  Chunking the query/MLP rows of a block does
not change the block's result, so the oracle is the plain definition of one
unchunked block.  The paper prints none of the block's arithmetic; every
convention below is one of the readings R1-R11 listed in this package's
docstring.  In short, for each batch element:

  1. m = W_ada c + b_ada, split as (shift1, scale1, gate1, shift2, scale2, gate2)
  2. h  = LN(x) * (1 + scale1) + shift1            (LN without affine, biased var)
  3. [q|k|v] = h W_qkv^T + b_qkv; head j owns columns [j d, (j+1) d) of each
  4. q <- q / sqrt(mean(q^2) + eps_qk) * gamma_q, the same for k with gamma_k
  5. 3D RoPE of q and k for visual tokens (interleaved pairs, theta = 10000)
  6. o = softmax(q k^T / sqrt(d)) v over all L tokens, per head (no mask)
  7. x1 = x + gate1 * (o W_o^T + b_o)
  8. h2 = LN(x1) * (1 + scale2) + shift2
  9. g = GELU_tanh(h2 W_1^T + b_1)
 10. out = x1 + gate2 * (g W_2^T + b_2)

Dual-stream modulation (reading R24): when the weights carry a second AdaLN
map (ada_txt_w, ada_txt_b), the text tokens (positions below L_t) take their
shift, scale and gate from m_txt = W_ada_txt c + b_ada_txt, split the same way,
and the visual tokens from m; every other weight stays shared.

Library primitives used as steps: numpy matmul (for the Linear maps and for
q k^T and P v), numpy exp/tanh/sqrt.  No blocking beyond splitting the query
rows of step 6 into row groups so memory stays bounded (each query row's
softmax is still taken over all L keys at once).
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence, Tuple

import numpy as np

# -- step 1: AdaLN modulation ---------------------------------------------------


def adaln_modulation(cond: np.ndarray, w_ada: np.ndarray, b_ada: np.ndarray) -> np.ndarray:
    """m = W_ada c + b_ada for each batch row: [B, D_c] -> [B, 6D].
    Reading R2: a plain linear map of the conditioning vector (no SiLU)."""
    return cond @ w_ada.T + b_ada


def row_modulation(cond: np.ndarray, w: Dict[str, np.ndarray], text_len: int, L: int,
                   rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """The modulation vector of every token, or of the sequence positions in
    `rows`: [B, L or len(rows), 6D].  One AdaLN map for all tokens (reading
    R1), or with a second map for the text tokens (reading R24): positions
    below text_len take m_txt, the rest m."""
    sel = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    m = adaln_modulation(cond, w["ada_w"], w["ada_b"])
    out = np.repeat(m[:, None, :], sel.size, axis=1)
    if "ada_txt_w" in w:
        m_txt = adaln_modulation(cond, w["ada_txt_w"], w["ada_txt_b"])
        out[:, sel < text_len, :] = m_txt[:, None, :]
    return out


def split_modulation(m: np.ndarray) -> Tuple[np.ndarray, ...]:
    """Split [B, 6D] into (shift1, scale1, gate1, shift2, scale2, gate2), each
    [B, D], in that order (reading R2)."""
    return tuple(np.split(m, 6, axis=-1))


# -- steps 2 and 8: LayerNorm + modulation -------------------------------------


def layer_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis without affine parameters, with the biased
    variance (reading R3)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def modulate(xhat: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """AdaLN modulation xhat * (1 + scale) + shift (reading R2)."""
    return xhat * (1.0 + scale) + shift


# -- step 3 / 7 / 9 / 10: Linear -----------------------------------------------


def linear(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """y = x W^T + b with W in [out, in] layout (reading R9: every Linear has a bias)."""
    return x @ w.T + b


# -- step 4: QK-RMSNorm --------------------------------------------------------


def rms_norm(z: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """z / sqrt(mean(z^2) + eps) * gamma over the last axis (one head vector);
    gamma is shared by all heads (reading R4)."""
    return z / np.sqrt((z * z).mean(axis=-1, keepdims=True) + eps) * gamma


# -- step 5: 3D rotary position embedding ---------------------------------------


def token_coords(text_len: int, grid: Tuple[int, int, int]) -> np.ndarray:
    """(t, y, w) latent-grid coordinates of every token, -1 for text tokens.
    Token order (reading R6): text first, then visual tokens in t-major, then
    row (y), then column (w) order."""
    gt, gh, gw = grid
    n_vis = gt * gh * gw
    coords = -np.ones((text_len + n_vis, 3), dtype=np.int64)
    v = np.arange(n_vis)
    coords[text_len:, 0] = v // (gh * gw)
    coords[text_len:, 1] = (v // gw) % gh
    coords[text_len:, 2] = v % gw
    return coords


def rope_angles(coords: np.ndarray, rope_dims: Sequence[int], head_dim: int,
                theta: float) -> np.ndarray:
    """Rotation angle of every (token, pair) as an [L, head_dim/2] array.

    The head vector is split into contiguous segments [t | y | w] of widths
    (d_t, d_h, d_w) (reading R5).  Inside a segment of width d_a, pair j covers
    elements (2j, 2j+1) and turns by position * theta^(-2j/d_a).  Text tokens and
    the elements past d_t+d_h+d_w keep angle 0 (no rotation)."""
    L = coords.shape[0]
    ang = np.zeros((L, head_dim // 2), dtype=np.float64)
    pair0 = 0
    for axis, da in enumerate(rope_dims):
        if da == 0:
            continue
        j = np.arange(da // 2, dtype=np.float64)
        inv_freq = theta ** (-2.0 * j / da)
        pos = coords[:, axis].astype(np.float64)
        visual = coords[:, axis] >= 0
        seg = np.outer(pos, inv_freq)
        seg[~visual] = 0.0
        ang[:, pair0:pair0 + da // 2] = seg
        pair0 += da // 2
    return ang


def rope_rotate(z: np.ndarray, angles: np.ndarray) -> np.ndarray:
    """Rotate interleaved pairs: (u0, u1) -> (u0 cos - u1 sin, u0 sin + u1 cos).
    z is [L, H, d]; angles is [L, d/2] and is the same for every head."""
    c = np.cos(angles)[:, None, :]
    s = np.sin(angles)[:, None, :]
    u0 = z[..., 0::2]
    u1 = z[..., 1::2]
    out = np.empty_like(z)
    out[..., 0::2] = u0 * c - u1 * s
    out[..., 1::2] = u0 * s + u1 * c
    return out


# -- step 6: attention ------------------------------------------------------------


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax with the row maximum subtracted first (two passes)."""
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, row_group: int = 1024) -> np.ndarray:
    """Full bidirectional attention for one head (reading R7): q [Lq, d],
    k and v [L, d] -> [Lq, d].  Queries are processed in row groups only to
    bound memory; every row's softmax spans all L keys."""
    d = q.shape[-1]
    out = np.empty((q.shape[0], v.shape[-1]), dtype=np.float64)
    scale = 1.0 / np.sqrt(d)
    for r0 in range(0, q.shape[0], row_group):
        s = (q[r0:r0 + row_group] @ k.T) * scale
        out[r0:r0 + row_group] = softmax_rows(s) @ v
    return out


# -- step 9: GELU ------------------------------------------------------------------


def gelu_tanh(u: np.ndarray) -> np.ndarray:
    """GELU, tanh form: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3))) (reading R8)."""
    return 0.5 * u * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (u + 0.044715 * u ** 3)))


# -- the whole block ----------------------------------------------------------------


def qkv_heads(h: np.ndarray, w: Dict[str, np.ndarray], heads: int, head_dim: int,
              coords: np.ndarray, rope_dims, theta: float, qk_eps: float):
    """Steps 3-5 for one sequence: h [L, D] -> q, k, v each [L, H, d]."""
    L = h.shape[0]
    D = heads * head_dim
    qkv = linear(h, w["qkv_w"], w["qkv_b"])
    q = qkv[:, 0:D].reshape(L, heads, head_dim)
    k = qkv[:, D:2 * D].reshape(L, heads, head_dim)
    v = qkv[:, 2 * D:3 * D].reshape(L, heads, head_dim)
    q = rms_norm(q, w["q_gamma"], qk_eps)
    k = rms_norm(k, w["k_gamma"], qk_eps)
    ang = rope_angles(coords, rope_dims, head_dim, theta)
    return rope_rotate(q, ang), rope_rotate(k, ang), v


def block_prepare(x: np.ndarray, cond: np.ndarray, w: Dict[str, np.ndarray], *,
                  heads: int, head_dim: int, text_len: int, grid: Tuple[int, int, int],
                  rope_dims: Sequence[int], rope_theta: float = 10000.0,
                  ln_eps: float = 1e-6, qk_eps: float = 1e-6,
                  coords: Optional[np.ndarray] = None) -> dict:
    """Steps 1-5 for every token of every sequence: the normalised and rotated
    q, k and the v of each batch element, which every output row needs (a
    query attends to all L keys).  Returns a dict that block_rows consumes."""
    B, L, D = x.shape
    if coords is None:
        coords = token_coords(text_len, grid)
    assert coords.shape[0] == L and heads * head_dim == D
    qkv = []
    for b in range(B):
        # the modulation vectors of 8192 rows at a time (LayerNorm is per row,
        # so the row blocks only bound memory)
        h = np.empty((L, D), dtype=np.float64)
        for r0 in range(0, L, 8192):
            sel = np.arange(r0, min(L, r0 + 8192))
            m = row_modulation(cond[b:b + 1], w, text_len, L, rows=sel)[0]
            h[sel] = modulate(layer_norm(x[b, sel], ln_eps), m[:, 0:D], m[:, D:2 * D])
        qkv.append(qkv_heads(h, w, heads, head_dim, coords, rope_dims, rope_theta, qk_eps))
    return {"x": x, "cond": cond, "w": w, "qkv": qkv, "heads": heads, "head_dim": head_dim,
            "text_len": text_len, "ln_eps": ln_eps}


def block_rows(prep: dict, rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Steps 6-10 for the sequence positions in `rows` (all when None) of
    every batch element: [B, len(rows), D]."""
    x, w, heads, head_dim = prep["x"], prep["w"], prep["heads"], prep["head_dim"]
    B, L, D = x.shape
    sel = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    _, _, gate1, shift2, scale2, gate2 = split_modulation(
        row_modulation(prep["cond"], w, prep["text_len"], L, rows=sel))  # each [B, R, D]
    out = np.empty((B, sel.size, D), dtype=np.float64)
    for b in range(B):
        q, k, v = prep["qkv"][b]
        o = np.empty((sel.size, heads, head_dim), dtype=np.float64)
        for j in range(heads):
            o[:, j, :] = attention(q[sel, j, :], k[:, j, :], v[:, j, :])
        x1 = x[b][sel] + gate1[b] * linear(o.reshape(sel.size, D), w["o_w"], w["o_b"])
        h2 = modulate(layer_norm(x1, prep["ln_eps"]), shift2[b], scale2[b])
        g = gelu_tanh(linear(h2, w["up_w"], w["up_b"]))
        out[b] = x1 + gate2[b] * linear(g, w["down_w"], w["down_b"])
    return out


def block_forward(x: np.ndarray, cond: np.ndarray, w: Dict[str, np.ndarray], *,
                  heads: int, head_dim: int, text_len: int, grid: Tuple[int, int, int],
                  rope_dims: Sequence[int], rope_theta: float = 10000.0,
                  ln_eps: float = 1e-6, qk_eps: float = 1e-6,
                  rows: Optional[Sequence[int]] = None,
                  coords: Optional[np.ndarray] = None) -> np.ndarray:
    """One DiT block forward in fp64.

    x [B, L, D], cond [B, D_c], w: the twelve weights (fp64), plus ada_txt_w
    and ada_txt_b for dual-stream modulation (reading R24).  Returns
    [B, L, D], or [B, len(rows), D] when `rows` selects output rows (keys and
    values are still formed from every token).  `coords` overrides the token
    grid coordinates (used only by tests that move the grid)."""
    prep = block_prepare(x, cond, w, heads=heads, head_dim=head_dim, text_len=text_len, grid=grid,
                         rope_dims=rope_dims, rope_theta=rope_theta, ln_eps=ln_eps, qk_eps=qk_eps,
                         coords=coords)
    return block_rows(prep, rows)


def prepare_shape(inputs) -> dict:
    """block_prepare on a workloads.Inputs bundle (bf16 values upcast exactly)."""
    s = inputs.shape
    return block_prepare(inputs.f64("x"), inputs.f64("cond"), inputs.weights_f64(),
                         heads=s.heads, head_dim=s.head_dim, text_len=s.text_len,
                         grid=s.grid, rope_dims=s.rope_dims, rope_theta=s.rope_theta,
                         ln_eps=s.ln_eps, qk_eps=s.qk_eps)


def block_forward_shape(inputs, rows=None) -> np.ndarray:
    """block_forward on a workloads.Inputs bundle (bf16 values upcast exactly)."""
    return block_rows(prepare_shape(inputs), rows)
