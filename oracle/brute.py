"""Scalar pure-Python DiT block forward for tiny shapes (test infrastructure).

The same definition as oracle.block, written again with explicit scalar loops
and the math module only (no numpy arithmetic), so that a mistake in one of the
two does not hide in a shared helper.  Runs in seconds only for tiny shapes
(a few dozen tokens, hidden size of a few dozen).
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

Vec = List[float]


def _matvec(w, b, x) -> Vec:
    """w is a list of rows [out][in]."""
    return [sum(w[o][i] * x[i] for i in range(len(x))) + b[o] for o in range(len(w))]


def _ln(x: Vec, eps: float) -> Vec:
    n = len(x)
    mu = sum(x) / n
    var = sum((xi - mu) * (xi - mu) for xi in x) / n
    r = 1.0 / math.sqrt(var + eps)
    return [(xi - mu) * r for xi in x]


def _gelu(u: float) -> float:
    return 0.5 * u * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u * u * u)))


def _coords(i: int, text_len: int, grid) -> Tuple[int, int, int]:
    if i < text_len:
        return (-1, -1, -1)
    v = i - text_len
    gt, gh, gw = grid
    t = v // (gh * gw)
    rem = v - t * gh * gw
    return (t, rem // gw, rem % gw)


def _rope(z: Vec, pos: Tuple[int, int, int], dims, theta: float) -> Vec:
    out = list(z)
    off = 0
    for axis in range(3):
        da = dims[axis]
        p = pos[axis]
        for j in range(da // 2):
            if p >= 0:
                phi = p * theta ** (-2.0 * j / da)
                c, s = math.cos(phi), math.sin(phi)
                u0, u1 = z[off + 2 * j], z[off + 2 * j + 1]
                out[off + 2 * j] = u0 * c - u1 * s
                out[off + 2 * j + 1] = u0 * s + u1 * c
        off += da
    return out


def block_forward(x, cond, w: Dict, *, heads: int, head_dim: int, text_len: int, grid,
                  rope_dims: Sequence[int], rope_theta: float = 10000.0,
                  ln_eps: float = 1e-6, qk_eps: float = 1e-6):
    """x: nested lists [B][L][D]; cond [B][Dc]; w: nested lists.  Returns [B][L][D]."""
    B = len(x)
    L = len(x[0])
    D = heads * head_dim
    out = []
    for b in range(B):
        m_vis = _matvec(w["ada_w"], w["ada_b"], cond[b])
        # reading R24: a second AdaLN map, when given, modulates the text tokens
        m_txt = _matvec(w["ada_txt_w"], w["ada_txt_b"], cond[b]) if "ada_txt_w" in w else m_vis

        def mod(i, part):
            m = m_txt if i < text_len else m_vis
            return m[part * D:(part + 1) * D]

        qs, ks, vs = [], [], []
        for i in range(L):
            sh1, sc1 = mod(i, 0), mod(i, 1)
            xh = _ln(x[b][i], ln_eps)
            h = [xh[c] * (1.0 + sc1[c]) + sh1[c] for c in range(D)]
            qkv = _matvec(w["qkv_w"], w["qkv_b"], h)
            pos = _coords(i, text_len, grid)
            qi, ki, vi = [], [], []
            for j in range(heads):
                a = j * head_dim
                qh = qkv[a:a + head_dim]
                kh = qkv[D + a:D + a + head_dim]
                vh = qkv[2 * D + a:2 * D + a + head_dim]
                rq = 1.0 / math.sqrt(sum(t * t for t in qh) / head_dim + qk_eps)
                rk = 1.0 / math.sqrt(sum(t * t for t in kh) / head_dim + qk_eps)
                qh = [qh[e] * rq * w["q_gamma"][e] for e in range(head_dim)]
                kh = [kh[e] * rk * w["k_gamma"][e] for e in range(head_dim)]
                qi.append(_rope(qh, pos, rope_dims, rope_theta))
                ki.append(_rope(kh, pos, rope_dims, rope_theta))
                vi.append(vh)
            qs.append(qi)
            ks.append(ki)
            vs.append(vi)
        rows = []
        for i in range(L):
            o = []
            for j in range(heads):
                s = [sum(qs[i][j][e] * ks[t][j][e] for e in range(head_dim)) / math.sqrt(head_dim)
                     for t in range(L)]
                mx = max(s)
                p = [math.exp(si - mx) for si in s]
                z = sum(p)
                for e in range(head_dim):
                    o.append(sum(p[t] * vs[t][j][e] for t in range(L)) / z)
            g1, sh2, sc2, g2 = mod(i, 2), mod(i, 3), mod(i, 4), mod(i, 5)
            ao = _matvec(w["o_w"], w["o_b"], o)
            x1 = [x[b][i][c] + g1[c] * ao[c] for c in range(D)]
            xh2 = _ln(x1, ln_eps)
            h2 = [xh2[c] * (1.0 + sc2[c]) + sh2[c] for c in range(D)]
            g = [_gelu(u) for u in _matvec(w["up_w"], w["up_b"], h2)]
            mo = _matvec(w["down_w"], w["down_b"], g)
            rows.append([x1[c] + g2[c] * mo[c] for c in range(D)])
        out.append(rows)
    return out
