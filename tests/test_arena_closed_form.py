"""The block's arena size against a closed form derived by hand (CPU only).

The planner (csrc/plan.cpp) and the oracle's layout (oracle/layout.py) each
carry a slot table and pack it with Algorithm 1 (Sec. 6.1); those two are
checked against each other elsewhere.  This test pins both to a formula
written from the block's data flow alone, so a slot that is too large, too
small or live too long shows up as a byte count that differs.

Derivation.  R(n) rounds n up to 256 bytes (every slot is 256-byte aligned).
B sequences of L tokens, chunk c (c = L unchunked), hidden D, MLP width F,
Lp = L rounded up to 128, S = 2 modulation maps for a dual-stream block else 1.

  always live (steps 0-9):  the AdaLN vectors R(24 B D S) (fp32 [S, B, 6D]),
                            the range flags R(16),
                            Q, K and V^T, 3 R(2 B D Lp) (fp16, all tokens;
                            every query chunk reads every key)
  phase A peak (step 1):    the RoPE table R(8 sum_a G_a d_a / 2) (fp32
                            cos, sin per axis position and pair) + the LN1
                            rows R(2 B c D); the QKV projection writes the
                            heads itself, so no [c, 3D] intermediate exists
  phase B peak (step 8):    the fp16 copies of W_o, W_up, W_down,
                            R(2 D^2) + 2 R(2 F D) (none when the caller
                            passes them in fp16), x1 R(4 B c D) (fp32),
                            the LN2 rows R(2 B c D), the MLP hidden rows
                            R(2 B c F) and, when chunked, the attention
                            rows R(2 B c D), kept live so that the next
                            chunk's attention can overlap this chunk's MLP
  (step 6, attention rows + x1 + copies, never exceeds step 8)

  arena(c) = always + max(phase A, phase B)

Against the simpler estimate arena(c) = 6 B L D + B c max(8D, 6D + 2F) +
24 B D, this adds the 128-token padding of Q/K/V, the RoPE table, the status
words and the weight copies, drops the qkv intermediate (8D -> 2D per token
in phase A) and keeps the attention rows live when chunked.  Algorithm 1
cannot go below this max-live bound; the packer reaching it exactly is part
of what is tested.
"""
import pytest

import oracle.layout as OL
import paper_2607_11136_amd as X
import workloads as W


def R(n: int) -> int:
    return -(-n // 256) * 256


def closed_form_arena(s: W.BlockShape, chunk: int, weights_f16: int) -> int:
    B, L, D, F = s.batch, s.seq_len, s.hidden, s.mlp_hidden
    c = L if chunk <= 0 or chunk >= L else chunk
    Lp = -(-L // 128) * 128
    S = 2 if s.modulation_streams == 2 else 1
    always = R(24 * B * D * S) + R(16) + 3 * R(2 * B * D * Lp)
    rope = R(8 * sum(g * (da // 2) for g, da in zip(s.grid, s.rope_dims)))
    phase_a = rope + R(2 * B * c * D)
    copies = 0 if weights_f16 else R(2 * D * D) + 2 * R(2 * F * D)
    phase_b = copies + R(4 * B * c * D) + R(2 * B * c * D) + R(2 * B * c * F) + (R(2 * B * c * D) if c < L else 0)
    return always + max(phase_a, phase_b)


def _cfg(s, wf16):
    return X.block_cfg(s.hidden, s.heads, s.head_dim, s.mlp_hidden, s.cond_dim, s.rope_dims,
                       s.rope_theta, s.ln_eps, s.qk_eps, s.modulation_streams, wf16)


@pytest.mark.parametrize("name", sorted(W.CONFIGS))
@pytest.mark.parametrize("wf16", [0, 1])
def test_arena_equals_closed_form(name, wf16):
    s = W.CONFIGS[name]
    req = X.request(s.batch, s.text_len, *s.grid)
    for chunk in sorted({0, 1, 64, 256, 1000, 2048, 4096, 8192} | set(s.chunks)):
        want = closed_form_arena(s, chunk, wf16)
        got = X.xema_workspace_bytes(_cfg(s, wf16), req, chunk)
        assert got == want, (name, chunk, wf16, got, want)
        assert OL.workspace_bytes(s.with_(weights_f16=wf16), chunk) == want


def test_closed_form_at_the_video_shape_by_hand():
    """The video workload (B 1, L 17776, D 3072, F 12288, unchunked) worked
    out term by term: Lp = 17792; always = 73,728 (AdaLN vectors) + 256
    (flags) + 3 x 109,314,048 (Q, K, V^T); phase A = 8,192 (RoPE table, 8,032
    rounded) + 109,215,744 (LN1 rows); phase B = 18,874,368 + 2 x 75,497,472
    (weight copies) + 218,431,488 (x1) + 109,215,744 (LN2 rows) +
    436,862,976 (hidden rows) = 934,379,520, larger than phase A."""
    s = W.VIDEO
    assert closed_form_arena(s, 0, 0) == 73728 + 256 + 3 * 109314048 + 934379520 == 1262395648
    assert closed_form_arena(s, 0, 1) == 1262395648 - (18874368 + 2 * 75497472)
