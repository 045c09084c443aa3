"""Offline static memory layout and budget planning (test infrastructure only).

Algorithm 1 of the paper (Sec. 6.1, "Offline static layout"): tensors are
rectangles on an address-time plane, lifetime as width and size as height;
tensors whose lifetimes overlap must get disjoint address ranges, and the goal
is a low highest-used address.  Tensors are taken largest first; each one goes
into the smallest address gap (among the gaps left by the already-placed
tensors whose lifetimes overlap its own) that can hold it, at the gap's bottom;
if no gap is big enough, it goes directly above every overlapping tensor.

Readings where the paper leaves details open (R17):
  * sizes are rounded up to 256 bytes before packing;
  * equal sizes are ordered by lifetime start, then by slot id;
  * lifetimes are half-open [b, e);
  * the gaps of tensor i are the holes of the union of [a_j, a_j + s_j) over
    the overlapping placed tensors j, inside [0, top), where top is the highest
    end address among them (so a hole at address 0 counts);
  * among equal-size gaps the lower address wins;
  * "above all tensors" means at top (0 when nothing overlaps).

The budget planner follows "only as much mitigation as needed" (Sec. 5.1, the
pi* objective): chunking is the mitigation, its intensity is the chunk size,
and latency does not grow with a bigger chunk, so the plan is the largest
candidate chunk whose arena fits the budget.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

ALIGN = 256
GRANULE = 256          # candidate chunk sizes are multiples of this, or "all"
SEQ_PAD = 128          # per-head sequence storage is padded to this many tokens

SLOT_NAMES = ("mod", "rope", "q", "k", "vt", "ln1", "qkv", "wo16", "wup16", "wdown16",
              "attn", "x1", "ln2", "hid", "status")
STATUS_BYTES = 16      # four range-flag words


def round_up(x: int, a: int) -> int:
    return (x + a - 1) // a * a


@dataclasses.dataclass(frozen=True)
class Tensor:
    sid: int
    size: int
    begin: int
    end: int          # half-open


def overlaps(a: Tensor, b: Tensor) -> bool:
    return a.begin < b.end and b.begin < a.end


def static_layout(tensors: Sequence[Tensor]) -> Tuple[List[int], int]:
    """Algorithm 1.  Returns (offset per tensor in input order, peak address)."""
    sized = [dataclasses.replace(t, size=round_up(t.size, ALIGN)) for t in tensors]
    order = sorted(range(len(sized)), key=lambda i: (-sized[i].size, sized[i].begin, sized[i].sid))
    offset: List[Optional[int]] = [None] * len(sized)
    placed: List[int] = []
    for i in order:
        ti = sized[i]
        conflicts = [j for j in placed if overlaps(ti, sized[j])]
        ivals = sorted((offset[j], offset[j] + sized[j].size) for j in conflicts)
        top = max((hi for _, hi in ivals), default=0)
        # holes of the union of the conflict intervals inside [0, top)
        gaps = []
        cursor = 0
        for lo, hi in ivals:
            if lo > cursor:
                gaps.append((cursor, lo - cursor))
            cursor = max(cursor, hi)
        fitting = [g for g in gaps if g[1] >= ti.size]
        if fitting:
            best = min(fitting, key=lambda g: (g[1], g[0]))
            offset[i] = best[0]
        else:
            offset[i] = top
        placed.append(i)
    peak = max((offset[i] + sized[i].size for i in range(len(sized))), default=0)
    return [int(o) for o in offset], int(peak)


def max_live_bytes(tensors: Sequence[Tensor]) -> int:
    """Largest total (256-rounded) size alive at one time: a lower bound of any layout."""
    steps = sorted({t.begin for t in tensors})
    best = 0
    for s in steps:
        best = max(best, sum(round_up(t.size, ALIGN) for t in tensors if t.begin <= s < t.end))
    return best


# -- the block's slot table ---------------------------------------------------------


def padded_len(seq_len: int) -> int:
    return round_up(seq_len, SEQ_PAD)


def rope_table_bytes(grid: Sequence[int], rope_dims: Sequence[int]) -> int:
    """cos/sin (fp32 pair) per position and rotated pair, per axis."""
    return 8 * sum(int(g) * (int(da) // 2) for g, da in zip(grid, rope_dims))


def block_tensors(batch: int, seq_len: int, hidden: int, mlp_hidden: int,
                  grid: Sequence[int], rope_dims: Sequence[int], chunk: int,
                  modulation_streams: int = 1, weights_f16: int = 0) -> List[Tensor]:
    """Slot table of one block call with `chunk` tokens per sequence per chunk.

    Steps (folded over the chunk loops): 0 = AdaLN map and RoPE table;
    phase A (per token chunk) 1 = LN1, 2 = QKV projection, 3 = QK-norm/RoPE
    scatter; 4 = fp16 copies of the three phase-B weight matrices; phase B (per
    query chunk) 5 = attention, 6 = out-projection with gated residual, 7 = LN2,
    8 = MLP up + GELU, 9 = MLP down + gated residual.  Per-chunk slots are
    reused by every chunk; Q, K, V hold all tokens, padded to a multiple of
    SEQ_PAD tokens.  In a chunked call the attention buffer stays live
    through the chunk's MLP (steps 5-9), so the next chunk's attention may
    run meanwhile on a second stream.  A dual-stream block (reading R24) keeps both modulation
    vectors, so its mod slot doubles.  The QKV projection writes Q, K and V^T
    itself (reading R28; head_dim is 64 or 128), so the [tokens, 3D] qkv slot
    is empty.  With weights_f16 the caller passes W_o, W_up and W_down in
    fp16 and the three copy slots are empty.  The status slot holds the
    range flags for the whole call."""
    B, D, F = batch, hidden, mlp_hidden
    c = seq_len if chunk <= 0 or chunk >= seq_len else chunk
    lp = padded_len(seq_len)
    spec = [
        ("mod", 24 * B * D * modulation_streams, 0, 10),
        ("rope", rope_table_bytes(grid, rope_dims), 0, 4),
        ("q", 2 * B * D * lp, 1, 10),
        ("k", 2 * B * D * lp, 1, 10),
        ("vt", 2 * B * D * lp, 1, 10),
        ("ln1", 2 * B * c * D, 1, 3),
        ("qkv", 0, 2, 4),
        ("wo16", 0 if weights_f16 else 2 * D * D, 4, 10),
        ("wup16", 0 if weights_f16 else 2 * F * D, 4, 10),
        ("wdown16", 0 if weights_f16 else 2 * D * F, 4, 10),
        ("attn", 2 * B * c * D, 5, 10 if c < seq_len else 7),
        ("x1", 4 * B * c * D, 6, 10),
        ("ln2", 2 * B * c * D, 7, 9),
        ("hid", 2 * B * c * F, 8, 10),
        ("status", STATUS_BYTES, 0, 10),
    ]
    assert tuple(n for n, *_ in spec) == SLOT_NAMES
    return [Tensor(i, s, b, e) for i, (_, s, b, e) in enumerate(spec)]


def workspace_bytes(shape, chunk: int) -> int:
    """Arena bytes (Algorithm 1 peak) for a workloads.BlockShape and chunk size."""
    ts = block_tensors(shape.batch, shape.seq_len, shape.hidden, shape.mlp_hidden,
                       shape.grid, shape.rope_dims, chunk, shape.modulation_streams,
                       getattr(shape, "weights_f16", 0))
    return static_layout(ts)[1]


def chunk_candidates(seq_len: int) -> List[int]:
    """All candidate chunk sizes, largest first: every multiple of the granule
    below L, and L itself ("all")."""
    return [seq_len] + list(range((seq_len - 1) // GRANULE * GRANULE, 0, -GRANULE))


def plan(shape, budget_bytes: int):
    """Largest candidate chunk whose arena fits `budget_bytes`.
    Returns (chunk or None, arena bytes at that chunk, the smallest arena over
    the candidates)."""
    cands = chunk_candidates(shape.seq_len)
    smallest = min(workspace_bytes(shape, c) for c in cands)
    for c in cands:
        ws = workspace_bytes(shape, c)
        if ws <= budget_bytes:
            return c, ws, smallest
    return None, None, smallest


CUS = 256  # compute units of the modelled GPU


def block_ms(shape, group: int, chunk: int, tflops: float) -> float:
    """Modelled time of one block in ms (the latency model, reading R30):
    with the batch in groups of `group` sequences and chunks of `chunk`
    tokens, the sum over its launches of the rounds of workgroups over the
    256 CUs, a round costing one workgroup's FLOPs at tflops / 256 per CU
    (GEMM tiles of 256 x 256; attention query blocks of 512 queries at
    head_dim 64 and 256 at 128, each over all L keys)."""
    s = shape
    B, L, D, F, H, d = s.batch, s.seq_len, s.hidden, s.mlp_hidden, s.heads, s.head_dim
    c = L if chunk <= 0 or chunk >= L else chunk
    qwg = 512 if d == 64 else 256

    def rounds(n):
        return math.ceil(n / CUS)

    def gemm(m, n, k):
        return rounds(math.ceil(m / 256) * (n // 256)) * 2.0 * 256 * 256 * k

    flops = 0.0
    for t0 in range(0, L, c):
        ck = min(c, L - t0)
        m = group * ck
        flops += gemm(m, 3 * D, D) + gemm(m, D, D) + gemm(m, F, D) + gemm(m, D, F)
        flops += rounds(math.ceil(ck / qwg) * H * group) * 4.0 * qwg * L * d
    return flops * (B // group) / (tflops * 1e12 / CUS) * 1e3



PLAN_TFLOPS = 1000.0  # any positive rate ranks the same


def plan_serial(shape, budget_bytes: int):
    """Temporary serialization (Sec. 5.2) together with chunking, choosing
    the mitigation with the least latency overhead (Sec. 5.1, pi*) by the
    latency model: for each equal group size g (the batch split into groups
    of g sequences run through the block one after another), the largest
    chunk c whose arena fits `budget_bytes`; among those (g, c) the least
    block_ms, then the larger g.  Returns (g, chunk, arena bytes) or None."""
    B = shape.batch
    best = None
    for g in range(B, 0, -1):
        if B % g:
            continue
        for c in chunk_candidates(shape.seq_len):
            need = workspace_bytes(shape.with_(batch=g), c)
            if need <= budget_bytes:
                ms = block_ms(shape, g, c, PLAN_TFLOPS)
                if best is None or ms < best[3] * (1.0 - 1e-12):
                    best = (g, c, need, ms)
                break
    return None if best is None else best[:3]
