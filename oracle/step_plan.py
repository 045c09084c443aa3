"""Whole-step planning of an N-block denoising step: TEST INFRASTRUCTURE.

Only tests/ may import this module; the HIP path shares no code with it.

What it computes, on plain integers and floats:

* The step's lifetime trace (the memory analyzer's trace, Sec. 7.2, written
  out from the block's slot table instead of recorded from a shape-only
  run): every block i contributes the slots of its arena (oracle.layout's
  slot table for a g-sequence request at chunk c) at steps 10 i + s, where s
  is the block's own step; the fp32 residual stream between blocks
  contributes the buffers x_{i+1} the workspace holds (block i's output, for
  N - 1 - i odd; the caller's output holds the others), alive through block
  i+1's last step from the first step of the loop that writes them: block
  i writes x_{i+1} at its step 9, which repeats for every chunk (the steps
  5-9 of phase B) and, with several groups, with the whole block, so the
  first write precedes later chunks' or groups' use of the block's other
  slots (step 5 when chunked, step 0 with several groups, step 9 for one
  unchunked pass); the staging slots of offloaded
  weights are alive for the whole step.
* Algorithm 1 (Sec. 6.1) over that trace: oracle.layout.static_layout.
* The latency model (reading R30): a block's time is the sum over its
  launches of the rounds of workgroups over the 256 CUs, a round costing one
  workgroup's FLOPs at block_tflops / 256 per CU (GEMM tiles of 256 x 256,
  attention query blocks of 512 queries at head_dim 64 and 256 at 128, each
  over all L keys); a copy of one block's weights takes slot bytes at
  h2d GB/s; copies run in order on a copy stream, the copy of offloaded block
  k starting after copy k-1 and after offloaded block k - S (which used its
  staging slot) has finished; a block starts after its predecessor and, if
  offloaded, its copy.
* The plan (Sec. 5.1, pi*, with offloading, serialization and chunking as
  the mitigations, and one device budget over the resident weights and the
  workspace): the (K, g, c) with the least modelled time, ties to fewer
  offloaded blocks, then the larger group, then the larger chunk.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Tuple

from . import layout as LY
from . import offload as OF
from .layout import block_ms  # the latency model (reading R30), shared with the block plan

STEPS_PER_BLOCK = 10


def step_tensors(shape, n_blocks: int, group: int, chunk: int, n_staging: int, slot_bytes: int,
                 weights_f16: int = 0) -> Tuple[List[LY.Tensor], Dict[int, tuple]]:
    """The step's trace: tensors (ids in block-major order, then the residual
    buffers, then the staging slots) and what each id is."""
    s = shape
    block = LY.block_tensors(group, s.seq_len, s.hidden, s.mlp_hidden, s.grid, s.rope_dims, chunk,
                             s.modulation_streams, weights_f16)
    ns = len(block)
    out, what = [], {}
    for i in range(n_blocks):
        for t in block:
            if t.size > 0:
                tid = i * ns + t.sid
                out.append(LY.Tensor(tid, t.size, STEPS_PER_BLOCK * i + t.begin, STEPS_PER_BLOCK * i + t.end))
                what[tid] = ("slot", i, t.sid)
    resid = 4 * s.batch * s.seq_len * s.hidden
    c = s.seq_len if chunk <= 0 or chunk >= s.seq_len else chunk
    first = 0 if group < s.batch else (5 if c < s.seq_len else 9)
    for i in range(n_blocks - 1):
        if (n_blocks - 1 - i) % 2 == 1:
            tid = n_blocks * ns + i
            out.append(LY.Tensor(tid, resid, STEPS_PER_BLOCK * i + first, STEPS_PER_BLOCK * i + 20))
            what[tid] = ("resid", i)
    for j in range(n_staging):
        tid = n_blocks * ns + n_blocks + j
        out.append(LY.Tensor(tid, slot_bytes, 0, STEPS_PER_BLOCK * n_blocks))
        what[tid] = ("staging", j)
    return out, what


def step_workspace(shape, n_blocks: int, group: int, chunk: int, n_staging: int, slot_bytes: int,
                   weights_f16: int = 0) -> int:
    ts, _ = step_tensors(shape, n_blocks, group, chunk, n_staging, slot_bytes, weights_f16)
    return LY.static_layout(ts)[1]


def step_ms(n_blocks: int, offloaded: List[int], n_staging: int, t_blk: float, t_x: float) -> float:
    """The event schedule of the two streams (see the module docstring)."""
    S = max(n_staging, 1)
    off = set(offloaded)
    order = sorted(off)
    block_end, copy_end = {}, []
    copy_free = 0.0
    t = 0.0
    k = 0
    for i in range(n_blocks):
        start = t
        if i in off:
            while len(copy_end) <= k:
                j = len(copy_end)
                ready = copy_free if j < S else max(copy_free, block_end[order[j - S]])
                copy_free = ready + t_x
                copy_end.append(copy_free)
            start = max(start, copy_end[k])
            k += 1
        block_end[i] = start + t_blk
        t = block_end[i]
    return t


def plan_fixed(shape, n_blocks: int, k: int, n_staging: int, group: int, chunk: int,
               h2d_gbps: float = 56.0, tflops: float = 1000.0) -> dict:
    s = shape
    sizes = OF.block_weight_sizes(s.hidden, s.mlp_hidden, s.cond_dim, s.head_dim, s.modulation_streams)
    op = OF.plan(n_blocks, k, n_staging, sizes)
    L = s.seq_len
    c = L if chunk <= 0 or chunk >= L else chunk
    ws = step_workspace(s.with_(batch=s.batch), n_blocks, group, c, op["n_staging"], op["block_weight_bytes"],
                        getattr(s, "weights_f16", 0))
    t_x = op["block_weight_bytes"] / (h2d_gbps * 1e9) * 1e3
    est = step_ms(n_blocks, op["offloaded"], op["n_staging"], block_ms(s, group, c, tflops), t_x)
    return {"k": k, "group": group, "chunk": c, "offloaded": op["offloaded"], "n_staging": op["n_staging"],
            "workspace_bytes": ws, "device_bytes": op["resident_weight_bytes"] + ws, "est_ms": est}


def plan_budget(shape, n_blocks: int, n_staging: int, budget: int, h2d_gbps: float = 56.0,
                tflops: float = 1000.0) -> Optional[dict]:
    """The feasible (K, g, c) with the least modelled time (ties: fewer
    offloaded blocks, larger group, larger chunk), or None."""
    s = shape
    groups = [g for g in range(s.batch, 0, -1) if s.batch % g == 0]
    best = None
    for k in range(n_blocks + 1):
        for g in groups:
            for c in LY.chunk_candidates(s.seq_len):
                p = plan_fixed(s, n_blocks, k, n_staging, g, c, h2d_gbps, tflops)
                if p["device_bytes"] > budget:
                    continue
                key = (p["est_ms"], k, -g, -c)
                if best is None or key < best[0]:
                    best = (key, p)
    return None if best is None else best[1]
