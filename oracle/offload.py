"""Selective weight offloading for an N-block denoising step: TEST INFRASTRUCTURE.

The paper applies only as much mitigation as needed (Sec. 5.1, objective
pi*): with block offloading as the mitigation, the plan is the smallest
number K of offloaded blocks whose device-resident weights fit the budget,
and the K blocks are spread uniformly over the stack so that about N/K
blocks of computation separate two transfers ("Selective offloading and
HSDP").  This module writes that definition out on plain integers.

Device weight bytes for K offloaded blocks = the (N - K) resident blocks'
tensors + min(S, K) staging slots (S requested), a slot holding one block's
twelve tensors each rounded up to 256 bytes.  Offloaded positions: block
floor((j + 1) N / K) - 1 for j = 0 .. K-1 (the end of each of K equal spans).
"""
from __future__ import annotations

from typing import List, Optional, Sequence

ALIGN = 256


def block_weight_sizes(hidden: int, mlp_hidden: int, cond_dim: int, head_dim: int,
                       modulation_streams: int = 1) -> List[int]:
    """Bytes of the bf16 weight tensors of one block, in the order ada_w,
    ada_b, qkv_w, qkv_b, q_gamma, k_gamma, o_w, o_b, up_w, up_b, down_w,
    down_b, then for a dual-stream block the text tokens' ada_txt_w, ada_txt_b."""
    D, F, Dc, d = hidden, mlp_hidden, cond_dim, head_dim
    elems = [6 * D * Dc, 6 * D, 3 * D * D, 3 * D, d, d, D * D, D, F * D, F, D * F, D]
    if modulation_streams == 2:
        elems += [6 * D * Dc, 6 * D]
    return [2 * e for e in elems]


def slot_bytes(sizes: Sequence[int]) -> int:
    return sum((s + ALIGN - 1) // ALIGN * ALIGN for s in sizes)


def offloaded_positions(n_blocks: int, k: int) -> List[int]:
    return [(j + 1) * n_blocks // k - 1 for j in range(k)]


def plan(n_blocks: int, k: int, n_staging: int, sizes: Sequence[int]) -> dict:
    staging = min(n_staging, k) if k > 0 else 0
    resident = (n_blocks - k) * sum(sizes)
    return {"n_offloaded": k, "n_staging": staging, "offloaded": offloaded_positions(n_blocks, k),
            "block_weight_bytes": slot_bytes(sizes), "resident_weight_bytes": resident,
            "staging_bytes": staging * slot_bytes(sizes),
            "device_weight_bytes": resident + staging * slot_bytes(sizes)}


def plan_for_budget(n_blocks: int, budget: int, n_staging: int, sizes: Sequence[int]) -> Optional[dict]:
    """The smallest K whose device weight bytes fit `budget`, or None."""
    for k in range(n_blocks + 1):
        p = plan(n_blocks, k, n_staging, sizes)
        if p["device_weight_bytes"] <= budget:
            return p
    return None
