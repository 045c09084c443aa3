"""N-block denoising step in fp64: TEST INFRASTRUCTURE.

The denoiser applies its DiT blocks in sequence (Sec. 2.1), each with its own
weights and the same conditioning: x_{i+1} = block_i(x_i).  Offloading moves
weights between host and device memory and changes nothing here.
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np

from .block import block_forward


def step_forward(x: np.ndarray, cond: np.ndarray, weights: Sequence[Dict[str, np.ndarray]],
                 **block_kw) -> np.ndarray:
    for w in weights:
        x = block_forward(x, cond, w, **block_kw)
    return x
