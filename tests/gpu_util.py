"""Helpers shared by the GPU tests: upload seeded inputs, run the block through
the C ABI, compare against the oracle with the tolerances of the parity bar."""
from __future__ import annotations

import numpy as np
import torch

import paper_2607_11136_amd as X
import workloads as W

DEV = "cuda:0"

# Parity bar for the block output (fp64 oracle vs GPU): elementwise
# |g - o| / max(|o|, 1) <= 2e-2 and mean |g - o| <= 2e-3.
MAX_REL = 2e-2
MAE = 2e-3


def bf16_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def f64_to_f16_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.asarray(a, dtype=np.float16)).to(DEV)


def cfg_of(s: W.BlockShape) -> X.BlockCfg:
    return X.block_cfg(s.hidden, s.heads, s.head_dim, s.mlp_hidden, s.cond_dim, s.rope_dims,
                       s.rope_theta, s.ln_eps, s.qk_eps, s.modulation_streams)


def req_of(s: W.BlockShape) -> X.Request:
    return X.request(s.batch, s.text_len, *s.grid)


class Device:
    """Seeded inputs of one shape resident on the GPU."""

    def __init__(self, inputs: W.Inputs):
        self.inputs = inputs
        self.shape = inputs.shape
        self.x = bf16_dev(inputs.x)
        self.cond = bf16_dev(inputs.cond)
        self.w = {k: bf16_dev(v) for k, v in inputs.weights.items()}
        self.weights = X.block_weights(self.w)
        self.cfg = cfg_of(self.shape)
        self.req = req_of(self.shape)

    def run(self, chunk: int = 0, ws: torch.Tensor | None = None, stream=None):
        """Block forward; returns (out fp32 [B, L, D] on device, workspace, plan)."""
        s = self.shape
        plan = X.xema_workspace_layout(self.cfg, self.req, chunk)
        if ws is None or ws.numel() < plan.workspace_bytes:
            ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
        out = torch.empty((s.batch, s.seq_len, s.hidden), dtype=torch.float32, device=DEV)
        X.xema_dit_block_fwd(self.cfg, self.req, self.x, self.weights, self.cond, chunk, ws,
                             ws.numel(), out, stream)
        torch.cuda.synchronize()
        return out, ws, plan


def slot_view(ws: torch.Tensor, plan: X.Plan, name: str, dtype, shape) -> torch.Tensor:
    off, nbytes, _, _ = plan.slots()[name]
    n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
    assert n <= nbytes
    return ws[off:off + n].view(dtype).view(*shape)


def errors(gpu: np.ndarray, ref: np.ndarray):
    d = np.abs(gpu.astype(np.float64) - ref)
    return {"mae": float(d.mean()), "max_rel": float(np.max(d / np.maximum(np.abs(ref), 1.0))),
            "max_abs": float(d.max())}


def assert_parity(gpu: np.ndarray, ref: np.ndarray, what: str):
    e = errors(gpu, ref)
    print(f"{what}: {e}", flush=True)
    assert np.all(np.isfinite(gpu)), what
    assert e["max_rel"] <= MAX_REL and e["mae"] <= MAE, (what, e)
    return e
