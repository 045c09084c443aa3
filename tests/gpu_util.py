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
                       s.rope_theta, s.ln_eps, s.qk_eps, s.modulation_streams, s.weights_f16)


def req_of(s: W.BlockShape) -> X.Request:
    return X.request(s.batch, s.text_len, *s.grid)


PHASE_B_WEIGHTS = ("o_w", "up_w", "down_w")


def poison(t: torch.Tensor) -> torch.Tensor:
    """Fill a device buffer with 0xFF bytes (an fp16/bf16/fp32 NaN pattern),
    so that any element a kernel fails to write shows up as NaN."""
    t.view(torch.uint8).fill_(0xFF)
    return t


class Device:
    """Seeded inputs of one shape resident on the GPU.  With the shape's
    weights_f16 set, W_o, W_up and W_down are handed over as fp16 (the bf16
    values converted exactly once, as a serving process would at load)."""

    def __init__(self, inputs: W.Inputs):
        self.inputs = inputs
        self.shape = inputs.shape
        self.x = bf16_dev(inputs.x)
        self.cond = bf16_dev(inputs.cond)
        self.w = {k: bf16_dev(v) for k, v in inputs.weights.items()}
        if self.shape.weights_f16:
            for k in PHASE_B_WEIGHTS:
                self.w[k] = self.w[k].to(torch.float16)
        self.weights = X.block_weights(self.w)
        self.cfg = cfg_of(self.shape)
        self.req = req_of(self.shape)

    def run(self, chunk: int = 0, ws: torch.Tensor | None = None, stream=None, check_status: bool = True):
        """Block forward into a poisoned output and workspace; returns (out
        fp32 [B, L, D] on device, workspace, plan).  Asserts a clean range
        status unless told not to."""
        s = self.shape
        plan = X.xema_workspace_layout(self.cfg, self.req, chunk)
        if ws is None or ws.numel() < plan.workspace_bytes:
            ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
        poison(ws)
        out = poison(torch.empty((s.batch, s.seq_len, s.hidden), dtype=torch.float32, device=DEV))
        X.xema_dit_block_fwd(self.cfg, self.req, self.x, self.weights, self.cond, chunk, ws,
                             ws.numel(), out, stream)
        torch.cuda.synchronize()
        if check_status:
            assert X.xema_block_status(plan, ws) == 0, "fp16 range status raised"
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
