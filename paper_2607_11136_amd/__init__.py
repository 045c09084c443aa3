"""Python binding of libxema, the MI355X (gfx950) DiT block forward.

A thin ctypes layer over the C ABI declared in include/xema.h and
include/xema_ops.h: the functions keep the C names, take torch tensors (device
memory) or plain integers, and raise XemaError on a non-zero status.  Every
step of the block runs in the library's HIP kernels; torch only provides device
memory and the stream.  The shared library is loaded from this directory on
first use; if it is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libxema.so")

XEMA_OK = 0
XEMA_ERR_INVALID_ARG = -1
XEMA_ERR_UNSUPPORTED = -2
XEMA_ERR_BUDGET_TOO_SMALL = -3
XEMA_ERR_WORKSPACE_TOO_SMALL = -4
XEMA_ERR_MISALIGNED = -5
XEMA_ERR_HIP = -6
XEMA_ERR_RANGE = -7

# range status bits (xema_block_status)
XEMA_RANGE_QKV, XEMA_RANGE_LN2, XEMA_RANGE_MLP, XEMA_RANGE_WEIGHTS = 1, 2, 4, 8
XEMA_STATUS_WORDS = 4

XEMA_MAX_SLOTS = 16
XEMA_CHUNK_GRANULE = 256
XEMA_SEQ_PAD = 128

XEMA_BF16, XEMA_F16, XEMA_F32 = 0, 1, 2
XEMA_EPI_BIAS, XEMA_EPI_BIAS_GELU, XEMA_EPI_GATED_RESIDUAL = 0, 1, 2

SLOT_NAMES = ("mod", "rope", "q", "k", "vt", "ln1", "qkv", "wo16", "wup16", "wdown16",
              "attn", "x1", "ln2", "hid", "status")
SLOT = {n: i for i, n in enumerate(SLOT_NAMES)}

WEIGHT_FIELDS = ("ada_w", "ada_b", "qkv_w", "qkv_b", "q_gamma", "k_gamma",
                 "o_w", "o_b", "up_w", "up_b", "down_w", "down_b")
# the text tokens' AdaLN map of a dual-stream block (modulation_streams = 2)
TEXT_MOD_FIELDS = ("ada_txt_w", "ada_txt_b")


class XemaError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {xema_status_str(status)} ({status})")


class BlockCfg(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("mlp_hidden", ctypes.c_int32), ("cond_dim", ctypes.c_int32),
                ("rope_dims", ctypes.c_int32 * 3), ("rope_theta", ctypes.c_float),
                ("ln_eps", ctypes.c_float), ("qk_eps", ctypes.c_float),
                ("modulation_streams", ctypes.c_int32), ("weights_f16", ctypes.c_int32)]


class Request(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("text_len", ctypes.c_int32), ("grid_t", ctypes.c_int32),
                ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32)]

    @property
    def seq_len(self) -> int:
        return self.text_len + self.grid_t * self.grid_h * self.grid_w


class BlockWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_FIELDS + TEXT_MOD_FIELDS]


class Plan(ctypes.Structure):
    _fields_ = [("chunk_tokens", ctypes.c_int32), ("n_slots", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_int64), ("min_workspace_bytes", ctypes.c_int64),
                ("slot_offset", ctypes.c_int64 * XEMA_MAX_SLOTS),
                ("slot_bytes", ctypes.c_int64 * XEMA_MAX_SLOTS),
                ("slot_begin", ctypes.c_int32 * XEMA_MAX_SLOTS),
                ("slot_end", ctypes.c_int32 * XEMA_MAX_SLOTS)]

    def slots(self) -> Dict[str, tuple]:
        """name -> (offset, bytes, begin, end)"""
        return {SLOT_NAMES[i]: (self.slot_offset[i], self.slot_bytes[i], self.slot_begin[i],
                                self.slot_end[i]) for i in range(self.n_slots)}


class RowMap(ctypes.Structure):
    _fields_ = [("rows_per_batch", ctypes.c_int64), ("batch_stride", ctypes.c_int64),
                ("row_offset", ctypes.c_int64)]


class GemmArgs(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("a", ctypes.c_void_p), ("M", ctypes.c_int64),
                ("K", ctypes.c_int32), ("b", ctypes.c_void_p), ("N", ctypes.c_int32),
                ("bias", ctypes.c_void_p), ("epilogue", ctypes.c_int32),
                ("c", ctypes.c_void_p), ("c_dtype", ctypes.c_int32), ("c_map", RowMap),
                ("ldc", ctypes.c_int64), ("resid", ctypes.c_void_p), ("resid_dtype", ctypes.c_int32),
                ("resid_map", RowMap), ("ld_resid", ctypes.c_int64),
                ("gate", ctypes.c_void_p), ("gate_stride", ctypes.c_int64)]


XEMA_MAX_BLOCKS = 256


class OffloadPlan(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("n_offloaded", ctypes.c_int32),
                ("n_staging", ctypes.c_int32), ("offloaded", ctypes.c_int32 * XEMA_MAX_BLOCKS),
                ("block_weight_bytes", ctypes.c_int64), ("resident_weight_bytes", ctypes.c_int64),
                ("staging_bytes", ctypes.c_int64), ("device_weight_bytes", ctypes.c_int64)]

    def offloaded_blocks(self) -> List[int]:
        return [i for i in range(self.n_blocks) if self.offloaded[i]]


class StepCosts(ctypes.Structure):
    _fields_ = [("h2d_gbytes_per_s", ctypes.c_double), ("block_tflops", ctypes.c_double)]


class StepPlan(ctypes.Structure):
    _fields_ = [("offload", OffloadPlan), ("batch_group", ctypes.c_int32), ("chunk_tokens", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_int64), ("device_bytes", ctypes.c_int64), ("est_ms", ctypes.c_double)]


_P = ctypes.c_void_p
_I32, _I64, _F32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
_SIGNATURES = {
    "xema_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "xema_request_from_template": (ctypes.c_int, [ctypes.POINTER(BlockCfg), _I32, _I32, _I32, _I32,
                                                  _I32, ctypes.POINTER(Request)]),
    "xema_workspace_layout": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _I32,
                                             ctypes.POINTER(Plan)]),
    "xema_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _I32,
                                            ctypes.POINTER(_I64)]),
    "xema_workspace_plan": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _I64,
                                           ctypes.POINTER(Plan)]),
    "xema_dit_block_fwd": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P,
                                          ctypes.POINTER(BlockWeights), _P, _I32, _P, _I64, _P, _P]),
    "xema_op_adaln": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _I32, _P, _P]),
    "xema_op_ln_modulate": (ctypes.c_int, [_P, _I32, RowMap, _I64, _I32, _P, _P, _I64, _F32, _P,
                                           _I32, _P]),
    "xema_op_gemm": (ctypes.c_int, [ctypes.POINTER(GemmArgs), _P]),
    "xema_op_rope_table": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P, _P]),
    "xema_op_qk_norm_rope": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P,
                                            _I32, _I32, _P, _P, _P, _P, _P, _P, _P]),
    "xema_op_attention": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _P, _P]),
    "xema_op_convert_f16": (ctypes.c_int, [_P, _P, _I64, _P]),
    "xema_workspace_plan_serial": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request),
                                                  _I64, ctypes.POINTER(_I32), ctypes.POINTER(Plan)]),
    "xema_dit_block_fwd_serial": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P,
                                                 ctypes.POINTER(BlockWeights), _P, _I32, _I32, _P, _I64,
                                                 _P, _P]),
    "xema_offload_plan_k": (ctypes.c_int, [ctypes.POINTER(BlockCfg), _I32, _I32, _I32,
                                           ctypes.POINTER(OffloadPlan)]),
    "xema_offload_plan_budget": (ctypes.c_int, [ctypes.POINTER(BlockCfg), _I32, _I64, _I32,
                                                ctypes.POINTER(OffloadPlan)]),
    "xema_step_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request),
                                                 _I32, ctypes.POINTER(OffloadPlan),
                                                 ctypes.POINTER(_I64)]),
    "xema_dit_step_fwd": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P,
                                         ctypes.POINTER(BlockWeights), ctypes.POINTER(OffloadPlan),
                                         _P, _I32, _P, _I64, _P, _P, _P]),
    "xema_step_plan_fixed": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _I32, _I32, _I32,
                                            _I32, _I32, ctypes.POINTER(StepCosts), ctypes.POINTER(StepPlan)]),
    "xema_step_plan_budget": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _I32, _I32, _I64,
                                             ctypes.POINTER(StepCosts), ctypes.POINTER(StepPlan)]),
    "xema_dit_step_fwd_planned": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P,
                                                 ctypes.POINTER(BlockWeights), ctypes.POINTER(StepPlan), _P, _P,
                                                 _I64, _P, _P, _P]),
    "xema_dit_block_fwd_pipelined": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P,
                                                    ctypes.POINTER(BlockWeights), _P, _I32, _I32, _P, _I64, _P,
                                                    _P, _P]),
    "xema_block_status": (ctypes.c_int, [ctypes.POINTER(Plan), _P, _P, ctypes.POINTER(ctypes.c_uint32)]),
    "xema_dit_block_fwd_static": (ctypes.c_int, [ctypes.POINTER(BlockCfg), ctypes.POINTER(Request), _P,
                                                 ctypes.POINTER(BlockWeights), _P, _I32, _P, _P]),
    "xema_vae_upconv_weight_bytes": (ctypes.c_int, [_I32, _I32, ctypes.POINTER(_I64)]),
    "xema_vae_upconv_prepare": (ctypes.c_int, [_P, _I32, _I32, _P, _P]),
    "xema_vae_upconv": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _P, _P, _I32, _I32, _I32, _P, _P]),
}
EXPORTED = tuple(_SIGNATURES)

_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """The loaded libxema.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_11136_amd.build` (needs hipcc)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def _check(status: int, what: str) -> None:
    if status != XEMA_OK:
        raise XemaError(status, what)


def _ptr(x) -> Optional[int]:
    """Device address of a torch tensor, or an integer address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# -- construction helpers ----------------------------------------------------------


def block_cfg(hidden: int, heads: int, head_dim: int, mlp_hidden: int, cond_dim: int,
              rope_dims: Sequence[int], rope_theta: float = 10000.0, ln_eps: float = 1e-6,
              qk_eps: float = 1e-6, modulation_streams: int = 1, weights_f16: int = 0) -> BlockCfg:
    c = BlockCfg()
    c.hidden, c.heads, c.head_dim, c.mlp_hidden, c.cond_dim = hidden, heads, head_dim, mlp_hidden, cond_dim
    for i in range(3):
        c.rope_dims[i] = int(rope_dims[i])
    c.rope_theta, c.ln_eps, c.qk_eps = rope_theta, ln_eps, qk_eps
    c.modulation_streams = modulation_streams
    c.weights_f16 = weights_f16
    return c


def request(batch: int, text_len: int, grid_t: int, grid_h: int, grid_w: int) -> Request:
    r = Request()
    r.batch, r.text_len, r.grid_t, r.grid_h, r.grid_w = batch, text_len, grid_t, grid_h, grid_w
    return r


def block_weights(tensors: Dict[str, object]) -> BlockWeights:
    """The weight struct from named tensors: the twelve of WEIGHT_FIELDS, plus
    the TEXT_MOD_FIELDS of a dual-stream block when present."""
    w = BlockWeights()
    for n in WEIGHT_FIELDS:
        setattr(w, n, _ptr(tensors[n]))
    for n in TEXT_MOD_FIELDS:
        if n in tensors:
            setattr(w, n, _ptr(tensors[n]))
    return w


def rowmap(rows_per_batch: int, batch_stride: int = 0, row_offset: int = 0) -> RowMap:
    m = RowMap()
    m.rows_per_batch, m.batch_stride, m.row_offset = rows_per_batch, batch_stride, row_offset
    return m


# -- the C entry points ------------------------------------------------------------------


def xema_status_str(status: int) -> str:
    return lib().xema_status_str(status).decode()


def xema_request_from_template(cfg: BlockCfg, height: int, width: int, frames: int, batch: int,
                               text_len: int) -> Request:
    r = Request()
    _check(lib().xema_request_from_template(ctypes.byref(cfg), height, width, frames, batch,
                                            text_len, ctypes.byref(r)), "xema_request_from_template")
    return r


def xema_workspace_layout(cfg: BlockCfg, req: Request, chunk_tokens: int = 0) -> Plan:
    p = Plan()
    _check(lib().xema_workspace_layout(ctypes.byref(cfg), ctypes.byref(req), chunk_tokens,
                                       ctypes.byref(p)), "xema_workspace_layout")
    return p


def xema_workspace_bytes(cfg: BlockCfg, req: Request, chunk_tokens: int = 0) -> int:
    n = _I64()
    _check(lib().xema_workspace_bytes(ctypes.byref(cfg), ctypes.byref(req), chunk_tokens,
                                      ctypes.byref(n)), "xema_workspace_bytes")
    return n.value


def xema_workspace_plan(cfg: BlockCfg, req: Request, budget_bytes: int) -> Plan:
    """Largest chunk whose arena fits the budget.  Raises XemaError
    (XEMA_ERR_BUDGET_TOO_SMALL) when none fits; the error carries the plan
    with min_workspace_bytes as `.plan`."""
    p = Plan()
    st = lib().xema_workspace_plan(ctypes.byref(cfg), ctypes.byref(req), int(budget_bytes),
                                   ctypes.byref(p))
    if st != XEMA_OK:
        e = XemaError(st, "xema_workspace_plan")
        e.plan = p
        raise e
    return p


def xema_dit_block_fwd(cfg: BlockCfg, req: Request, tokens, weights: BlockWeights, cond,
                       chunk_tokens: int, workspace, workspace_bytes: int, out,
                       stream=None) -> None:
    _check(lib().xema_dit_block_fwd(ctypes.byref(cfg), ctypes.byref(req), _ptr(tokens),
                                    ctypes.byref(weights), _ptr(cond), chunk_tokens,
                                    _ptr(workspace), int(workspace_bytes), _ptr(out),
                                    _stream(stream)), "xema_dit_block_fwd")


def xema_block_status(plan: Plan, workspace, stream=None) -> int:
    """Range flags (XEMA_RANGE_* bits, 0 when clean) of the last block call
    on this workspace; waits for the stream."""
    flags = ctypes.c_uint32()
    st = lib().xema_block_status(ctypes.byref(plan), _ptr(workspace), _stream(stream), ctypes.byref(flags))
    if st not in (XEMA_OK, XEMA_ERR_RANGE):
        raise XemaError(st, "xema_block_status")
    return flags.value


XEMA_STATIC_ARENA_BYTES = 64 << 20


def xema_dit_block_fwd_static(cfg: BlockCfg, req: Request, tokens, weights: BlockWeights, cond,
                              chunk_tokens: int, out, stream=None) -> None:
    """The block forward with its arena in the library's static device array
    (no workspace, no allocation; xema_static.h)."""
    _check(lib().xema_dit_block_fwd_static(ctypes.byref(cfg), ctypes.byref(req), _ptr(tokens),
                                           ctypes.byref(weights), _ptr(cond), chunk_tokens, _ptr(out),
                                           _stream(stream)), "xema_dit_block_fwd_static")


def xema_workspace_plan_serial(cfg: BlockCfg, req: Request, budget_bytes: int):
    """(batch_group, plan): temporary serialization only when chunking alone
    cannot fit the budget.  Raises XemaError (XEMA_ERR_BUDGET_TOO_SMALL, the
    plan with min_workspace_bytes as `.plan`)."""
    p = Plan()
    g = _I32()
    st = lib().xema_workspace_plan_serial(ctypes.byref(cfg), ctypes.byref(req), int(budget_bytes),
                                          ctypes.byref(g), ctypes.byref(p))
    if st != XEMA_OK:
        e = XemaError(st, "xema_workspace_plan_serial")
        e.plan = p
        raise e
    return g.value, p


def xema_dit_block_fwd_pipelined(cfg: BlockCfg, req: Request, tokens, weights: BlockWeights, cond,
                                 batch_group: int, chunk_tokens: int, workspace, workspace_bytes: int, out,
                                 stream=None, aux_stream=None) -> None:
    """xema_dit_block_fwd_serial with each chunk's attention on aux_stream."""
    _check(lib().xema_dit_block_fwd_pipelined(ctypes.byref(cfg), ctypes.byref(req), _ptr(tokens),
                                              ctypes.byref(weights), _ptr(cond), batch_group, chunk_tokens,
                                              _ptr(workspace), int(workspace_bytes), _ptr(out), _stream(stream),
                                              _stream(aux_stream)), "xema_dit_block_fwd_pipelined")


def xema_dit_block_fwd_serial(cfg: BlockCfg, req: Request, tokens, weights: BlockWeights, cond,
                              batch_group: int, chunk_tokens: int, workspace, workspace_bytes: int, out,
                              stream=None) -> None:
    _check(lib().xema_dit_block_fwd_serial(ctypes.byref(cfg), ctypes.byref(req), _ptr(tokens),
                                           ctypes.byref(weights), _ptr(cond), batch_group, chunk_tokens,
                                           _ptr(workspace), int(workspace_bytes), _ptr(out),
                                           _stream(stream)), "xema_dit_block_fwd_serial")


def xema_op_adaln(cond, w, bias, batch: int, cond_dim: int, out_dim: int, mod, stream=None) -> None:
    _check(lib().xema_op_adaln(_ptr(cond), _ptr(w), _ptr(bias), batch, cond_dim, out_dim,
                               _ptr(mod), _stream(stream)), "xema_op_adaln")


def xema_op_ln_modulate(x, x_dtype: int, xmap: RowMap, rows: int, dim: int, shift, scale,
                        mod_stride: int, eps: float, y, y_dtype: int, stream=None) -> None:
    _check(lib().xema_op_ln_modulate(_ptr(x), x_dtype, xmap, rows, dim, _ptr(shift), _ptr(scale),
                                     mod_stride, eps, _ptr(y), y_dtype, _stream(stream)),
           "xema_op_ln_modulate")


def xema_op_gemm(args: GemmArgs, stream=None) -> None:
    _check(lib().xema_op_gemm(ctypes.byref(args), _stream(stream)), "xema_op_gemm")


def gemm_args(dtype: int, a, M: int, K: int, b, N: int, bias, epilogue: int, c, c_dtype: int,
              ldc: int, c_map: Optional[RowMap] = None, resid=None, resid_dtype: int = XEMA_F32,
              resid_map: Optional[RowMap] = None, ld_resid: int = 0, gate=None,
              gate_stride: int = 0) -> GemmArgs:
    g = GemmArgs()
    g.dtype, g.a, g.M, g.K, g.b, g.N = dtype, _ptr(a), M, K, _ptr(b), N
    g.bias, g.epilogue, g.c, g.c_dtype, g.ldc = _ptr(bias), epilogue, _ptr(c), c_dtype, ldc
    g.c_map = c_map if c_map is not None else rowmap(max(M, 1), max(M, 1), 0)
    g.resid, g.resid_dtype, g.ld_resid = _ptr(resid), resid_dtype, ld_resid
    g.resid_map = resid_map if resid_map is not None else rowmap(max(M, 1), max(M, 1), 0)
    g.gate, g.gate_stride = _ptr(gate), gate_stride
    return g


def xema_op_rope_table(cfg: BlockCfg, req: Request, table, stream=None) -> None:
    _check(lib().xema_op_rope_table(ctypes.byref(cfg), ctypes.byref(req), _ptr(table),
                                    _stream(stream)), "xema_op_rope_table")


def xema_op_qk_norm_rope(cfg: BlockCfg, req: Request, qkv, tok_begin: int, tok_count: int,
                         q_gamma, k_gamma, table, q, k, vt, stream=None) -> None:
    _check(lib().xema_op_qk_norm_rope(ctypes.byref(cfg), ctypes.byref(req), _ptr(qkv), tok_begin,
                                      tok_count, _ptr(q_gamma), _ptr(k_gamma), _ptr(table), _ptr(q),
                                      _ptr(k), _ptr(vt), _stream(stream)), "xema_op_qk_norm_rope")


def xema_op_attention(q, k, vt, batch: int, heads: int, head_dim: int, seq_len: int,
                      padded_len: int, q_begin: int, q_count: int, o, stream=None) -> None:
    _check(lib().xema_op_attention(_ptr(q), _ptr(k), _ptr(vt), batch, heads, head_dim, seq_len,
                                   padded_len, q_begin, q_count, _ptr(o), _stream(stream)),
           "xema_op_attention")


def xema_op_convert_f16(src, dst, n: int, stream=None) -> None:
    _check(lib().xema_op_convert_f16(_ptr(src), _ptr(dst), n, _stream(stream)), "xema_op_convert_f16")


def padded_len(seq_len: int) -> int:
    return (seq_len + XEMA_SEQ_PAD - 1) // XEMA_SEQ_PAD * XEMA_SEQ_PAD


# -- the N-block step with selective weight offloading (xema_step.h) ---------------


def xema_offload_plan_k(cfg: BlockCfg, n_blocks: int, n_offloaded: int, n_staging: int = 2) -> OffloadPlan:
    p = OffloadPlan()
    _check(lib().xema_offload_plan_k(ctypes.byref(cfg), n_blocks, n_offloaded, n_staging,
                                     ctypes.byref(p)), "xema_offload_plan_k")
    return p


def xema_offload_plan_budget(cfg: BlockCfg, n_blocks: int, weight_budget_bytes: int,
                             n_staging: int = 2) -> OffloadPlan:
    """Smallest K that fits the weight budget.  Raises XemaError
    (XEMA_ERR_BUDGET_TOO_SMALL, with the K = n_blocks plan as `.plan`)."""
    p = OffloadPlan()
    st = lib().xema_offload_plan_budget(ctypes.byref(cfg), n_blocks, int(weight_budget_bytes),
                                        n_staging, ctypes.byref(p))
    if st != XEMA_OK:
        e = XemaError(st, "xema_offload_plan_budget")
        e.plan = p
        raise e
    return p


def xema_step_workspace_bytes(cfg: BlockCfg, req: Request, chunk_tokens: int, plan: OffloadPlan) -> int:
    n = _I64()
    _check(lib().xema_step_workspace_bytes(ctypes.byref(cfg), ctypes.byref(req), chunk_tokens,
                                           ctypes.byref(plan), ctypes.byref(n)),
           "xema_step_workspace_bytes")
    return n.value


def xema_dit_step_fwd(cfg: BlockCfg, req: Request, tokens, weights: Sequence[BlockWeights],
                      plan: OffloadPlan, cond, chunk_tokens: int, workspace, workspace_bytes: int,
                      out, stream=None, copy_stream=None) -> None:
    arr = (BlockWeights * len(weights))(*weights)
    cs = None if copy_stream is None else (copy_stream if isinstance(copy_stream, int)
                                           else copy_stream.cuda_stream)
    _check(lib().xema_dit_step_fwd(ctypes.byref(cfg), ctypes.byref(req), _ptr(tokens), arr,
                                   ctypes.byref(plan), _ptr(cond), chunk_tokens, _ptr(workspace),
                                   int(workspace_bytes), _ptr(out), _stream(stream), cs),
           "xema_dit_step_fwd")


def step_costs(h2d_gbytes_per_s: float = 56.0, block_tflops: float = 1000.0) -> StepCosts:
    """The latency model's rates (defaults: one MI355X, measured)."""
    k = StepCosts()
    k.h2d_gbytes_per_s, k.block_tflops = h2d_gbytes_per_s, block_tflops
    return k


def xema_step_plan_fixed(cfg: BlockCfg, req: Request, n_blocks: int, n_offloaded: int, n_staging: int,
                         batch_group: int, chunk_tokens: int, costs: Optional[StepCosts] = None) -> StepPlan:
    p = StepPlan()
    _check(lib().xema_step_plan_fixed(ctypes.byref(cfg), ctypes.byref(req), n_blocks, n_offloaded, n_staging,
                                      batch_group, chunk_tokens, ctypes.byref(costs or step_costs()),
                                      ctypes.byref(p)), "xema_step_plan_fixed")
    return p


def xema_step_plan_budget(cfg: BlockCfg, req: Request, n_blocks: int, n_staging: int, device_budget_bytes: int,
                          costs: Optional[StepCosts] = None) -> StepPlan:
    """Raises XemaError (XEMA_ERR_BUDGET_TOO_SMALL, the plan with the least
    device_bytes as `.plan`) when nothing fits."""
    p = StepPlan()
    st = lib().xema_step_plan_budget(ctypes.byref(cfg), ctypes.byref(req), n_blocks, n_staging,
                                     int(device_budget_bytes), ctypes.byref(costs or step_costs()), ctypes.byref(p))
    if st != XEMA_OK:
        e = XemaError(st, "xema_step_plan_budget")
        e.plan = p
        raise e
    return p


def xema_dit_step_fwd_planned(cfg: BlockCfg, req: Request, tokens, weights: Sequence[BlockWeights],
                              plan: StepPlan, cond, workspace, workspace_bytes: int, out, stream=None,
                              copy_stream=None) -> None:
    arr = (BlockWeights * len(weights))(*weights)
    cs = None if copy_stream is None else (copy_stream if isinstance(copy_stream, int)
                                           else copy_stream.cuda_stream)
    _check(lib().xema_dit_step_fwd_planned(ctypes.byref(cfg), ctypes.byref(req), _ptr(tokens), arr,
                                           ctypes.byref(plan), _ptr(cond), _ptr(workspace), int(workspace_bytes),
                                           _ptr(out), _stream(stream), cs), "xema_dit_step_fwd_planned")


# -- the VAE decoder's fused upsampling stage (include/xema_vae.h) -------------------------------


def xema_vae_upconv_weight_bytes(ci: int, co: int) -> int:
    n = _I64()
    _check(lib().xema_vae_upconv_weight_bytes(ci, co, ctypes.byref(n)), "xema_vae_upconv_weight_bytes")
    return n.value


def xema_vae_upconv_prepare(w, ci: int, co: int, wp, stream=None) -> None:
    _check(lib().xema_vae_upconv_prepare(_ptr(w), ci, co, _ptr(wp), _stream(stream)),
           "xema_vae_upconv_prepare")


def xema_vae_upconv(x, n: int, h: int, w: int, ci: int, wp, bias, co: int, row_begin: int,
                    row_count: int, y, stream=None) -> None:
    _check(lib().xema_vae_upconv(_ptr(x), n, h, w, ci, _ptr(wp), _ptr(bias), co, row_begin, row_count,
                                 _ptr(y), _stream(stream)), "xema_vae_upconv")
