// Host driver of libxema: argument validation, the per-step entry points of
// xema_ops.h and the chunked block forward of xema.h.
//
// xema_dit_block_fwd runs the block in two phases over token chunks, the
// "only as much as needed" chunking of Sec. 5.1 applied around DiT attention
// (Sec. 5.2, "Localized chunking and fusion"):
//   step 0   AdaLN map (a0; two maps for a dual-stream block) and the RoPE
//            table, once per call
//   phase A  for each chunk of c tokens: LN1 (a1) -> QKV GEMM (a2) ->
//            QK-RMSNorm + RoPE scatter (a3), filling Q, K, V^T for all tokens
//            (a2 and a3 are one kernel)
//   step 4   fp16 copies of W_o, W_up, W_down
//   phase B  for each chunk of c queries: attention over all keys (a4) ->
//            out-projection + gated residual (a5) -> LN2 (a6) -> MLP up +
//            GELU (a7) -> MLP down + gated residual into `out` (a8)
// Every intermediate lives in the caller's arena at the offsets Algorithm 1
// (Sec. 6.1) assigned to its slot, so runtime allocation is the table lookup
// of Sec. 8 ("Static memory runtime").
#include <algorithm>
#include <cmath>
#include <cstring>

#include "kernels.h"
#include "xema_internal.h"

using namespace xema;

namespace {

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool overlaps(const void* a, int64_t an, const void* b, int64_t bn) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)bn && b0 < a0 + (uintptr_t)an;
}

int hip_status(hipError_t e) { return e == hipSuccess ? XEMA_OK : XEMA_ERR_HIP; }

RowMap to_map(const xema_rowmap& m) { return RowMap{m.rows_per_batch, m.batch_stride, m.row_offset}; }

RopeGeom geom_of(const xema_block_cfg& c, const xema_request& r) {
  RopeGeom g;
  g.grid[0] = r.grid_t; g.grid[1] = r.grid_h; g.grid[2] = r.grid_w;
  for (int a = 0; a < 3; ++a) g.dims[a] = c.rope_dims[a];
  return g;
}

}  // namespace

// ---------------------------------------------------------------------------
// per-step entry points
// ---------------------------------------------------------------------------

extern "C" int xema_op_adaln(const void* cond, const void* w, const void* bias, int32_t batch,
                             int32_t cond_dim, int32_t out_dim, float* mod, void* stream) {
  if (!cond || !w || !bias || !mod || batch <= 0 || cond_dim <= 0 || out_dim <= 0)
    return XEMA_ERR_INVALID_ARG;
  if (cond_dim % 8) return XEMA_ERR_UNSUPPORTED;
  if (!aligned(cond, 16) || !aligned(w, 16) || !aligned(bias, 2) || !aligned(mod, 4))
    return XEMA_ERR_MISALIGNED;
  return hip_status(launch_adaln((const uint16_t*)cond, (const uint16_t*)w,
                                 (const uint16_t*)bias, batch, cond_dim, out_dim, mod,
                                 (hipStream_t)stream));
}

extern "C" int xema_op_ln_modulate(const void* x, int32_t x_dtype, xema_rowmap xmap, int64_t rows,
                                   int32_t dim, const float* shift, const float* scale,
                                   int64_t mod_stride, float eps, void* y, int32_t y_dtype,
                                   void* stream) {
  if (!x || !shift || !scale || !y || rows < 0 || dim <= 0 || xmap.rows_per_batch <= 0 ||
      !(eps > 0.f))
    return XEMA_ERR_INVALID_ARG;
  if (dim % 256 || dim > 8192) return XEMA_ERR_UNSUPPORTED;
  if ((x_dtype != XEMA_BF16 && x_dtype != XEMA_F32) || (y_dtype != XEMA_BF16 && y_dtype != XEMA_F16))
    return XEMA_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(y, 16) || !aligned(shift, 16) || !aligned(scale, 16) ||
      mod_stride % 4)
    return XEMA_ERR_MISALIGNED;
  if (rows == 0) return XEMA_OK;
  return hip_status(launch_ln_modulate(x, x_dtype, to_map(xmap), rows, dim, shift, scale,
                                       mod_stride, ModSel{0, 0, 0}, eps, y, y_dtype,
                                       (hipStream_t)stream));
}

static int check_gemm(const xema_gemm_args* a) {
  if (!a || !a->a || !a->b || !a->bias || !a->c || a->M < 0 || a->N <= 0 || a->K <= 0 ||
      a->c_map.rows_per_batch <= 0 || a->ldc < a->N)
    return XEMA_ERR_INVALID_ARG;
  if (a->N % 256 || a->K % 64) return XEMA_ERR_UNSUPPORTED;
  if (a->dtype != XEMA_BF16 && a->dtype != XEMA_F16) return XEMA_ERR_UNSUPPORTED;
  if (a->M > ((int64_t)1 << 31) || (int64_t)256 * a->K * 2 >= ((int64_t)1 << 31))
    return XEMA_ERR_UNSUPPORTED;
  if (!aligned(a->a, 16) || !aligned(a->b, 16) || !aligned(a->bias, 8) || !aligned(a->c, 16) ||
      a->ldc % 8)
    return XEMA_ERR_MISALIGNED;
  switch (a->epilogue) {
    case XEMA_EPI_BIAS:
    case XEMA_EPI_BIAS_GELU:
      if (a->c_dtype != XEMA_BF16 && a->c_dtype != XEMA_F16) return XEMA_ERR_UNSUPPORTED;
      break;
    case XEMA_EPI_GATED_RESIDUAL:
      if (a->c_dtype != XEMA_F32) return XEMA_ERR_UNSUPPORTED;
      if (!a->resid || !a->gate || a->resid_map.rows_per_batch <= 0 || a->ld_resid < a->N)
        return XEMA_ERR_INVALID_ARG;
      if (a->resid_dtype != XEMA_BF16 && a->resid_dtype != XEMA_F32) return XEMA_ERR_UNSUPPORTED;
      if (!aligned(a->resid, 16) || !aligned(a->gate, 16) || a->ld_resid % 8 ||
          a->gate_stride % 4)
        return XEMA_ERR_MISALIGNED;
      break;
    default:
      return XEMA_ERR_INVALID_ARG;
  }
  return XEMA_OK;
}

static GemmParams to_params(const xema_gemm_args& a) {
  GemmParams p{};
  p.dtype = a.dtype; p.a = a.a; p.b = a.b; p.M = a.M; p.N = a.N; p.K = a.K;
  p.bias = (const uint16_t*)a.bias; p.epilogue = a.epilogue;
  p.c = a.c; p.c_dtype = a.c_dtype; p.c_map = to_map(a.c_map); p.ldc = a.ldc;
  p.resid = a.resid; p.resid_dtype = a.resid_dtype; p.resid_map = to_map(a.resid_map);
  p.ld_resid = a.ld_resid; p.gate = a.gate; p.gate_stride = a.gate_stride;
  p.gate_sel = ModSel{0, 0, 0};
  p.status = nullptr;
  return p;
}

extern "C" int xema_op_gemm(const xema_gemm_args* args, void* stream) {
  const int st = check_gemm(args);
  if (st != XEMA_OK) return st;
  if (args->M == 0) return XEMA_OK;
  return hip_status(launch_gemm(to_params(*args), (hipStream_t)stream));
}

extern "C" int xema_op_rope_table(const xema_block_cfg* cfg, const xema_request* req,
                                  float* table, void* stream) {
  const int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  if (!table) return XEMA_ERR_INVALID_ARG;
  if (!aligned(table, 8)) return XEMA_ERR_MISALIGNED;
  return hip_status(launch_rope_table(geom_of(*cfg, *req), cfg->rope_theta, table,
                                      (hipStream_t)stream));
}

static QkRopeArgs qk_args(const xema_block_cfg& cfg, const xema_request& req, const void* qkv,
                          int tok_begin, int tok_count, const void* q_gamma, const void* k_gamma,
                          const float* table, void* q, void* k, void* vt) {
  const int64_t L = seq_len(req), Lp = padded_len(L);
  QkRopeArgs a;
  a.qkv = (const _Float16*)qkv;
  a.q_gamma = (const uint16_t*)q_gamma;
  a.k_gamma = (const uint16_t*)k_gamma;
  a.table = (const float2*)table;
  a.q = (_Float16*)q; a.k = (_Float16*)k; a.vt = (_Float16*)vt;
  a.batch = req.batch; a.heads = cfg.heads; a.text_len = req.text_len; a.padded_len = (int)Lp;
  a.tok_begin = tok_begin; a.tok_count = tok_count;
  a.count_ext = tok_count + ((int64_t)tok_begin + tok_count == L ? (int)(Lp - L) : 0);
  a.qk_eps = cfg.qk_eps;
  a.q_scale = (float)(1.4426950408889634 / std::sqrt((double)cfg.head_dim));
  a.geom = geom_of(cfg, req);
  return a;
}

extern "C" int xema_op_qk_norm_rope(const xema_block_cfg* cfg, const xema_request* req,
                                    const void* qkv, int32_t tok_begin, int32_t tok_count,
                                    const void* q_gamma, const void* k_gamma, const float* table,
                                    void* q, void* k, void* vt, void* stream) {
  const int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  const int64_t L = seq_len(*req);
  if (!qkv || !q_gamma || !k_gamma || !q || !k || !vt || tok_begin < 0 || tok_count <= 0 ||
      (int64_t)tok_begin + tok_count > L)
    return XEMA_ERR_INVALID_ARG;
  const int rot = cfg->rope_dims[0] + cfg->rope_dims[1] + cfg->rope_dims[2];
  if (rot > 0 && !table) return XEMA_ERR_INVALID_ARG;
  if (!aligned(qkv, 16) || !aligned(q_gamma, 16) || !aligned(k_gamma, 16) || !aligned(q, 16) ||
      !aligned(k, 16) || !aligned(vt, 16) || (table && !aligned(table, 8)))
    return XEMA_ERR_MISALIGNED;
  const QkRopeArgs a = qk_args(*cfg, *req, qkv, tok_begin, tok_count, q_gamma, k_gamma, table, q,
                               k, vt);
  return hip_status(launch_qk_norm_rope(a, cfg->head_dim, (hipStream_t)stream));
}

extern "C" int xema_op_attention(const void* q, const void* k, const void* vt, int32_t batch,
                                 int32_t heads, int32_t head_dim, int32_t seq_len_,
                                 int32_t padded_len_, int32_t q_begin, int32_t q_count, void* o,
                                 void* stream) {
  if (!q || !k || !vt || !o || batch <= 0 || heads <= 0 || seq_len_ <= 0 || q_begin < 0 ||
      q_count <= 0 || (int64_t)q_begin + q_count > seq_len_ || padded_len_ < seq_len_)
    return XEMA_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return XEMA_ERR_UNSUPPORTED;
  if (padded_len_ % XEMA_SEQ_PAD) return XEMA_ERR_UNSUPPORTED;
  if ((int64_t)padded_len_ * head_dim * 2 >= ((int64_t)1 << 31)) return XEMA_ERR_UNSUPPORTED;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(vt, 16) || !aligned(o, 16))
    return XEMA_ERR_MISALIGNED;
  AttnParams p;
  p.q = (const _Float16*)q; p.k = (const _Float16*)k; p.vt = (const _Float16*)vt;
  p.o = (_Float16*)o;
  p.batch = batch; p.heads = heads; p.seq_len = seq_len_; p.padded_len = padded_len_;
  p.q_begin = q_begin; p.q_count = q_count;
  return hip_status(launch_attention(p, head_dim, (hipStream_t)stream));
}

extern "C" int xema_op_convert_f16(const void* src, void* dst, int64_t n, void* stream) {
  if (!src || !dst || n < 0) return XEMA_ERR_INVALID_ARG;
  if (n % 8) return XEMA_ERR_UNSUPPORTED;
  if (!aligned(src, 16) || !aligned(dst, 16)) return XEMA_ERR_MISALIGNED;
  if (overlaps(src, n * 2, dst, n * 2)) return XEMA_ERR_INVALID_ARG;
  return hip_status(launch_convert_f16((const uint16_t*)src, (_Float16*)dst, n,
                                       (hipStream_t)stream));
}

// ---------------------------------------------------------------------------
// the block forward
// ---------------------------------------------------------------------------

namespace xema {

// The block's launches on stream s, arguments already validated: x is
// [B, L, D] bf16 or fp32 (x_dtype), the arena at ws follows `plan` for chunk
// ch, out is [B, L, D] fp32.
int run_block(const xema_block_cfg& c, const xema_request& r, const void* tokens, int x_dtype,
              const xema_block_weights& w, const void* cond, int64_t ch, uint8_t* ws,
              const xema_plan& plan, float* out, hipStream_t s, hipStream_t aux, bool clear_status) {
  const int64_t B = r.batch, L = seq_len(r), D = c.hidden, F = c.mlp_hidden, Dc = c.cond_dim;
  const int64_t Lp = padded_len(L);
  auto slot = [&](int id) { return (void*)(ws + plan.slot_offset[id]); };
  float* mod = (float*)slot(XEMA_SLOT_MOD);
  float* rope = (float*)slot(XEMA_SLOT_ROPE);
  void* Q = slot(XEMA_SLOT_Q);
  void* Kk = slot(XEMA_SLOT_K);
  void* VT = slot(XEMA_SLOT_VT);
  void* ln1 = slot(XEMA_SLOT_LN1);
  void* qkv = slot(XEMA_SLOT_QKV);  // empty: the QKV GEMM writes the heads itself
  // fp16 phase-B weights: the caller's (cfg.weights_f16) or this call's copies
  const bool copy_w = c.weights_f16 == 0;
  const void* wo16 = copy_w ? slot(XEMA_SLOT_WO16) : w.o_w;
  const void* wup16 = copy_w ? slot(XEMA_SLOT_WUP16) : w.up_w;
  const void* wdown16 = copy_w ? slot(XEMA_SLOT_WDOWN16) : w.down_w;
  uint32_t* status = (uint32_t*)slot(XEMA_SLOT_STATUS);  // range flags, one word per kind
  void* attn = slot(XEMA_SLOT_ATTN);
  float* x1 = (float*)slot(XEMA_SLOT_X1);
  void* ln2 = slot(XEMA_SLOT_LN2);
  void* hid = slot(XEMA_SLOT_HID);
  const RopeGeom geom = geom_of(c, r);

#define XEMA_TRY(expr)                          \
  do {                                          \
    if ((expr) != hipSuccess) return XEMA_ERR_HIP; \
  } while (0)

  // A dual-stream block keeps the text tokens' modulation right after the
  // visual tokens' in the mod slot; rows pick theirs by sequence position.
  const int64_t txt_delta = dual_stream(c) ? B * 6 * D : 0;
  auto sel_at = [&](int64_t t0) { return ModSel{t0, r.text_len, txt_delta}; };

  // step 0 (the first launch of a call also clears the range flags)
  XEMA_TRY(launch_adaln((const uint16_t*)cond, (const uint16_t*)w.ada_w,
                        (const uint16_t*)w.ada_b, (int)B, (int)Dc, (int)(6 * D), mod, s,
                        clear_status ? status : nullptr));
  if (dual_stream(c))
    XEMA_TRY(launch_adaln((const uint16_t*)cond, (const uint16_t*)w.ada_txt_w,
                          (const uint16_t*)w.ada_txt_b, (int)B, (int)Dc, (int)(6 * D),
                          mod + txt_delta, s));
  XEMA_TRY(launch_rope_table(geom, c.rope_theta, rope, s));

  // phase A: LN1 -> QKV -> QK-norm/RoPE scatter, per token chunk.  The QKV
  // GEMM's epilogue does the scatter itself (a head per wave at head dim 64,
  // per two waves at 128; the shape checks admit only these), so the qkv
  // slot stays empty; the padding tokens are zeroed once.
  for (int64_t t0 = 0; t0 < L; t0 += ch) {
    const int64_t cc = std::min(ch, L - t0);
    const RowMap xmap{cc, L, t0};
    XEMA_TRY(launch_ln_modulate(tokens, x_dtype, xmap, B * cc, (int)D, mod, mod + D, 6 * D,
                                sel_at(t0), c.ln_eps, ln1, XEMA_BF16, s));
    const QkRopeArgs qa = qk_args(c, r, qkv, (int)t0, (int)cc, w.q_gamma, w.k_gamma, rope, Q, Kk, VT);
    GemmParams g{};
    g.dtype = XEMA_BF16; g.a = ln1; g.b = w.qkv_w; g.M = B * cc; g.N = (int)(3 * D); g.K = (int)D;
    g.bias = (const uint16_t*)w.qkv_b;
    g.epilogue = c.head_dim == 64 ? EPI_QKV_HEADS : EPI_QKV_HEADS_128;
    g.c = qkv; g.c_dtype = XEMA_F16; g.c_map = RowMap{cc, cc, 0}; g.ldc = 3 * D;
    g.qk = qa;
    g.status = status + 0;
    XEMA_TRY(launch_gemm(g, s));
  }
  XEMA_TRY(launch_qkv_pad(qk_args(c, r, qkv, 0, 0, w.q_gamma, w.k_gamma, rope, Q, Kk, VT),
                          c.head_dim, (int)L, s));

  // step 4: fp16 copies of the phase-B weights, unless the caller passed them
  if (copy_w) {
    XEMA_TRY(launch_convert_f16((const uint16_t*)w.o_w, (_Float16*)wo16, D * D, s, status + 3));
    XEMA_TRY(launch_convert_f16((const uint16_t*)w.up_w, (_Float16*)wup16, F * D, s, status + 3));
    XEMA_TRY(launch_convert_f16((const uint16_t*)w.down_w, (_Float16*)wdown16, D * F, s, status + 3));
  }

  // phase B: attention -> out-proj -> LN2 -> MLP, per query chunk
  auto attention_of = [&](int64_t t0, void* dst, hipStream_t q) {
    AttnParams ap;
    ap.q = (const _Float16*)Q; ap.k = (const _Float16*)Kk; ap.vt = (const _Float16*)VT;
    ap.o = (_Float16*)dst; ap.batch = (int)B; ap.heads = c.heads; ap.seq_len = (int)L;
    ap.padded_len = (int)Lp; ap.q_begin = (int)t0; ap.q_count = (int)std::min(ch, L - t0);
    return launch_attention(ap, c.head_dim, q);
  };
  // the out-projection of the chunk at t0 (reading attention output src),
  // then `used` (if any) is recorded, then LN2 and the MLP
  auto projections_of = [&](int64_t t0, const void* src, hipEvent_t used) {
    const int64_t cc = std::min(ch, L - t0);
    const RowMap ident{cc, cc, 0};
    GemmParams g{};
    g.dtype = XEMA_F16; g.a = src; g.b = wo16; g.M = B * cc; g.N = (int)D; g.K = (int)D;
    g.bias = (const uint16_t*)w.o_b; g.epilogue = XEMA_EPI_GATED_RESIDUAL;
    g.c = x1; g.c_dtype = XEMA_F32; g.c_map = ident; g.ldc = D;
    g.resid = tokens; g.resid_dtype = x_dtype; g.resid_map = RowMap{cc, L, t0}; g.ld_resid = D;
    g.gate = mod + 2 * D; g.gate_stride = 6 * D; g.gate_sel = sel_at(t0);
    if (launch_gemm(g, s) != hipSuccess) return hipErrorLaunchFailure;
    if (used && hipEventRecord(used, s) != hipSuccess) return hipErrorLaunchFailure;

    hipError_t e = launch_ln_modulate(x1, XEMA_F32, ident, B * cc, (int)D, mod + 3 * D, mod + 4 * D,
                                      6 * D, sel_at(t0), c.ln_eps, ln2, XEMA_F16, s, status + 1);
    if (e != hipSuccess) return e;

    GemmParams u{};
    u.dtype = XEMA_F16; u.a = ln2; u.b = wup16; u.M = B * cc; u.N = (int)F; u.K = (int)D;
    u.bias = (const uint16_t*)w.up_b; u.epilogue = XEMA_EPI_BIAS_GELU;
    u.c = hid; u.c_dtype = XEMA_F16; u.c_map = ident; u.ldc = F;
    u.status = status + 2;
    if ((e = launch_gemm(u, s)) != hipSuccess) return e;

    GemmParams d{};
    d.dtype = XEMA_F16; d.a = hid; d.b = wdown16; d.M = B * cc; d.N = (int)D; d.K = (int)F;
    d.bias = (const uint16_t*)w.down_b; d.epilogue = XEMA_EPI_GATED_RESIDUAL;
    d.c = out; d.c_dtype = XEMA_F32; d.c_map = RowMap{cc, L, t0}; d.ldc = D;
    d.resid = x1; d.resid_dtype = XEMA_F32; d.resid_map = ident; d.ld_resid = D;
    d.gate = mod + 5 * D; d.gate_stride = 6 * D; d.gate_sel = sel_at(t0);
    return launch_gemm(d, s);
  };

  const int64_t n_chunks = (L + ch - 1) / ch;
  if (!aux || aux == s || n_chunks < 2) {
    for (int64_t t0 = 0; t0 < L; t0 += ch) {
      XEMA_TRY(attention_of(t0, attn, s));
      XEMA_TRY(projections_of(t0, attn, nullptr));
    }
    return XEMA_OK;
  }

  // Two streams: the attention of chunk k runs on `aux` once the
  // out-projection of chunk k-1 has read the attention buffer, alongside the
  // LN2 and MLP of chunk k-1 on `s`; one kernel's last, partly filled round
  // overlaps the other's.  (The chunked layout keeps the attention buffer
  // apart from x1, LN2 and the MLP's hidden buffer.)  Every operation and its
  // inputs are those of the one-stream order, so the output is the same bit
  // for bit.
  hipEvent_t ev[3] = {};  // phase A done, attention done, buffer read
  int made = 0;
  auto finish = [&](int status) {
    for (int i = 0; i < made; ++i) (void)hipEventDestroy(ev[i]);  // released once complete
    return status;
  };
  for (; made < 3; ++made)
    if (hipEventCreateWithFlags(&ev[made], hipEventDisableTiming) != hipSuccess) return finish(XEMA_ERR_HIP);
  if (hipEventRecord(ev[0], s) != hipSuccess || hipStreamWaitEvent(aux, ev[0], 0) != hipSuccess)
    return finish(XEMA_ERR_HIP);
  for (int64_t k = 0; k < n_chunks; ++k) {
    const int64_t t0 = k * ch;
    if (k > 0 && hipStreamWaitEvent(aux, ev[2], 0) != hipSuccess) return finish(XEMA_ERR_HIP);
    if (attention_of(t0, attn, aux) != hipSuccess || hipEventRecord(ev[1], aux) != hipSuccess ||
        hipStreamWaitEvent(s, ev[1], 0) != hipSuccess)
      return finish(XEMA_ERR_HIP);
    if (projections_of(t0, attn, ev[2]) != hipSuccess) return finish(XEMA_ERR_HIP);
  }
  return finish(XEMA_OK);
#undef XEMA_TRY
  return XEMA_OK;
}

}  // namespace xema


// Validation shared by the block entry points: everything but the arena
// size, which depends on the group size.
static int check_block_call(const xema_block_cfg* cfg, const xema_request* req, const void* tokens,
                            const xema_block_weights* w, const void* cond, void* workspace,
                            int64_t workspace_bytes, void* out) {
  int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  if (!tokens || !w || !cond || !workspace || !out || workspace_bytes <= 0)
    return XEMA_ERR_INVALID_ARG;
  const xema_block_cfg& c = *cfg;
  int64_t wbytes[kWeightTensors];
  block_weight_sizes(c, wbytes);  // size 0: a tensor the block does not use
  const void* const* wp = weight_ptrs(*w);
  for (int i = 0; i < kWeightTensors; ++i)
    if (wbytes[i] && !wp[i]) return XEMA_ERR_INVALID_ARG;
  for (int i = 0; i < kWeightTensors; ++i)
    if (wbytes[i] && !aligned(wp[i], 16)) return XEMA_ERR_MISALIGNED;
  if (!aligned(tokens, 16) || !aligned(cond, 16) || !aligned(out, 16)) return XEMA_ERR_MISALIGNED;
  if (!aligned(workspace, 256)) return XEMA_ERR_MISALIGNED;

  const xema_request& r = *req;
  const int64_t B = r.batch, L = seq_len(r), D = c.hidden, Dc = c.cond_dim;
  const int64_t out_bytes = B * L * D * 4;
  // out is written while everything else is read: it must overlap nothing
  if (overlaps(out, out_bytes, tokens, B * L * D * 2) ||
      overlaps(out, out_bytes, cond, B * Dc * 2) ||
      overlaps(out, out_bytes, workspace, workspace_bytes))
    return XEMA_ERR_INVALID_ARG;
  for (int i = 0; i < kWeightTensors; ++i)
    if (wbytes[i] && overlaps(out, out_bytes, wp[i], wbytes[i])) return XEMA_ERR_INVALID_ARG;
  // inputs must not live inside the arena the block writes
  if (overlaps(workspace, workspace_bytes, tokens, B * L * D * 2) ||
      overlaps(workspace, workspace_bytes, cond, B * Dc * 2))
    return XEMA_ERR_INVALID_ARG;
  for (int i = 0; i < kWeightTensors; ++i)
    if (wbytes[i] && overlaps(workspace, workspace_bytes, wp[i], wbytes[i]))
      return XEMA_ERR_INVALID_ARG;
  return XEMA_OK;
}

int xema::block_fwd(const xema_block_cfg* cfg, const xema_request* req, const void* tokens,
                    const xema_block_weights* w, const void* cond, int32_t batch_group,
                    int32_t chunk_tokens, void* workspace, int64_t workspace_bytes, void* out,
                    void* stream, void* aux_stream) {
  int st = check_block_call(cfg, req, tokens, w, cond, workspace, workspace_bytes, out);
  if (st != XEMA_OK) return st;
  if (batch_group < 1) return XEMA_ERR_INVALID_ARG;
  const xema_block_cfg& c = *cfg;
  const int64_t B = req->batch, L = seq_len(*req), D = c.hidden, Dc = c.cond_dim;
  const int64_t g = std::min<int64_t>(batch_group, B);
  const int64_t ch = effective_chunk(L, chunk_tokens);
  // groups of g sequences, one after another; a shorter last group runs with
  // the layout of its own request.  Both layouts are checked before any launch.
  xema_request rg = *req, rl = *req;
  rg.batch = (int32_t)g;
  rl.batch = (int32_t)(B % g == 0 ? g : B % g);
  xema_plan plan_g, plan_l;
  st = layout_for_chunk(c, rg, ch, &plan_g);
  if (st != XEMA_OK) return st;
  st = layout_for_chunk(c, rl, ch, &plan_l);
  if (st != XEMA_OK) return st;
  if (workspace_bytes < plan_g.workspace_bytes || workspace_bytes < plan_l.workspace_bytes)
    return XEMA_ERR_WORKSPACE_TOO_SMALL;
  for (int64_t b0 = 0; b0 < B; b0 += g) {
    const bool last = b0 + g >= B;
    st = run_block(c, last ? rl : rg, (const uint16_t*)tokens + b0 * L * D, XEMA_BF16, *w,
                   (const uint16_t*)cond + b0 * Dc, ch, (uint8_t*)workspace, last ? plan_l : plan_g,
                   (float*)out + b0 * L * D, (hipStream_t)stream, (hipStream_t)aux_stream, b0 == 0);
    if (st != XEMA_OK) return st;
  }
  return XEMA_OK;
}

extern "C" int xema_dit_block_fwd_serial(const xema_block_cfg* cfg, const xema_request* req,
                                         const void* tokens, const xema_block_weights* w,
                                         const void* cond, int32_t batch_group,
                                         int32_t chunk_tokens, void* workspace,
                                         int64_t workspace_bytes, void* out, void* stream) {
  return block_fwd(cfg, req, tokens, w, cond, batch_group, chunk_tokens, workspace, workspace_bytes, out,
                   stream, nullptr);
}

extern "C" int xema_dit_block_fwd(const xema_block_cfg* cfg, const xema_request* req,
                                  const void* tokens, const xema_block_weights* w,
                                  const void* cond, int32_t chunk_tokens, void* workspace,
                                  int64_t workspace_bytes, void* out, void* stream) {
  return block_fwd(cfg, req, tokens, w, cond, req ? req->batch : 1, chunk_tokens, workspace,
                   workspace_bytes, out, stream, nullptr);
}

extern "C" int xema_block_status(const xema_plan* plan, const void* workspace, void* stream,
                                 uint32_t* flags) {
  if (!plan || !flags) return XEMA_ERR_INVALID_ARG;
  if (!workspace) {  // the static arena of xema_dit_block_fwd_static on this device
    void* a = nullptr;
    const int st = static_arena(&a);
    if (st != XEMA_OK) return st;
    workspace = a;
  }
  if (plan->n_slots <= XEMA_SLOT_STATUS || plan->slot_bytes[XEMA_SLOT_STATUS] < 4 * XEMA_STATUS_WORDS ||
      plan->slot_offset[XEMA_SLOT_STATUS] < 0)
    return XEMA_ERR_INVALID_ARG;
  uint32_t words[XEMA_STATUS_WORDS];
  const hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(words, (const uint8_t*)workspace + plan->slot_offset[XEMA_SLOT_STATUS],
                     sizeof(words), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return XEMA_ERR_HIP;
  uint32_t f = 0;
  for (int i = 0; i < XEMA_STATUS_WORDS; ++i)
    if (words[i]) f |= 1u << i;
  *flags = f;
  return f ? XEMA_ERR_RANGE : XEMA_OK;
}

extern "C" int xema_dit_block_fwd_pipelined(const xema_block_cfg* cfg, const xema_request* req,
                                            const void* tokens, const xema_block_weights* w,
                                            const void* cond, int32_t batch_group,
                                            int32_t chunk_tokens, void* workspace,
                                            int64_t workspace_bytes, void* out, void* stream,
                                            void* aux_stream) {
  return block_fwd(cfg, req, tokens, w, cond, batch_group, chunk_tokens, workspace, workspace_bytes, out,
                   stream, aux_stream);
}
