/*
 * xema_ops.h -- the individual steps of the DiT block forward as C entry
 * points (gfx950).  xema_dit_block_fwd (xema.h) chains exactly these launches;
 * they are exported so each step can be checked and timed on its own.
 *
 * Conventions are those of xema.h: status return, host-side validation before
 * any launch, caller-owned device buffers, no allocation, asynchronous on
 * `stream` (a hipStream_t, NULL = default stream), 16-byte aligned pointers.
 * Element types are given by xema_dtype codes.
 *
 * fp16 outputs (y of xema_op_ln_modulate and c of xema_op_gemm with
 * XEMA_F16, q, k and vt of xema_op_qk_norm_rope, o of xema_op_attention,
 * dst of xema_op_convert_f16) have the fp16 range of +-65504 that xema.h's
 * precision contract states: larger values round to +-inf.  These
 * single-step entry points do not check it (no range flags); the block
 * entry points of xema.h do, through xema_block_status.
 */
#ifndef XEMA_OPS_H_
#define XEMA_OPS_H_

#include <stdint.h>

#include "xema.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { XEMA_BF16 = 0, XEMA_F16 = 1, XEMA_F32 = 2 } xema_dtype;

/* Row map used for chunked access to [B, L, ...] tensors: GEMM/LN row r
 * (0 <= r < rows) belongs to batch element b = r / rows_per_batch and maps to
 * storage row  b * batch_stride + row_offset + (r - b * rows_per_batch).
 * The identity map is {rows_per_batch = rows, batch_stride = 0, row_offset = 0}. */
typedef struct {
  int64_t rows_per_batch, batch_stride, row_offset;
} xema_rowmap;

/* Step a0, AdaLN map (the block's conditioning, reading: no SiLU):
 *   mod[b][n] = sum_k w[n][k] cond[b][k] + bias[n]
 * cond bf16 [batch, cond_dim], w bf16 [out_dim, cond_dim], bias bf16 [out_dim],
 * mod fp32 [batch, out_dim].  Each row's dot product is summed in one fixed
 * order.  Requires cond_dim % 8 == 0.                                        */
XEMA_API int xema_op_adaln(const void* cond, const void* w, const void* bias, int32_t batch,
                  int32_t cond_dim, int32_t out_dim, float* mod, void* stream);

/* Steps a1 / a6, LayerNorm (no affine, biased variance, fp32 statistics) and
 * AdaLN modulation:
 *   y[r] = (x[map(r)] - mean) / sqrt(var + eps) * (1 + scale[b]) + shift[b]
 * x: x_dtype XEMA_BF16 or XEMA_F32, rows of `dim` elements at stride `dim`,
 * addressed through xmap; y: y_dtype XEMA_BF16 or XEMA_F16, [rows, dim]
 * contiguous; shift/scale fp32 with batch stride mod_stride (elements).
 * Requires dim % 256 == 0 and dim <= 8192.                                   */
XEMA_API int xema_op_ln_modulate(const void* x, int32_t x_dtype, xema_rowmap xmap, int64_t rows,
                        int32_t dim, const float* shift, const float* scale,
                        int64_t mod_stride, float eps, void* y, int32_t y_dtype,
                        void* stream);

typedef enum {
  XEMA_EPI_BIAS = 0,            /* c = acc + bias                       -> c_dtype */
  XEMA_EPI_BIAS_GELU = 1,       /* c = GELU_tanh(acc + bias)            -> c_dtype */
  XEMA_EPI_GATED_RESIDUAL = 2   /* c = resid + gate * (acc + bias)      -> fp32    */
} xema_epilogue;

/* Steps a2, a5, a7, a8: C = A B^T with an epilogue, fp32 accumulation on
 * MFMA.  A [M, K] and B [N, K] are row-major (both K-contiguous, B in
 * nn.Linear layout), element type `dtype` (XEMA_BF16 or XEMA_F16); bias is
 * bf16 [N].  Row r of C is stored at row c_map(r) with leading dimension ldc;
 * for XEMA_EPI_GATED_RESIDUAL, resid row resid_map(r) (resid_dtype XEMA_BF16
 * or XEMA_F32, leading dimension ld_resid) and gate fp32
 * gate[(r / c_map.rows_per_batch) * gate_stride + n] are read and C is fp32;
 * otherwise C has c_dtype XEMA_BF16 or XEMA_F16.  Each output element's
 * K-reduction order is fixed (ascending K tiles), independent of M and of the
 * row maps.  Requires N % 256 == 0 and K % 64 == 0.                          */
typedef struct {
  int32_t dtype;
  const void* a; int64_t M; int32_t K;
  const void* b; int32_t N;
  const void* bias;
  int32_t epilogue;
  void* c; int32_t c_dtype; xema_rowmap c_map; int64_t ldc;
  const void* resid; int32_t resid_dtype; xema_rowmap resid_map; int64_t ld_resid;
  const float* gate; int64_t gate_stride;
} xema_gemm_args;

XEMA_API int xema_op_gemm(const xema_gemm_args* args, void* stream);

/* RoPE cos/sin table (step 0): for axis a in (t, y, w), position p <
 * grid_a and pair j < rope_dims[a] / 2, entry (cos, sin) of
 * p * theta^(-2j / rope_dims[a]), computed in fp64 and stored as fp32 pairs,
 * axes concatenated in (t, y, w) order.  table must hold
 * 8 * sum_a grid_a * rope_dims[a] / 2 bytes.                                 */
XEMA_API int xema_op_rope_table(const xema_block_cfg* cfg, const xema_request* req, float* table,
                       void* stream);

/* Step a3, QK-RMSNorm + 3D RoPE + scatter into per-head storage, for tokens
 * [tok_begin, tok_begin + tok_count) of every sequence:
 *   qkv fp16 [batch * tok_count, 3D] (row b * tok_count + i is token
 *   tok_begin + i of sequence b), q_gamma / k_gamma bf16 [d], table as made
 *   by xema_op_rope_table;
 *   q, k fp16 [batch, H, Lp, d]; vt fp16 [batch, H, d, Lp] (V transposed),
 *   Lp = L rounded up to XEMA_SEQ_PAD.
 * k <- RoPE(k / sqrt(mean(k^2) + qk_eps) * k_gamma); q is normalised and
 * rotated the same way with q_gamma and then multiplied by log2(e)/sqrt(d),
 * the factor the attention softmax applies to every score (one fp16 rounding
 * of the product); v is copied.  When the range ends at L, the padding tokens
 * [L, Lp) of q, k, vt are zeroed.                                              */
XEMA_API int xema_op_qk_norm_rope(const xema_block_cfg* cfg, const xema_request* req, const void* qkv,
                         int32_t tok_begin, int32_t tok_count, const void* q_gamma,
                         const void* k_gamma, const float* table, void* q, void* k,
                         void* vt, void* stream);

/* Step a4, joint full self-attention (no mask) for queries
 * [q_begin, q_begin + q_count) of every (batch, head), over all L keys:
 *   o[b * q_count + i][h * d + e] = sum_j softmax_j(q_i . k_j / sqrt(d)) v_j[e]
 * given qs = q * log2(e)/sqrt(d) (as xema_op_qk_norm_rope stores it), i.e.
 * with weights 2^(qs_i . k_j) normalised over j.
 * qs, k fp16 [batch, heads, padded_len, d]; vt fp16 [batch, heads, d,
 * padded_len]; o fp16 [batch * q_count, heads * d].  padded_len must be a
 * multiple of XEMA_SEQ_PAD with seq_len <= padded_len, and the padding
 * columns of vt must be finite (xema_op_qk_norm_rope zeroes them).  Keys are
 * visited in one fixed ascending order; each query's result depends only on
 * that query and the keys.  head_dim 64 or 128.  The exponents qs_i . k_j
 * must stay below 2^16 in magnitude (the d = 64 kernel keeps its reference
 * max in fp16); RMS-normalised queries and keys are far inside that.        */
XEMA_API int xema_op_attention(const void* q, const void* k, const void* vt, int32_t batch,
                      int32_t heads, int32_t head_dim, int32_t seq_len, int32_t padded_len,
                      int32_t q_begin, int32_t q_count, void* o, void* stream);

/* Step 4: bf16 -> fp16 copy of n elements (round to nearest even; exact for
 * 2^-17 <= |x| <= 65504).  n % 8 == 0.                                       */
XEMA_API int xema_op_convert_f16(const void* src, void* dst, int64_t n, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* XEMA_OPS_H_ */
