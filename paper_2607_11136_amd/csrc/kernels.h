// Launch functions of the gfx950 kernels (host-callable, asynchronous).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attention.h"
#include "xema_ops.h"

namespace xema {

struct RowMap {
  int64_t rows_per_batch, batch_stride, row_offset;
};

// Which modulation vector a row of a dual-stream block takes: a row whose
// sequence position (pos_offset + its index within the batch element's rows)
// is below text_len reads the text tokens' vectors, text_delta floats past the
// visual ones.  A single-stream block passes text_delta = 0.
struct ModSel {
  int64_t pos_offset, text_len, text_delta;
};

struct RopeGeom {
  int grid[3];  // (G_t, G_h, G_w)
  int dims[3];  // (d_t, d_h, d_w)
};

struct QkRopeArgs {
  const _Float16* qkv;
  const uint16_t* q_gamma;
  const uint16_t* k_gamma;
  const float2* table;
  _Float16* q;
  _Float16* k;
  _Float16* vt;
  int batch, heads, text_len, padded_len;
  int tok_begin, tok_count, count_ext;  // count_ext adds the zeroed padding tokens
  float qk_eps;
  float q_scale;  // log2(e) / sqrt(head_dim), folded into the stored queries
  RopeGeom geom;
};

struct GemmParams {
  int dtype;  // XEMA_BF16 / XEMA_F16 operands
  const void* a;
  const void* b;
  int64_t M;
  int N, K;
  const uint16_t* bias;
  int epilogue;
  void* c;
  int c_dtype;
  RowMap c_map;
  int64_t ldc;
  const void* resid;
  int resid_dtype;
  RowMap resid_map;
  int64_t ld_resid;
  const float* gate;
  int64_t gate_stride;
  ModSel gate_sel;  // per-row choice of the gate vector (positions within c_map's rows)
  QkRopeArgs qk;    // EPI_QKV_HEADS: rows are tokens [qk.tok_begin, +c_map.rows_per_batch)
  uint32_t* status; // range flag set when an fp16 output leaves the fp16 range (may be null)
};

// Internal epilogues of the QKV GEMM (steps a2 + a3 in one kernel): bias,
// QK-RMSNorm, 3D RoPE and the scatter into Q, K and V^T, without the
// [tokens, 3D] intermediate, at head_dim 64 and 128.  Not accepted by
// xema_op_gemm.
constexpr int EPI_QKV_HEADS = 3;
constexpr int EPI_QKV_HEADS_128 = 4;

// The VAE decoder's fused upsampling stage (k_upconv.hip).
struct UpconvParams {
  const uint16_t* x;     // bf16 [n, h, w, ci]
  const uint16_t* wp;    // bf16 phase-summed weights [4][co][4][ci]
  const uint16_t* bias;  // bf16 [co]
  uint16_t* y;           // bf16 [n, 2h, 2w, co]
  int n, h, w, ci, co;
  int row_begin, row_count;  // source rows computed; output rows 2*row_begin ..
};

hipError_t launch_upconv_prep(const uint16_t* w, int ci, int co, uint16_t* wp, hipStream_t s);
hipError_t launch_upconv(const UpconvParams& p, hipStream_t s);

// status_clear (may be null): XEMA_STATUS_WORDS range flags zeroed by the launch.
hipError_t launch_adaln(const uint16_t* cond, const uint16_t* w, const uint16_t* bias, int batch,
                        int cond_dim, int out_dim, float* mod, hipStream_t s,
                        uint32_t* status_clear = nullptr);
// status (may be null): set when an fp16 output leaves the fp16 range.
hipError_t launch_ln_modulate(const void* x, int x_dtype, RowMap m, int64_t rows, int dim,
                              const float* shift, const float* scale, int64_t mod_stride,
                              ModSel sel, float eps, void* y, int y_dtype, hipStream_t s,
                              uint32_t* status = nullptr);
hipError_t launch_rope_table(RopeGeom g, float theta, float* table, hipStream_t s);
hipError_t launch_qk_norm_rope(const QkRopeArgs& a, int head_dim, hipStream_t s);
// Zeros for the padding tokens [L, Lp) of Q, K and V^T (all batch rows, heads).
hipError_t launch_qkv_pad(const QkRopeArgs& a, int head_dim, int seq_len, hipStream_t s);
// status (may be null): set when a converted value leaves the fp16 range.
hipError_t launch_convert_f16(const uint16_t* src, _Float16* dst, int64_t n, hipStream_t s,
                              uint32_t* status = nullptr);
hipError_t launch_gemm(const GemmParams& p, hipStream_t s);

}  // namespace xema
