// HBM-bound kernels of the DiT block for gfx950: AdaLN map (a0), LayerNorm +
// modulation (a1, a6), RoPE table (step 0), QK-RMSNorm + RoPE + per-head
// scatter (a3) and the bf16 -> fp16 weight copy (step 4).
//
// Every reduction here has one fixed order per output (lane-strided partial
// sums followed by a butterfly), so a row's result never depends on which
// chunk, workgroup or position it is processed in.
#include "device_common.h"
#include "kernels.h"

#include <algorithm>

namespace xema {

// ---------------------------------------------------------------------------
// a0: mod[b][n] = sum_k w[n][k] cond[b][k] + bias[n].  One wave per output row
// n; each lane reads 16-byte slices of the row; up to 8 batch rows per pass.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_adaln(const uint16_t* __restrict__ cond,
                                               const uint16_t* __restrict__ w,
                                               const uint16_t* __restrict__ bias, int batch,
                                               int cond_dim, int out_dim,
                                               float* __restrict__ mod,
                                               uint32_t* __restrict__ status_clear) {
  const int lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  // the block's range flags start clear (the first launch of every call)
  if (status_clear != nullptr && blockIdx.x == 0 && threadIdx.x < XEMA_STATUS_WORDS)
    status_clear[threadIdx.x] = 0u;
  if (n >= out_dim) return;
  const uint16_t* wrow = w + n * cond_dim;
  const float bn = bf16_bits_to_f32(bias[n]);
  for (int b0 = 0; b0 < batch; b0 += 8) {
    const int nb = min(8, batch - b0);
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    // four 16-byte weight slices in flight per lane before their FMAs
    for (int k0 = lane * 8; k0 < cond_dim; k0 += 4 * 512) {
      u32x4 wv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (k0 + u * 512 < cond_dim) wv[u] = *reinterpret_cast<const u32x4*>(wrow + k0 + u * 512);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = k0 + u * 512;
        if (k >= cond_dim) break;
        float wf[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          wf[2 * e] = __uint_as_float(wv[u][e] << 16);
          wf[2 * e + 1] = __uint_as_float(wv[u][e] & 0xffff0000u);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (i < nb) {
            const u32x4 cv =
                *reinterpret_cast<const u32x4*>(cond + (int64_t)(b0 + i) * cond_dim + k);
            float s = acc[i];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              s = fmaf(wf[2 * e], __uint_as_float(cv[e] << 16), s);
              s = fmaf(wf[2 * e + 1], __uint_as_float(cv[e] & 0xffff0000u), s);
            }
            acc[i] = s;
          }
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i < nb) {
        const float s = wave_sum(acc[i]);
        if (lane == 0) mod[(int64_t)(b0 + i) * out_dim + n] = s + bn;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// a1 / a6: LayerNorm + AdaLN modulation.  One wave per row; lane l owns
// elements [s*64*E + E*l, s*64*E + E*l + E) for s = 0 .. dim/(64 E) - 1:
// E = 8 for 16-bit rows whose width 512 divides (16-byte loads), else E = 4
// (fp32 rows keep each load instruction on one contiguous KiB).  A row
// of a dual-stream block picks its shift/scale by its sequence position
// (ModSel).
// ---------------------------------------------------------------------------
template <typename XT>
__device__ __forceinline__ void load4(const XT* p, float v[4]);
template <>
__device__ __forceinline__ void load4<uint16_t>(const uint16_t* p, float v[4]) {
  const u32x2 u = *reinterpret_cast<const u32x2*>(p);
  v[0] = __uint_as_float(u[0] << 16);
  v[1] = __uint_as_float(u[0] & 0xffff0000u);
  v[2] = __uint_as_float(u[1] << 16);
  v[3] = __uint_as_float(u[1] & 0xffff0000u);
}
template <>
__device__ __forceinline__ void load4<float>(const float* p, float v[4]) {
  const f32x4 u = *reinterpret_cast<const f32x4*>(p);
  v[0] = u[0]; v[1] = u[1]; v[2] = u[2]; v[3] = u[3];
}

template <typename YT>
__device__ __forceinline__ void store4(YT* p, const float v[4]) {
  typedef YT y4 __attribute__((ext_vector_type(4)));
  y4 o;
  o[0] = from_f32<YT>(v[0]); o[1] = from_f32<YT>(v[1]);
  o[2] = from_f32<YT>(v[2]); o[3] = from_f32<YT>(v[3]);
  *reinterpret_cast<y4*>(p) = o;
}

// E consecutive elements (E = 4 or 8) to and from fp32
template <typename XT, int E>
__device__ __forceinline__ void load_e(const XT* p, float (&v)[E]) {
  if constexpr (E == 8 && sizeof(XT) == 2) {
    const u32x4 u = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(u[e] << 16);
      v[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int h = 0; h < E / 4; ++h) load4<XT>(p + 4 * h, v + 4 * h);
  }
}
template <typename YT, int E>
__device__ __forceinline__ void store_e(YT* p, const float (&v)[E]) {
  typedef YT ye __attribute__((ext_vector_type(E)));
  ye o;
#pragma unroll
  for (int e = 0; e < E; ++e) o[e] = from_f32<YT>(v[e]);
  *reinterpret_cast<ye*>(p) = o;
}

template <typename XT, typename YT, int NS, int E>
__global__ __launch_bounds__(256) void k_ln_modulate(const XT* __restrict__ x, RowMap xmap,
                                                     int64_t rows, int dim,
                                                     const float* __restrict__ shift,
                                                     const float* __restrict__ scale,
                                                     int64_t mod_stride, ModSel sel, float eps,
                                                     YT* __restrict__ y,
                                                     uint32_t* __restrict__ status) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int64_t b = r / xmap.rows_per_batch;
  const int64_t within = r - b * xmap.rows_per_batch;
  const int64_t src = b * xmap.batch_stride + xmap.row_offset + within;
  const XT* xr = x + src * dim;
  float v[NS][E];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    load_e<XT, E>(xr + i * 64 * E + lane * E, v[i]);
#pragma unroll
    for (int h = 0; h < E / 4; ++h)
      s += (v[i][4 * h] + v[i][4 * h + 1]) + (v[i][4 * h + 2] + v[i][4 * h + 3]);
  }
  const float mean = wave_sum(s) / (float)dim;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NS; ++i) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      v[i][e] -= mean;
      q = fmaf(v[i][e], v[i][e], q);
    }
  }
  const float var = wave_sum(q) / (float)dim;
  const float rstd = 1.0f / sqrtf(var + eps);
  const int64_t moff = b * mod_stride + (sel.pos_offset + within < sel.text_len ? sel.text_delta : 0);
  const float* sh = shift + moff;
  const float* sc = scale + moff;
  YT* yr = y + r * dim;
  bool bad = false;
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const int c = i * 64 * E + lane * E;
    float o[E];
#pragma unroll
    for (int h = 0; h < E / 4; ++h) {
      const f32x4 s4 = *reinterpret_cast<const f32x4*>(sc + c + 4 * h);
      const f32x4 h4 = *reinterpret_cast<const f32x4*>(sh + c + 4 * h);
#pragma unroll
      for (int e = 0; e < 4; ++e) o[4 * h + e] = fmaf(v[i][4 * h + e] * rstd, 1.0f + s4[e], h4[e]);
    }
    if constexpr (__is_same(YT, f16)) {
#pragma unroll
      for (int e = 0; e < E; ++e) bad |= !fits_f16(o[e]);
    }
    store_e<YT, E>(yr + c, o);
  }
  raise_flag(status, bad);
}

// ---------------------------------------------------------------------------
// Step 0: RoPE table.  Entry (axis a, position p, pair j) = (cos, sin) of
// p * theta^(-2j/d_a), computed in fp64.
// ---------------------------------------------------------------------------
__global__ void k_rope_table(RopeGeom g, float theta, float2* __restrict__ table) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  int base = 0;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    const int np = g.dims[a] / 2;
    const int n = g.grid[a] * np;
    if (i >= base && i < base + n) {
      const int p = (i - base) / np, j = (i - base) % np;
      const double ang = (double)p * pow((double)theta, -2.0 * (double)j / (double)g.dims[a]);
      double sn, cs;
      sincos(ang, &sn, &cs);
      table[i] = make_float2((float)cs, (float)sn);
    }
    base += n;
  }
}

// ---------------------------------------------------------------------------
// a3: QK-RMSNorm + 3D RoPE + scatter.  Queries are stored multiplied by
// log2(e)/sqrt(d), the factor the attention softmax applies to every score,
// so that attention can exponentiate scores with 2^x directly.  Workgroup =
// 64 tokens of one sequence x one head.  Q/K: one 16-byte slice (8 elements, 4 RoPE pairs) per item,
// D/8 lanes per token vector reduce the sum of squares with a butterfly.
// V: transposed through LDS so that V^T rows of 64 tokens are stored as 128
// contiguous bytes.  Tokens in [L, Lp) are written as zeros.
// ---------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(256) void k_qk_norm_rope(QkRopeArgs a) {
  constexpr int SL = HD / 8;               // 16-byte slices per head vector
  constexpr int TOK = 64;
  static_assert(256 % SL == 0, "a thread keeps one slice");
  __shared__ f16 vs[TOK][HD + 8];
  __shared__ int tpos[TOK][3];             // (t, y, w) of each visual token, -1 for text
  const int h = blockIdx.y, b = blockIdx.z;
  const int t0 = blockIdx.x * TOK;         // offset inside [0, count_ext)
  const int tid = threadIdx.x;
  const int64_t D = (int64_t)a.heads * HD;
  const int64_t head_base = ((int64_t)b * a.heads + h) * a.padded_len;

  if (tid < TOK) {
    const int vi = a.tok_begin + t0 + tid - a.text_len;
    // (a text-only request has an empty grid; its tokens never reach the division)
    const int gw = max(a.geom.grid[2], 1), hw = max(a.geom.grid[1] * a.geom.grid[2], 1);
    tpos[tid][0] = vi < 0 ? -1 : vi / hw;
    tpos[tid][1] = vi < 0 ? 0 : (vi % hw) / gw;
    tpos[tid][2] = vi < 0 ? 0 : vi % gw;
  }
  // This thread's slice never changes: find the RoPE axis, the pair index in
  // that axis and the axis' table base for each of its 4 pairs (axis -1: the
  // pair lies past the rotated dims).
  const int sl = tid % SL;
  int pax[4], pidx[4], pnp[4], pbase[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int pair = sl * 4 + e;
    int pair0 = 0, tbase = 0;
    pax[e] = -1; pidx[e] = 0; pnp[e] = 0; pbase[e] = 0;
#pragma unroll
    for (int ax = 0; ax < 3; ++ax) {
      const int np = a.geom.dims[ax] / 2;
      if (pax[e] < 0 && pair >= pair0 && pair < pair0 + np) {
        pax[e] = ax; pidx[e] = pair - pair0; pnp[e] = np; pbase[e] = tbase;
      }
      pair0 += np;
      tbase += a.geom.grid[ax] * np;
    }
  }
  float gq[8], gk[8];
  {
    const u32x4 vq = *reinterpret_cast<const u32x4*>(a.q_gamma + sl * 8);
    const u32x4 vk = *reinterpret_cast<const u32x4*>(a.k_gamma + sl * 8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      gq[2 * e] = __uint_as_float(vq[e] << 16);
      gq[2 * e + 1] = __uint_as_float(vq[e] & 0xffff0000u);
      gk[2 * e] = __uint_as_float(vk[e] << 16);
      gk[2 * e + 1] = __uint_as_float(vk[e] & 0xffff0000u);
    }
  }
  __syncthreads();

  // Q and K
  for (int ti = tid / SL; ti < TOK; ti += 256 / SL) {
    const int i = t0 + ti;                 // index inside the range
    const int tok = a.tok_begin + i;       // position in the sequence
    const bool in_range = i < a.count_ext;
    const bool real = i < a.tok_count;     // a token with input (tok < L)
    f16x8 u[2] = {};
    if (real) {
      const f16* row = a.qkv + ((int64_t)b * a.tok_count + i) * 3 * D + (int64_t)h * HD + sl * 8;
      u[0] = *reinterpret_cast<const f16x8*>(row);
      u[1] = *reinterpret_cast<const f16x8*>(row + D);
    }
    float2 cs[4];
    const int tp = tpos[ti][0];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      cs[e] = make_float2(1.f, 0.f);
      if (real && tp >= 0 && pax[e] >= 0) {
        const int pos = tpos[ti][pax[e]];
        cs[e] = a.table[pbase[e] + pos * pnp[e] + pidx[e]];
      }
    }
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (float)u[which][e];
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(v[e], v[e], ss);
#pragma unroll
      for (int o = SL / 2; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
      // 1/sqrt(mean + eps) with the hardware reciprocal square root (1 ulp)
      const float r = __builtin_amdgcn_rsqf(ss * (1.0f / (float)HD) + a.qk_eps);
      const float* g = which == 0 ? gq : gk;
      // queries also carry the softmax factor log2(e)/sqrt(d), applied after
      // the rotation with the normalisation, so there is one rounding
      const float f = which == 0 ? a.q_scale : 1.0f;
      f16x8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float u0 = v[2 * e] * r * g[2 * e], u1 = v[2 * e + 1] * r * g[2 * e + 1];
        o[2 * e] = (f16)(fmaf(u0, cs[e].x, -u1 * cs[e].y) * f);
        o[2 * e + 1] = (f16)(fmaf(u0, cs[e].y, u1 * cs[e].x) * f);
      }
      if (in_range) {
        f16* dst = (which == 0 ? a.q : a.k) + (head_base + tok) * HD + sl * 8;
        *reinterpret_cast<f16x8*>(dst) = o;
      }
    }
  }
  // V -> LDS (zeros for padding tokens)
  for (int item = tid; item < TOK * SL; item += 256) {
    const int ti = item / SL, sl = item % SL;
    const int i = t0 + ti;
    f16x8 u = {};
    if (i < a.tok_count)
      u = *reinterpret_cast<const f16x8*>(a.qkv + ((int64_t)b * a.tok_count + i) * 3 * D +
                                          2 * D + (int64_t)h * HD + sl * 8);
    *reinterpret_cast<f16x8*>(&vs[ti][sl * 8]) = u;
  }
  __syncthreads();
  // V^T rows: 64 tokens (8 groups of 8) per head dimension.  A full group at
  // an 8-aligned position is one 16-byte store; otherwise element stores, so
  // nothing outside [tok_begin, tok_begin + count_ext) is written.
  const bool aligned = (a.tok_begin & 7) == 0;
  for (int item = tid; item < HD * (TOK / 8); item += 256) {
    const int dim = item / (TOK / 8), ts = item % (TOK / 8);
    const int i = t0 + ts * 8;
    const int nv = min(8, a.count_ext - i);
    if (nv <= 0) continue;
    f16* dst = a.vt + (((int64_t)b * a.heads + h) * HD + dim) * a.padded_len + a.tok_begin + i;
    if (aligned && nv == 8) {
      f16x8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = vs[ts * 8 + e][dim];
      *reinterpret_cast<f16x8*>(dst) = o;
    } else {
      for (int e = 0; e < nv; ++e) dst[e] = vs[ts * 8 + e][dim];
    }
  }
}

// ---------------------------------------------------------------------------
// Step 4: bf16 -> fp16 copy, 8 elements per thread per iteration.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_convert_f16(const uint16_t* __restrict__ src,
                                                     f16* __restrict__ dst, int64_t n8,
                                                     uint32_t* __restrict__ status) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n8;
       i += (int64_t)gridDim.x * 256) {
    const u32x4 u = reinterpret_cast<const u32x4*>(src)[i];
    f16x8 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float w0 = __uint_as_float(u[e] << 16), w1 = __uint_as_float(u[e] & 0xffff0000u);
      bad |= !fits_f16(w0) || !fits_f16(w1);
      o[2 * e] = (f16)w0;
      o[2 * e + 1] = (f16)w1;
    }
    reinterpret_cast<f16x8*>(dst)[i] = o;
  }
  raise_flag(status, bad);
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_adaln(const uint16_t* cond, const uint16_t* w, const uint16_t* bias, int batch,
                        int cond_dim, int out_dim, float* mod, hipStream_t s, uint32_t* status_clear) {
  hipLaunchKernelGGL(k_adaln, dim3((out_dim + 3) / 4), dim3(256), 0, s, cond, w, bias, batch,
                     cond_dim, out_dim, mod, status_clear);
  return hipGetLastError();
}

template <typename XT, typename YT>
static hipError_t launch_ln_t(const XT* x, RowMap m, int64_t rows, int dim, const float* shift,
                              const float* scale, int64_t mod_stride, ModSel sel, float eps, YT* y,
                              hipStream_t s, uint32_t* status) {
  const dim3 grid((unsigned)((rows + 3) / 4));
  if constexpr (sizeof(XT) == 2) {
    if (dim % 512 == 0) {
      switch (dim / 512) {
#define XEMA_LN_CASE(NS)                                                                        \
  case NS:                                                                                      \
    hipLaunchKernelGGL((k_ln_modulate<XT, YT, NS, 8>), grid, dim3(256), 0, s, x, m, rows, dim,   \
                       shift, scale, mod_stride, sel, eps, y, status);                          \
    break;
        XEMA_LN_CASE(1) XEMA_LN_CASE(2) XEMA_LN_CASE(3) XEMA_LN_CASE(4) XEMA_LN_CASE(5)
        XEMA_LN_CASE(6) XEMA_LN_CASE(7) XEMA_LN_CASE(8) XEMA_LN_CASE(9) XEMA_LN_CASE(10)
        XEMA_LN_CASE(11) XEMA_LN_CASE(12) XEMA_LN_CASE(13) XEMA_LN_CASE(14) XEMA_LN_CASE(15)
        XEMA_LN_CASE(16)
#undef XEMA_LN_CASE
        default:
          return hipErrorInvalidValue;
      }
      return hipGetLastError();
    }
  }
  switch (dim / 256) {
#define XEMA_LN_CASE(NS)                                                                      \
  case NS:                                                                                    \
    hipLaunchKernelGGL((k_ln_modulate<XT, YT, NS, 4>), grid, dim3(256), 0, s, x, m, rows, dim, \
                       shift, scale, mod_stride, sel, eps, y, status);                        \
    break;
    XEMA_LN_CASE(1) XEMA_LN_CASE(2) XEMA_LN_CASE(3) XEMA_LN_CASE(4) XEMA_LN_CASE(5)
    XEMA_LN_CASE(6) XEMA_LN_CASE(7) XEMA_LN_CASE(8) XEMA_LN_CASE(9) XEMA_LN_CASE(10)
    XEMA_LN_CASE(11) XEMA_LN_CASE(12) XEMA_LN_CASE(13) XEMA_LN_CASE(14) XEMA_LN_CASE(15)
    XEMA_LN_CASE(16) XEMA_LN_CASE(17) XEMA_LN_CASE(18) XEMA_LN_CASE(19) XEMA_LN_CASE(20)
    XEMA_LN_CASE(21) XEMA_LN_CASE(22) XEMA_LN_CASE(23) XEMA_LN_CASE(24) XEMA_LN_CASE(25)
    XEMA_LN_CASE(26) XEMA_LN_CASE(27) XEMA_LN_CASE(28) XEMA_LN_CASE(29) XEMA_LN_CASE(30)
    XEMA_LN_CASE(31) XEMA_LN_CASE(32)
#undef XEMA_LN_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_ln_modulate(const void* x, int x_dtype, RowMap m, int64_t rows, int dim,
                              const float* shift, const float* scale, int64_t mod_stride,
                              ModSel sel, float eps, void* y, int y_dtype, hipStream_t s,
                              uint32_t* status) {
  if (x_dtype == XEMA_BF16 && y_dtype == XEMA_BF16)
    return launch_ln_t((const uint16_t*)x, m, rows, dim, shift, scale, mod_stride, sel, eps, (bf16*)y, s,
                       status);
  if (x_dtype == XEMA_BF16 && y_dtype == XEMA_F16)
    return launch_ln_t((const uint16_t*)x, m, rows, dim, shift, scale, mod_stride, sel, eps, (f16*)y, s,
                       status);
  if (x_dtype == XEMA_F32 && y_dtype == XEMA_BF16)
    return launch_ln_t((const float*)x, m, rows, dim, shift, scale, mod_stride, sel, eps, (bf16*)y, s,
                       status);
  if (x_dtype == XEMA_F32 && y_dtype == XEMA_F16)
    return launch_ln_t((const float*)x, m, rows, dim, shift, scale, mod_stride, sel, eps, (f16*)y, s,
                       status);
  return hipErrorInvalidValue;
}

hipError_t launch_rope_table(RopeGeom g, float theta, float* table, hipStream_t s) {
  int n = 0;
  for (int a = 0; a < 3; ++a) n += g.grid[a] * (g.dims[a] / 2);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, s, g, theta,
                     (float2*)table);
  return hipGetLastError();
}

// Zeros for the padding tokens [L, Lp) of Q and K ([B, H, Lp, d]) and V^T
// ([B, H, d, Lp]) when the QKV GEMM writes the heads itself; one workgroup
// per (head, batch row).
template <int HD>
__global__ __launch_bounds__(256) void k_qkv_pad(QkRopeArgs a, int seq_len) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int64_t Lp = a.padded_len;
  const int64_t hb = (int64_t)b * a.heads + h;
  const int n = (int)(Lp - seq_len) * HD;
  for (int i = threadIdx.x; i < n; i += 256) {
    const int64_t t = seq_len + i / HD;
    const int d = i % HD;
    a.q[(hb * Lp + t) * HD + d] = (f16)0.f;
    a.k[(hb * Lp + t) * HD + d] = (f16)0.f;
    a.vt[(hb * HD + d) * Lp + t] = (f16)0.f;
  }
}

hipError_t launch_qkv_pad(const QkRopeArgs& a, int head_dim, int seq_len, hipStream_t s) {
  if (a.padded_len <= seq_len || a.heads <= 0 || a.batch <= 0) return hipSuccess;
  const dim3 grid((unsigned)a.heads, (unsigned)a.batch);
  if (head_dim == 64)
    hipLaunchKernelGGL(k_qkv_pad<64>, grid, dim3(256), 0, s, a, seq_len);
  else if (head_dim == 128)
    hipLaunchKernelGGL(k_qkv_pad<128>, grid, dim3(256), 0, s, a, seq_len);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_qk_norm_rope(const QkRopeArgs& a, int head_dim, hipStream_t s) {
  const dim3 grid((unsigned)((a.count_ext + 63) / 64), (unsigned)a.heads, (unsigned)a.batch);
  if (head_dim == 64)
    hipLaunchKernelGGL(k_qk_norm_rope<64>, grid, dim3(256), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL(k_qk_norm_rope<128>, grid, dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_convert_f16(const uint16_t* src, f16* dst, int64_t n, hipStream_t s, uint32_t* status) {
  const int64_t n8 = n / 8;
  const int64_t blocks = std::min<int64_t>((n8 + 255) / 256, 256 * 16);
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(k_convert_f16, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, n8, status);
  return hipGetLastError();
}

}  // namespace xema
