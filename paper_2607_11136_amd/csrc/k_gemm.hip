// C = A B^T on gfx950 bf16/fp16 MFMA, with the block's fused epilogues
// (bias, bias + GELU-tanh, gated residual).  Steps a2, a5, a7, a8.
//
// Tiling: a 256 x 256 output tile per workgroup, K in steps of 64.  Four
// waves in a 2 x 2 grid each own a 128 x 128 sub-tile held as 4 x 4
// accumulators of v_mfma_f32_32x32x16.  Operand tiles go from HBM straight
// into LDS with buffer_load ... lds (no VGPR staging), double-buffered; the
// buffer descriptor of each tile covers only that tile's rows, so rows past M
// read as zero.  Each LDS row is 64 elements (128 bytes, eight 16-byte
// slots); slot j of row r is stored at slot j ^ (r & 7), which keeps the
// 16-byte fragment reads of eight consecutive lanes on distinct banks.
//
// The MFMA takes the weight fragment as its A operand and the activation
// fragment as its B operand, so each lane ends up holding four consecutive
// output features of one token row: epilogue loads/stores are 8/16 bytes.
//
// Workgroups are dispatched round-robin over the 8 XCDs; the tile order
// below gives each XCD a contiguous range of tiles, walked in groups of 8
// tile-rows, so tiles that share operand panels share an L2.
//
// Determinism: every output element is the sum over ascending 64-wide K
// tiles, each reduced by the same MFMA sequence, whatever M, the row maps or
// the tile position are; so chunked and unchunked calls agree bit for bit.
#include "device_common.h"
#include "kernels.h"

namespace xema {

namespace {

template <typename T>
struct Mfma;
template <>
struct Mfma<bf16> {
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x16 run(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<f16> {
  typedef f16x8 frag;
  static __device__ __forceinline__ f32x16 run(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int TILE_BYTES = BM * BK * 2;  // 32 KiB per operand tile
constexpr int GROUP_M = 8;
constexpr int BUF_FLAGS = 0x00020000;   // raw buffer, 32-bit dwords

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           BUF_FLAGS);
}

template <typename CT>
__device__ __forceinline__ void store4(CT* p, const float v[4]) {
  typedef CT c4 __attribute__((ext_vector_type(4)));
  c4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = from_f32<CT>(v[e]);
  *reinterpret_cast<c4*>(p) = o;
}

template <typename RT>
__device__ __forceinline__ void load4f(const RT* p, float v[4]);
template <>
__device__ __forceinline__ void load4f<float>(const float* p, float v[4]) {
  const f32x4 u = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = u[e];
}
template <>
__device__ __forceinline__ void load4f<uint16_t>(const uint16_t* p, float v[4]) {
  const u32x2 u = *reinterpret_cast<const u32x2*>(p);
  v[0] = __uint_as_float(u[0] << 16);
  v[1] = __uint_as_float(u[0] & 0xffff0000u);
  v[2] = __uint_as_float(u[1] << 16);
  v[3] = __uint_as_float(u[1] & 0xffff0000u);
}

}  // namespace

// EPI: XEMA_EPI_BIAS / XEMA_EPI_BIAS_GELU (CT = bf16 or f16) or
// XEMA_EPI_GATED_RESIDUAL (CT = float, RT = residual element type).
template <typename T, int EPI, typename CT, typename RT>
__global__ __launch_bounds__(256, 1) void k_gemm(GemmParams p) {
  typedef typename Mfma<T>::frag frag;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2][2][TILE_BYTES];

  const int K = p.K;
  const int tiles_m = (int)((p.M + BM - 1) / BM);
  const int tiles_n = p.N / BN;
  const int total = tiles_m * tiles_n;
  // XCD-aware tile order (see the file comment)
  const int wg = blockIdx.x;
  const int xcd = wg & 7, slot = wg >> 3;
  const int per = total >> 3, rem = total & 7;
  const int t = xcd * per + min(xcd, rem) + slot;
  const int group = t / (GROUP_M * tiles_n);
  const int first_m = group * GROUP_M;
  const int gsize = min(tiles_m - first_m, GROUP_M);
  const int in_group = t - group * GROUP_M * tiles_n;
  const int tm = first_m + in_group % gsize;
  const int tn = in_group / gsize;
  const int64_t m0 = (int64_t)tm * BM;
  const int n0 = tn * BN;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const T* A = reinterpret_cast<const T*>(p.a);
  const T* Bw = reinterpret_cast<const T*>(p.b);
  const int64_t rows_a = min<int64_t>(BM, p.M - m0);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + m0 * K, rows_a * K * 2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(Bw + (int64_t)n0 * K, (int64_t)BN * K * 2);

  // direct-to-LDS load plan: wave w fills 1 KiB chunks w*8 .. w*8+7 of each
  // operand tile; chunk c covers rows 8c .. 8c+7, lane l writes row 8c + l/8,
  // physical slot l%8, so it fetches logical slot (l%8) ^ (l/8).
  const int lrow = lane >> 3;
  const uint32_t voff = (uint32_t)(((wave * 64 + lrow) * K + (((lane & 7) ^ lrow) * 8)) * 2);
  const uint32_t chunk_stride = (uint32_t)(8 * K * 2);

  auto issue = [&](int kt, int stage) {
    const uint32_t kbyte = (uint32_t)(kt * BK * 2);
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
      const uint32_t so = cc * chunk_stride + kbyte;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ra, (lds_ptr_t)(&smem[stage][0][(wave * 8 + cc) * 1024]), 16, voff, so, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rb, (lds_ptr_t)(&smem[stage][1][(wave * 8 + cc) * 1024]), 16, voff, so, 0, 0);
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // fragment addressing: lane reads row (block + lane%32), k-slot kk*2 + lane/32
  const int r32 = lane & 31, hi = lane >> 5, sw = lane & 7;
  const int a_row0 = (wm * 128 + r32) * 128;  // byte offset of this lane's first A row
  const int b_row0 = (wn * 128 + r32) * 128;

  const int KT = K / BK;
  issue(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int stage = kt & 1;
    if (kt + 1 < KT) issue(kt + 1, stage ^ 1);
    const uint8_t* As = smem[stage][0];
    const uint8_t* Bs = smem[stage][1];
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int so = (((kk * 2 + hi) ^ sw) * 16);
      frag xa[4], wb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        xa[i] = *reinterpret_cast<const frag*>(As + a_row0 + i * 32 * 128 + so);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        wb[j] = *reinterpret_cast<const frag*>(Bs + b_row0 + j * 32 * 128 + so);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = Mfma<T>::run(wb[j], xa[i], acc[i][j]);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  // Epilogue.  acc[i][j][r] = C[m][n] with m = m0 + wm*128 + i*32 + r32 and
  // n = n0 + wn*128 + j*32 + 8*(r/4) + 4*hi + r%4.
  const int64_t rpb = p.c_map.rows_per_batch;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + wm * 128 + i * 32 + r32;
    if (m >= p.M) continue;
    const int64_t b = m / rpb;
    const int64_t within = m - b * rpb;
    const int64_t crow = b * p.c_map.batch_stride + p.c_map.row_offset + within;
    CT* crow_ptr = reinterpret_cast<CT*>(p.c) + crow * p.ldc;
    const RT* rrow_ptr = nullptr;
    const float* grow = nullptr;
    if (EPI == XEMA_EPI_GATED_RESIDUAL) {
      const int64_t rrow = b * p.resid_map.batch_stride + p.resid_map.row_offset + within;
      rrow_ptr = reinterpret_cast<const RT*>(p.resid) + rrow * p.ld_resid;
      grow = p.gate + b * p.gate_stride;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * 128 + j * 32 + 8 * q + 4 * hi;
        float bias[4], v[4];
        load4f<uint16_t>(p.bias + n, bias);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e] + bias[e];
        if (EPI == XEMA_EPI_BIAS_GELU) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = gelu_tanh(v[e]);
        }
        if (EPI == XEMA_EPI_GATED_RESIDUAL) {
          float res[4];
          load4f<RT>(rrow_ptr + n, res);
          const f32x4 g = *reinterpret_cast<const f32x4*>(grow + n);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = fmaf(g[e], v[e], res[e]);
        }
        store4<CT>(crow_ptr + n, v);
      }
    }
  }
}

hipError_t launch_gemm(const GemmParams& p, hipStream_t s) {
  const int64_t tiles = ((p.M + BM - 1) / BM) * (p.N / BN);
  if (tiles == 0) return hipSuccess;
  const dim3 grid((unsigned)tiles), block(256);
#define XEMA_GEMM(T, EPI, CT, RT) hipLaunchKernelGGL((k_gemm<T, EPI, CT, RT>), grid, block, 0, s, p)
  const bool h = p.dtype == XEMA_F16;
  switch (p.epilogue) {
    case XEMA_EPI_BIAS:
    case XEMA_EPI_BIAS_GELU: {
      const bool gelu = p.epilogue == XEMA_EPI_BIAS_GELU;
      const bool ch = p.c_dtype == XEMA_F16;
      if (h && ch && gelu) XEMA_GEMM(f16, XEMA_EPI_BIAS_GELU, f16, float);
      else if (h && ch) XEMA_GEMM(f16, XEMA_EPI_BIAS, f16, float);
      else if (h && gelu) XEMA_GEMM(f16, XEMA_EPI_BIAS_GELU, bf16, float);
      else if (h) XEMA_GEMM(f16, XEMA_EPI_BIAS, bf16, float);
      else if (ch && gelu) XEMA_GEMM(bf16, XEMA_EPI_BIAS_GELU, f16, float);
      else if (ch) XEMA_GEMM(bf16, XEMA_EPI_BIAS, f16, float);
      else if (gelu) XEMA_GEMM(bf16, XEMA_EPI_BIAS_GELU, bf16, float);
      else XEMA_GEMM(bf16, XEMA_EPI_BIAS, bf16, float);
      break;
    }
    case XEMA_EPI_GATED_RESIDUAL: {
      const bool rf = p.resid_dtype == XEMA_F32;
      if (h && rf) XEMA_GEMM(f16, XEMA_EPI_GATED_RESIDUAL, float, float);
      else if (h) XEMA_GEMM(f16, XEMA_EPI_GATED_RESIDUAL, float, uint16_t);
      else if (rf) XEMA_GEMM(bf16, XEMA_EPI_GATED_RESIDUAL, float, float);
      else XEMA_GEMM(bf16, XEMA_EPI_GATED_RESIDUAL, float, uint16_t);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
#undef XEMA_GEMM
  return hipGetLastError();
}

}  // namespace xema
