// Joint full self-attention (step a4) on gfx950: flash-style, online softmax
// in registers, K and V^T tiles double-buffered in LDS, fp16 MFMA with fp32
// accumulation.
//
// Formulation.  Each wave owns QB columns blocks of 32 queries and computes
// S^T = K Q^T with v_mfma_f32_32x32x16_f16: the key tile is the A operand, the
// queries the B operand, so every lane holds one query column (16 scores per
// 32-key block).  The row max and row sum of a query are then in-lane
// reductions plus one exchange between lanes l and l^32 (v_permlane32_swap).
// O^T = V^T P^T reuses the score registers directly as the B operand: the keys
// of the K tile are loaded in a permuted order so that the eight scores a lane
// holds for one k-group of the P V^T product are eight consecutive keys, which
// makes every V^T fragment one 16-byte read.
//
// Softmax.  Queries arrive scaled by log2(e)/sqrt(d) (the QK-norm/RoPE step
// stores them so), and P = 2^x is taken with v_exp_f32.  The running max is updated lazily: a query keeps the
// max it last rescaled to until a tile's max exceeds it by more than TAU, so P
// stays <= 2^TAU (well inside fp16) and the rescale of O and of the row sum
// is skipped for almost every tile.  A wave executes the rescale when any of
// its lanes needs it; lanes that do not need it multiply by exactly 1.0, so a
// query's result never depends on the other queries of its wave.
//
// Keys are visited in one fixed ascending order of 64-key tiles, and every
// operation is per query column, so a query's output does not depend on the
// other queries of its wave, workgroup or chunk: chunked and unchunked runs
// agree bit for bit.
//
// LDS layouts.  K tile: 64 rows (keys) of HD halves; V^T tile: HD rows (head
// dims) of 64 keys (128 bytes).  The 16-byte slots of each row are XOR-
// swizzled (swz_k, swz_v below) so that every 16-byte fragment read is free of
// bank conflicts.  Tiles are filled with buffer_load ... lds, 1 KiB per wave
// instruction.
//
// Workgroups: NW waves = NW * QB * 32 queries of one (batch, head).  The grid
// is 1-D and remapped so that all query blocks of a head run on one XCD and
// share its L2 copy of K and V.
#include "device_common.h"
#include "kernels.h"

#ifndef XEMA_ATT64_QB
#define XEMA_ATT64_QB 2
#endif
#ifndef XEMA_ATT64_NW
#define XEMA_ATT64_NW 8
#endif
#ifndef XEMA_ATT128_QB
#define XEMA_ATT128_QB 1
#endif
#ifndef XEMA_ATT128_NW
#define XEMA_ATT128_NW 8
#endif

namespace xema {

namespace {

constexpr int KV = 64;          // keys per tile
constexpr float TAU = 8.0f;     // lazy-rescale slack, log2 units
constexpr int BUF_FLAGS = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           BUF_FLAGS);
}

__device__ __forceinline__ f32x16 mma(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// values of lanes l and l^32 combined: r[0] is the low-half lane's value and
// r[1] the high-half lane's value in both lanes, so both get the same result.
__device__ __forceinline__ float pair_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// physical key (0..31 inside a 32-key block) behind MFMA row rho
__device__ __forceinline__ int kappa(int rho) {
  return ((rho >> 4) << 4) | (((rho >> 2) & 1) << 3) | (((rho >> 3) & 1) << 2) | (rho & 3);
}
// 16-byte slot swizzles.  The LDS has 64 four-byte banks and serves a
// 16-byte read for 16 lanes per cycle; each group of 16 lanes reads 16
// distinct rows (a permutation of 16 consecutive rows) at one logical slot.
// 128-byte rows: row pairs share a 256-byte bank line, so the slot is XORed
// with (r >> 1) & 7; 256-byte rows (K at d = 128): XOR with r & 15.
template <int HD>
__device__ __forceinline__ int swz_k(int r) { return HD == 64 ? (r >> 1) & 7 : r & 15; }
__device__ __forceinline__ int swz_v(int r) { return (r >> 1) & 7; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Queue the K and V^T tiles of one key tile into one LDS stage (this wave's
// share: NK + NV instructions of 1 KiB each).
template <int NK, int NV, int K_BYTES, int NW>
__device__ __forceinline__ void issue_kv(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                         const uint32_t (&k_off)[NK], const uint32_t (&v_off)[NV],
                                         uint8_t* stage, int wave, uint32_t kb, uint32_t vb) {
#pragma unroll
  for (int j = 0; j < NK; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr_t)(stage + (wave + NW * j) * 1024),
                                             16, k_off[j] + kb, 0, 0, 0);
#pragma unroll
  for (int j = 0; j < NV; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rv, (lds_ptr_t)(stage + K_BYTES + (wave + NW * j) * 1024), 16, v_off[j] + vb, 0, 0, 0);
}

}  // namespace

template <int HD, int QB, int NW>
__global__ __launch_bounds__(NW * 64) void k_attention(AttnParams p) {
  constexpr int K_BYTES = KV * HD * 2;        // K tile bytes
  constexpr int V_BYTES = HD * KV * 2;        // V^T tile bytes
  constexpr int NKK = HD / 16;                // k-steps of the QK^T MFMA
  constexpr int NDB = HD / 32;                // 32-dim blocks of O
  constexpr int QW = QB * 32;                 // queries per wave
  constexpr int QWG = QW * NW;                // queries per workgroup
  constexpr int K_INSTR = K_BYTES / 1024 / NW;
  constexpr int V_INSTR = V_BYTES / 1024 / NW;
  static_assert(K_INSTR * NW * 1024 == K_BYTES && V_INSTR * NW * 1024 == V_BYTES, "load split");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2][K_BYTES + V_BYTES];

  // 1-D grid -> (query block, head, batch), all query blocks of a head on one XCD
  const int nqb = (p.q_count + QWG - 1) / QWG;
  const int total = nqb * p.heads * p.batch;
  const int wg = blockIdx.x;
  const int xcd = wg & 7, slot = wg >> 3;
  const int per = total >> 3, rem = total & 7;
  const int t = xcd * per + min(xcd, rem) + slot;
  const int qb = t % nqb;
  const int bh = t / nqb;                     // b * heads + h
  const int b = bh / p.heads, h = bh - b * p.heads;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r32 = lane & 31, hi = lane >> 5;
  const int64_t Lp = p.padded_len;

  const f16* Qh = p.q + (int64_t)bh * Lp * HD;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(p.k + (int64_t)bh * Lp * HD, Lp * HD * 2);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(p.vt + (int64_t)bh * HD * Lp, (int64_t)HD * Lp * 2);

  // load plan for the K tile: instruction j of this wave writes bytes
  // [1024*(wave + NW j), +1024): row = byte / (2 HD), physical slot ps.
  // V^T tile: instruction j writes rows 8*(wave + NW j) .. +7.
  uint32_t k_off[K_INSTR], v_off[V_INSTR];
#pragma unroll
  for (int j = 0; j < K_INSTR; ++j) {
    const int byte = (wave + NW * j) * 1024 + lane * 16;
    const int row = byte / (2 * HD), ps = (byte % (2 * HD)) / 16;
    k_off[j] = (uint32_t)((row * HD + ((ps ^ swz_k<HD>(row)) * 8)) * 2);
  }
#pragma unroll
  for (int j = 0; j < V_INSTR; ++j) {
    const int row = (wave + NW * j) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ swz_v(row);
    v_off[j] = (uint32_t)((row * Lp + c * 8) * 2);
  }

  // Q fragments (B operand): lane holds Q[q][kk*16 + hi*8 .. +8] of its column
  const int q_first = p.q_begin + qb * QWG + wave * QW;
  // (the stored queries carry the log2(e)/sqrt(d) factor, so the score MFMA
  // yields the exponent of 2 directly)
  f16x8 qf[QB][NKK];
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    const int q = min(q_first + c * 32 + r32, (int)Lp - 1);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      qf[c][kk] = *reinterpret_cast<const f16x8*>(Qh + (int64_t)q * HD + kk * 16 + hi * 8);
  }

  f32x16 oacc[QB][NDB];
#pragma unroll
  for (int c = 0; c < QB; ++c)
#pragma unroll
    for (int d = 0; d < NDB; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[c][d][r] = 0.f;
  // mrow: the max in use (log2 units); lrow: this lane's share of the row sum
  float mrow[QB], lrow[QB];
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    mrow[c] = 0.f;
    lrow[c] = 0.f;
  }

  // fragment addressing inside the tiles
  const int krow = kappa(r32);                      // key row read by this lane
  const int kswz = swz_k<HD>(krow);
  const int nkv = (p.seq_len + KV - 1) / KV;
  const int tail = p.seq_len - (nkv - 1) * KV;      // valid keys in the last tile

  issue_kv<K_INSTR, V_INSTR, K_BYTES, NW>(rk, rv, k_off, v_off, smem[0], wave, 0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kv = 0; kv < nkv; ++kv) {
    const int stage = kv & 1;
    if (kv + 1 < nkv)
      issue_kv<K_INSTR, V_INSTR, K_BYTES, NW>(rk, rv, k_off, v_off, smem[stage ^ 1], wave,
                                              (uint32_t)((kv + 1) * KV * HD * 2),
                                              (uint32_t)((kv + 1) * KV * 2));
    const uint8_t* Ks = smem[stage];
    const uint8_t* Vs = smem[stage] + K_BYTES;

    // S^T = K Q^T for two 32-key blocks x QB query columns
    f32x16 s[2][QB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int row = kb * 32 + krow;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        const int slot16 = (kk * 2 + hi) ^ kswz;
        const f16x8 kf = *reinterpret_cast<const f16x8*>(Ks + row * (HD * 2) + slot16 * 16);
#pragma unroll
        for (int c = 0; c < QB; ++c) s[kb][c] = mma(kf, qf[c][kk], kk == 0 ? f32x16{} : s[kb][c]);
      }
    }
    if (kv == nkv - 1 && tail < KV) {
      // lane's score r of block kb is key kb*32 + 16*(r>>3) + 8*hi + (r&7)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb * 32 + 16 * (r >> 3) + 8 * hi + (r & 7);
          if (key >= tail) {
#pragma unroll
            for (int c = 0; c < QB; ++c) s[kb][c][r] = -INFINITY;
          }
        }
    }
    // Online softmax per query column with a lazy max.  A column "grows" when
    // its tile max exceeds mrow by more than TAU (and on the first tile, to
    // set mrow); only then does mrow move and O get rescaled.  The wave takes
    // the rescaling path when any lane grows; the other lanes keep their mrow
    // and multiply by exactly 1.0.
    f16x8 pf[QB][2][2];  // [column][key block][16-key half]
    float mxs[QB];
    bool grow_any = kv == 0;
#pragma unroll
    for (int c = 0; c < QB; ++c) {
      float mx = s[0][c][0];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][c][r]);
      mxs[c] = pair_max(mx);
      grow_any |= mxs[c] - mrow[c] > TAU;
    }
    if (__builtin_amdgcn_ballot_w64(grow_any)) {
#pragma unroll
      for (int c = 0; c < QB; ++c) {
        const bool grow = kv == 0 || mxs[c] - mrow[c] > TAU;
        const float alpha = kv == 0 ? 0.f : (grow ? fast_exp2(mrow[c] - mxs[c]) : 1.f);
        if (grow) mrow[c] = mxs[c];
        lrow[c] *= alpha;
#pragma unroll
        for (int d = 0; d < NDB; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[c][d][r] *= alpha;
      }
    }
#pragma unroll
    for (int c = 0; c < QB; ++c) {
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pv = fast_exp2(s[kb][c][8 * u + e] - mrow[c]);
            ls += pv;
            pf[c][kb][u][e] = (f16)pv;
          }
      lrow[c] += ls;
    }
    // O^T += V^T P^T
#pragma unroll
    for (int d = 0; d < NDB; ++d) {
      const int vrow = d * 32 + r32;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int slot16 = (kb * 4 + u * 2 + hi) ^ swz_v(vrow);
          const f16x8 vf = *reinterpret_cast<const f16x8*>(Vs + vrow * (KV * 2) + slot16 * 16);
#pragma unroll
          for (int c = 0; c < QB; ++c) oacc[c][d] = mma(vf, pf[c][kb][u], oacc[c][d]);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  // normalise and store O[b * q_count + (q - q_begin)][h*HD + dim]
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    const int q = q_first + c * 32 + r32;
    const float inv = 1.0f / pair_sum(lrow[c]);
    if (q >= p.q_begin + p.q_count) continue;
    f16* orow = p.o + ((int64_t)b * p.q_count + (q - p.q_begin)) * ((int64_t)p.heads * HD) +
                (int64_t)h * HD;
#pragma unroll
    for (int d = 0; d < NDB; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (f16)(oacc[c][d][4 * g + e] * inv);
        *reinterpret_cast<f16x4*>(orow + d * 32 + 8 * g + 4 * hi) = o;
      }
  }
}

template <int HD, int QB, int NW>
static hipError_t launch_t(const AttnParams& p, hipStream_t s) {
  constexpr int QWG = QB * 32 * NW;
  const int64_t nqb = (p.q_count + QWG - 1) / QWG;
  const int64_t total = nqb * p.heads * p.batch;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL((k_attention<HD, QB, NW>), dim3((unsigned)total), dim3(NW * 64), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnParams& p, int head_dim, hipStream_t s) {
  if (head_dim == 64) return launch_t<64, XEMA_ATT64_QB, XEMA_ATT64_NW>(p, s);
  if (head_dim == 128) return launch_t<128, XEMA_ATT128_QB, XEMA_ATT128_NW>(p, s);
  return hipErrorInvalidValue;
}

}  // namespace xema
