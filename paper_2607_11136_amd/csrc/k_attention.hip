// Joint full self-attention (step a4) on gfx950: flash-style, online softmax
// in registers, K and V^T tiles staged in LDS, fp16 MFMA with fp32
// accumulation.
//
// Formulation.  Each wave owns QB column blocks of 32 queries and computes
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
// stores them so), and P = 2^x is taken with v_exp_f32.  The running max is a
// lazy reference max: O and the row sum are rescaled only when a tile would
// push P out of a fixed range, which is rare after the first tiles.  Two
// kernels differ in how they detect that and in their schedule:
//   k_attention (used at d = 128): the reference max enters as the
//     accumulator input of the score MFMA, the trigger is the sum of a tile's
//     P exceeding PMAX = 2^12 (the sum of the packed fp16 P, which is also
//     the row sum), two wave groups run offset by a phase over a 3-stage LDS
//     ring so one group's softmax overlaps the other's MFMAs;
//   k_attention_lazy (used at d = 64): two column blocks per wave (half the
//     LDS reads per score) and a 2-stage ring.  The reference max enters as
//     the accumulator input of the first score MFMA as well, so P is taken
//     straight from the MFMA output, and the trigger is the same P sum as
//     above: the common path has no max reduction and no subtraction; the
//     rare rescaling path finds the tile max and recomputes P.  The two columns run offset
//     within a tile, so that MFMAs of one are issued beside the
//     exponentials of the other.  Scores must stay below 2^16 in log2 units.
// Measured on the workloads' own Q/K/V, each is the faster one at its width.
//
// Keys are visited in one fixed ascending order of 64-key tiles, and every
// operation is per query column (a wave takes the rescaling path when any of
// its columns needs it; the others rescale by exactly 1.0), so a query's
// output does not depend on the other queries of its wave, workgroup or chunk:
// chunked and unchunked runs agree bit for bit.
//
// LDS layouts.  K tile: 64 rows (keys) of HD halves; V^T tile: HD rows (head
// dims) of 64 keys (128 bytes).  The 16-byte slots of each row are XOR-
// swizzled (swz_k, swz_v below) so that every 16-byte fragment read is free of
// bank conflicts.  Tiles are filled with buffer_load ... lds, 1 KiB per wave
// instruction.
//
// Workgroups: NW = 8 waves = 8 * QB * 32 queries of one (batch, head).  The
// grid is 1-D and remapped so that all query blocks of a head run on one XCD
// and share its L2 copy of K and V.
#include "attention.h"
#include "device_common.h"

namespace xema {

namespace {

constexpr int KV = 64;          // keys per tile
constexpr float PMAX = 4096.0f; // bound on a lane's P sum over a tile before the max moves

// Whether the reference max enters through the score MFMA's accumulator input
// (16 more VGPRs per query column) or is subtracted before the exponential.
constexpr bool minit_in_mfma(int qb) { return qb <= 1; }
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

// P = 2^(s - shift) for the 32 scores a lane holds for one query column,
// packed to fp16 as the B operand of the P V^T product; returns the sum of
// the packed fp16 values.  The pairs are added as packed fp16 into two
// partial sums of eight pairs each, which two v_dot2 with (1, 1) add in fp32:
// a chain of sixteen v_dot2 per column, one per pair, cost about 5% of the
// kernel on the video workload and overlapped nothing.  The fp16 additions
// round with relative error 2^-11 each (the tile's sum enters the row sum and
// the rescale trigger; a P that overflows fp16 still makes the sum
// infinite).
template <bool SHIFT>
__device__ __forceinline__ float exp_pack(const f32x16& s0, const f32x16& s1, float shift,
                                          f16x8 (&pf)[2][2]) {
  const f16x2 one = {(f16)1.f, (f16)1.f};
  f16x2 part[2] = {{(f16)0.f, (f16)0.f}, {(f16)0.f, (f16)0.f}};
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const f32x16& sv = kb ? s1 : s0;
        const float x0 = SHIFT ? sv[8 * u + e] - shift : sv[8 * u + e];
        const float x1 = SHIFT ? sv[8 * u + e + 1] - shift : sv[8 * u + e + 1];
        const f16x2 h = {(f16)fast_exp2(x0), (f16)fast_exp2(x1)};
        part[(e >> 1) & 1] += h;
        pf[kb][u][e] = h[0];
        pf[kb][u][e + 1] = h[1];
      }
  return __builtin_amdgcn_fdot2(part[1], one, __builtin_amdgcn_fdot2(part[0], one, 0.f, false), false);
}

// Queue the K and V^T tiles of one key tile into one LDS stage (this wave's
// share: NK + NV instructions of 1 KiB each).
template <int NK, int NV, int K_BYTES, int NW>
__device__ __forceinline__ void issue_kv(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                         const uint32_t* k_off, const uint32_t* v_off,
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

// Per-wave softmax state of QB query columns.
template <int HD, int QB>
struct WaveState {
  f32x16 oacc[QB][HD / 32];  // O^T accumulators
  f32x16 minit[QB];          // -mrow in all 16 entries
  float mrow[QB];            // reference max in use (log2 units)
  float lrow[QB];            // this lane's share of the row sum
};

// S^T - mrow for two 32-key blocks of one query column: -mrow is the
// accumulator input of the first k-step, so the scores arrive shifted.
// (The key fragments are the same for every column; the compiler reads them
// from LDS once per tile.)  The first k-step of each block is written out
// with an early-clobber output, so that it reads minit where it lies: the
// builtin form made the compiler copy minit into the second block's
// accumulator on every tile (16 64-bit moves per tile and column pair, 1%
// of the kernel).  Its result feeds the next MFMA of the same opcode as
// that MFMA's accumulator, a dependency the compiler pads with wait states.
template <int HD>
__device__ __forceinline__ void scores_col(const uint8_t* Ks, const f16x8 (&qc)[HD / 16], const f32x16& minit,
                                           int krow, int kswz, int hi, f32x16 (&s)[2]) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int row = kb * 32 + krow;
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk) {
      const int slot16 = (kk * 2 + hi) ^ kswz;
      const f16x8 kf = *reinterpret_cast<const f16x8*>(Ks + row * (HD * 2) + slot16 * 16);
      if (kk == 0)
        asm("v_mfma_f32_32x32x16_f16 %0, %1, %2, %3" : "=&v"(s[kb]) : "v"(kf), "v"(qc[kk]), "v"(minit));
      else
        s[kb] = mma(kf, qc[kk], s[kb]);
    }
  }
}

// S^T = K Q^T - mrow for two 32-key blocks x QB query columns
template <int HD, int QB, bool MI>
__device__ __forceinline__ void tile_scores(const uint8_t* Ks, const f16x8 (&qf)[QB][HD / 16],
                                            const f32x16 (&minit)[QB], int krow, int kswz, int hi,
                                            f32x16 (&s)[2][QB]) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int row = kb * 32 + krow;
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk) {
      const int slot16 = (kk * 2 + hi) ^ kswz;
      const f16x8 kf = *reinterpret_cast<const f16x8*>(Ks + row * (HD * 2) + slot16 * 16);
#pragma unroll
      for (int c = 0; c < QB; ++c)
        s[kb][c] = mma(kf, qf[c][kk], kk == 0 ? (MI ? minit[c] : f32x16{}) : s[kb][c]);
    }
  }
}

// keys at or past `tail` in this tile get score -inf
template <int QB>
__device__ __forceinline__ void mask_tail(f32x16 (&s)[2][QB], int tail, int hi) {
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

// the same for one query column
__device__ __forceinline__ void mask_tail_col(f32x16 (&s)[2], int tail, int hi) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (kb * 32 + 16 * (r >> 3) + 8 * hi + (r & 7) >= tail) s[kb][r] = -INFINITY;
}

// Online softmax of one tile with a lazy reference max.  Scores arrive as
// score - mrow.  The common path takes P = 2^s directly.  A column "grows"
// when the sum of its tile's P exceeds PMAX (some score may then exceed mrow
// by about log2(PMAX)), and on the first tile, to set mrow: mrow moves to the
// tile max, O and the row sum are rescaled and P is recomputed.  The wave
// takes that path when any column grows; the other columns recompute the
// same P (shift 0) and scale by 1.0, so a query's result never depends on the
// other queries of its wave.
template <int HD, int QB>
__device__ __forceinline__ void tile_softmax(const f32x16 (&s)[2][QB], bool first,
                                             WaveState<HD, QB>& st, f16x8 (&pf)[QB][2][2]) {
  constexpr bool MI = minit_in_mfma(QB);
  float lsp[QB];
  bool grow_any = first;
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    lsp[c] = exp_pack<!MI>(s[0][c], s[1][c], MI ? 0.f : st.mrow[c], pf[c]);
    grow_any |= pair_max(lsp[c]) > PMAX;
  }
  if (__builtin_amdgcn_ballot_w64(grow_any)) {
#pragma unroll
    for (int c = 0; c < QB; ++c) {
      const bool grow = first || pair_max(lsp[c]) > PMAX;
      float mx = s[0][c][0];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][c][r]);
      mx = pair_max(mx) - (MI ? 0.f : st.mrow[c]);  // tile max relative to mrow
      const float shift = grow ? mx : 0.f;
      const float alpha = first ? 0.f : (grow ? fast_exp2(-shift) : 1.f);
      st.mrow[c] += shift;
      if (MI) {
#pragma unroll
        for (int r = 0; r < 16; ++r) st.minit[c][r] = -st.mrow[c];
      }
      lsp[c] = exp_pack<true>(s[0][c], s[1][c], MI ? shift : st.mrow[c], pf[c]);
      st.lrow[c] *= alpha;
#pragma unroll
      for (int d = 0; d < HD / 32; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) st.oacc[c][d][r] *= alpha;
    }
  }
#pragma unroll
  for (int c = 0; c < QB; ++c) st.lrow[c] += lsp[c];
}

// Online softmax for k_attention_lazy.  The scores arrive as s - mrow (the
// accumulator input of scores_col), so the common path packs P = 2^s straight
// from the MFMA output; its sum (exp_pack) is the row sum.  A column grows when
// the larger of its two lanes' sums exceeds PMAX (a P that overflows fp16
// makes its sum infinite, so it always grows) and on the first tile; then
// rescale_col moves mrow to the tile max, rounded to fp16 so that the
// shift (a difference of two such values) is exact in fp32, rescales O and the row sum, and recomputes P from the scores
// shifted by the move.  Lanes whose column does not grow shift by 0 and
// scale by 1.0, which reproduces their P bit for bit, so a query's result
// never depends on the others of its wave.
template <int HD, int QB>
__device__ __forceinline__ void rescale_col(const f32x16 (&s)[2], bool first, int c, float& lsp,
                                            WaveState<HD, QB>& st, f16x8 (&pfc)[2][2], int hi) {
  const bool grow = first || pair_max(lsp) > PMAX;
  float mx = s[0][0];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
  mx = pair_max(mx);
  float shift = 0.f;
  if (grow) {
    const float mnew = (float)(f16)(st.mrow[c] + mx);
    shift = mnew - st.mrow[c];
    st.mrow[c] = mnew;
  }
  const float alpha = first ? 0.f : (grow ? fast_exp2(-shift) : 1.f);
  st.lrow[c] *= alpha;
#pragma unroll
  for (int d = 0; d < HD / 32; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) st.oacc[c][d][r] *= alpha;
  lsp = exp_pack<true>(s[0], s[1], shift, pfc);   // x - 0 = x for the others
#pragma unroll
  for (int r = 0; r < 16; ++r) st.minit[c][r] = -st.mrow[c];
}

// O^T += V^T P^T
template <int HD, int QB>
__device__ __forceinline__ void tile_pv(const uint8_t* Vs, const f16x8 (&pf)[QB][2][2], int r32,
                                        int hi, f32x16 (&oacc)[QB][HD / 32]) {
#pragma unroll
  for (int d = 0; d < HD / 32; ++d) {
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
}

// One iteration of the key loop (tile kv), see k_attention.  LAST masks the
// keys at or past `tail` of the final tile.
template <int HD, int QB, int NW, int K_INSTR, int V_INSTR, bool LAST>
__device__ __forceinline__ void att_iter(uint8_t (*smem)[2 * KV * HD * 2], int kv, int nkv, int tail,
                                         bool lead, __amdgpu_buffer_rsrc_t rk,
                                         __amdgpu_buffer_rsrc_t rv, const uint32_t (&k_off)[K_INSTR],
                                         const uint32_t (&v_off)[V_INSTR], int wave,
                                         const f16x8 (&qf)[QB][HD / 16], int krow, int kswz, int r32,
                                         int hi, WaveState<HD, QB>& st, f32x16 (&s)[2][QB],
                                         f16x8 (&pf)[QB][2][2]) {
  constexpr int K_BYTES = KV * HD * 2;
  // tile kv has landed (this wave's part: vmcnt; the others': the barrier),
  // and every wave is done with the stage tile kv+1 goes to (it held kv-2)
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (!LAST)
    issue_kv<K_INSTR, V_INSTR, K_BYTES, NW>(rk, rv, k_off, v_off, smem[(kv + 1) % 3], wave,
                                            (uint32_t)((kv + 1) * KV * HD * 2),
                                            (uint32_t)((kv + 1) * KV * 2));
  const uint8_t* cur = smem[kv % 3];
  if (lead) {
    tile_scores<HD, QB, minit_in_mfma(QB)>(cur, qf, st.minit, krow, kswz, hi, s);
    if (LAST && tail < KV) mask_tail<QB>(s, tail, hi);
    tile_softmax<HD, QB>(s, kv == 0, st, pf);
    tile_pv<HD, QB>(cur + K_BYTES, pf, r32, hi, st.oacc);
  } else {
    if (kv > 0) tile_pv<HD, QB>(smem[(kv + 2) % 3] + K_BYTES, pf, r32, hi, st.oacc);
    tile_scores<HD, QB, minit_in_mfma(QB)>(cur, qf, st.minit, krow, kswz, hi, s);
    if (LAST && tail < KV) mask_tail<QB>(s, tail, hi);
    tile_softmax<HD, QB>(s, kv == 0, st, pf);
  }
}

// Two wave groups per workgroup, one wave of each on every SIMD, run the same
// work offset by a phase, so that one group's softmax (VALU) overlaps the
// other group's MFMAs.  In iteration j the leading group computes
// scores(j) -> softmax(j) -> P V(j); the trailing group computes P V(j-1) ->
// scores(j) -> softmax(j), carrying its P across the barrier.  Tiles live in
// a 3-stage LDS ring: tile j+1 loads while tile j (both groups) and V of tile
// j-1 (trailing group) are read.
template <int HD, int QB, int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void k_attention(AttnParams p) {
  constexpr int K_BYTES = KV * HD * 2;        // K tile bytes
  constexpr int V_BYTES = HD * KV * 2;        // V^T tile bytes
  constexpr int STAGE = K_BYTES + V_BYTES;
  constexpr int NKK = HD / 16;                // k-steps of the QK^T MFMA
  constexpr int QW = QB * 32;                 // queries per wave
  constexpr int QWG = QW * NW;                // queries per workgroup
  constexpr int K_INSTR = K_BYTES / 1024 / NW;
  constexpr int V_INSTR = V_BYTES / 1024 / NW;
  static_assert(K_INSTR * NW * 1024 == K_BYTES && V_INSTR * NW * 1024 == V_BYTES, "load split");
  static_assert(NW == 8, "one leading and one trailing wave per SIMD");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[3][STAGE];

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
  const bool lead = wave < NW / 2;            // waves w and w + NW/2 share a SIMD
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
  // (the stored queries carry the log2(e)/sqrt(d) factor, so the score MFMA
  // yields the exponent of 2 directly)
  const int q_first = p.q_begin + qb * QWG + wave * QW;
  f16x8 qf[QB][NKK];
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    const int q = min(q_first + c * 32 + r32, (int)Lp - 1);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      qf[c][kk] = *reinterpret_cast<const f16x8*>(Qh + (int64_t)q * HD + kk * 16 + hi * 8);
  }

  WaveState<HD, QB> st;
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    st.mrow[c] = 0.f;
    st.lrow[c] = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) st.minit[c][r] = 0.f;
#pragma unroll
    for (int d = 0; d < HD / 32; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.oacc[c][d][r] = 0.f;
  }

  // fragment addressing inside the tiles
  const int krow = kappa(r32);                      // key row read by this lane
  const int kswz = swz_k<HD>(krow);
  const int nkv = (p.seq_len + KV - 1) / KV;
  const int tail = p.seq_len - (nkv - 1) * KV;      // valid keys in the last tile

  f32x16 s[2][QB];
  f16x8 pf[QB][2][2];     // [column][key block][16-key half]; the trailing group
                          // carries its P across iterations
  issue_kv<K_INSTR, V_INSTR, K_BYTES, NW>(rk, rv, k_off, v_off, smem[0], wave, 0, 0);
  // all tiles but the last have no masked keys; the last is peeled off so that
  // the masking never enters the loop body
  for (int kv = 0; kv < nkv - 1; ++kv)
    att_iter<HD, QB, NW, K_INSTR, V_INSTR, false>(smem, kv, nkv, 0, lead, rk, rv, k_off, v_off, wave,
                                                  qf, krow, kswz, r32, hi, st, s, pf);
  att_iter<HD, QB, NW, K_INSTR, V_INSTR, true>(smem, nkv - 1, nkv, tail, lead, rk, rv, k_off, v_off,
                                               wave, qf, krow, kswz, r32, hi, st, s, pf);
  if (!lead) tile_pv<HD, QB>(smem[(nkv - 1) % 3] + K_BYTES, pf, r32, hi, st.oacc);

  // normalise and store O[b * q_count + (q - q_begin)][h*HD + dim]
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    const int q = q_first + c * 32 + r32;
    const float inv = 1.0f / pair_sum(st.lrow[c]);
    if (q >= p.q_begin + p.q_count) continue;
    f16* orow = p.o + ((int64_t)b * p.q_count + (q - p.q_begin)) * ((int64_t)p.heads * HD) +
                (int64_t)h * HD;
#pragma unroll
    for (int d = 0; d < HD / 32; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (f16)(st.oacc[c][d][4 * g + e] * inv);
        *reinterpret_cast<f16x4*>(orow + d * 32 + 8 * g + 4 * hi) = o;
      }
  }
}

// One key tile of k_attention_lazy (tile kv in stage kv & 1; the next tile
// is loaded into the other stage meanwhile).  LAST masks the keys at or past
// `tail` and loads nothing.  The two query columns run offset: the score
// MFMAs of column 1 are issued beside the exponentials of column 0, and the
// P V^T MFMAs of column 0 beside those of column 1 (their V^T fragments are
// kept for column 1).  Each column keeps its own order of operations.
template <int HD, int QB, int NW, int K_INSTR, int V_INSTR, bool LAST>
__device__ __forceinline__ void lazy_iter(uint8_t (*smem)[2 * KV * HD * 2], int kv, int tail,
                                          __amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                          const uint32_t (&k_off)[K_INSTR],
                                          const uint32_t (&v_off)[V_INSTR], int wave,
                                          const f16x8 (&qf)[QB][HD / 16], int krow, int kswz,
                                          int r32, int hi, WaveState<HD, QB>& st) {
  static_assert(QB == 2, "two query column blocks per wave");
  constexpr int K_BYTES = KV * HD * 2;
  const int stage = kv & 1;
  if (!LAST)
    issue_kv<K_INSTR, V_INSTR, K_BYTES, NW>(rk, rv, k_off, v_off, smem[stage ^ 1], wave,
                                            (uint32_t)((kv + 1) * KV * HD * 2),
                                            (uint32_t)((kv + 1) * KV * 2));
  const uint8_t* Ks = smem[stage];
  const uint8_t* Vs = smem[stage] + K_BYTES;
  const bool first = kv == 0;
  f32x16 s0[2], s1[2];
  f16x8 pf[QB][2][2];
  // the score MFMAs at a raised wave priority, so that the other wave of the
  // SIMD fills their shadow with its exponentials (1% faster; the P V^T
  // MFMAs raised too measured slower)
  __builtin_amdgcn_s_setprio(2);
  scores_col<HD>(Ks, qf[0], st.minit[0], krow, kswz, hi, s0);
  if (LAST && tail < KV) mask_tail_col(s0, tail, hi);
  scores_col<HD>(Ks, qf[1], st.minit[1], krow, kswz, hi, s1);
  __builtin_amdgcn_s_setprio(0);
  float lsp0 = exp_pack<false>(s0[0], s0[1], 0.f, pf[0]);
  if (__builtin_amdgcn_ballot_w64(first || lsp0 > PMAX))
    rescale_col<HD, QB>(s0, first, 0, lsp0, st, pf[0], hi);
  if (LAST && tail < KV) mask_tail_col(s1, tail, hi);
  f16x8 vf[HD / 32][2][2];
#pragma unroll
  for (int d = 0; d < HD / 32; ++d) {
    const int vrow = d * 32 + r32;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int slot16 = (kb * 4 + u * 2 + hi) ^ swz_v(vrow);
        vf[d][kb][u] = *reinterpret_cast<const f16x8*>(Vs + vrow * (KV * 2) + slot16 * 16);
        st.oacc[0][d] = mma(vf[d][kb][u], pf[0][kb][u], st.oacc[0][d]);
      }
  }
  float lsp1 = exp_pack<false>(s1[0], s1[1], 0.f, pf[1]);
  if (__builtin_amdgcn_ballot_w64(first || lsp1 > PMAX))
    rescale_col<HD, QB>(s1, first, 1, lsp1, st, pf[1], hi);
#pragma unroll
  for (int d = 0; d < HD / 32; ++d)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int u = 0; u < 2; ++u) st.oacc[1][d] = mma(vf[d][kb][u], pf[1][kb][u], st.oacc[1][d]);
  st.lrow[0] += lsp0;
  st.lrow[1] += lsp1;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Variant for narrow heads (d = 64): no group offset, two query column
// blocks per wave (halving the LDS reads per score), a two-stage ring, the
// reference max subtracted by the score MFMA and the P-sum trigger
// evaluated on the common path's own exponentials.  Measured faster than
// k_attention at d = 64, slower at d = 128.
template <int HD, int QB, int NW>
__global__ __launch_bounds__(NW * 64) void k_attention_lazy(AttnParams p) {
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

  WaveState<HD, QB> st;
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    st.mrow[c] = 0.f;
    st.lrow[c] = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) st.minit[c][r] = 0.f;
#pragma unroll
    for (int d = 0; d < NDB; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.oacc[c][d][r] = 0.f;
  }

  // fragment addressing inside the tiles
  const int krow = kappa(r32);                      // key row read by this lane
  const int kswz = swz_k<HD>(krow);
  const int nkv = (p.seq_len + KV - 1) / KV;
  const int tail = p.seq_len - (nkv - 1) * KV;      // valid keys in the last tile

  issue_kv<K_INSTR, V_INSTR, K_BYTES, NW>(rk, rv, k_off, v_off, smem[0], wave, 0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // the last tile, the only one with masked keys, is peeled off the loop
  for (int kv = 0; kv < nkv - 1; ++kv)
    lazy_iter<HD, QB, NW, K_INSTR, V_INSTR, false>(smem, kv, 0, rk, rv, k_off, v_off, wave, qf, krow,
                                                   kswz, r32, hi, st);
  lazy_iter<HD, QB, NW, K_INSTR, V_INSTR, true>(smem, nkv - 1, tail, rk, rv, k_off, v_off, wave, qf,
                                                krow, kswz, r32, hi, st);

  // normalise and store O[b * q_count + (q - q_begin)][h*HD + dim]
#pragma unroll
  for (int c = 0; c < QB; ++c) {
    const int q = q_first + c * 32 + r32;
    const float inv = 1.0f / pair_sum(st.lrow[c]);
    if (q >= p.q_begin + p.q_count) continue;
    f16* orow = p.o + ((int64_t)b * p.q_count + (q - p.q_begin)) * ((int64_t)p.heads * HD) +
                (int64_t)h * HD;
#pragma unroll
    for (int d = 0; d < NDB; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (f16)(st.oacc[c][d][4 * g + e] * inv);
        *reinterpret_cast<f16x4*>(orow + d * 32 + 8 * g + 4 * hi) = o;
      }
  }
}

template <int HD, int QB, int NW, bool LAZY>
static hipError_t launch_t(const AttnParams& p, hipStream_t s) {
  constexpr int QWG = QB * 32 * NW;
  const int64_t nqb = (p.q_count + QWG - 1) / QWG;
  const int64_t total = nqb * p.heads * p.batch;
  if (total == 0) return hipSuccess;
  if constexpr (LAZY)
    hipLaunchKernelGGL((k_attention_lazy<HD, QB, NW>), dim3((unsigned)total), dim3(NW * 64), 0, s, p);
  else
    hipLaunchKernelGGL((k_attention<HD, QB, NW>), dim3((unsigned)total), dim3(NW * 64), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnParams& p, int head_dim, hipStream_t s) {
  if (head_dim == 64) return launch_t<64, 2, 8, true>(p, s);
  if (head_dim == 128) return launch_t<128, 1, 8, false>(p, s);
  return hipErrorInvalidValue;
}

}  // namespace xema
