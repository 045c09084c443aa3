// The VAE decoder's upsampling stage, fused: nearest 2x upsampling followed
// by a 3x3 convolution (zero padding 1, bias), computed straight from the
// low-resolution input so the 4x larger upsampled image never exists.  The
// paper fuses the operators around VAE upsampling to cut its short-lived
// activation peak (Sec. 5.2, "Localized chunking and fusion"; Sec. 8, memory
// mitigation primitives).
//
// Phase form.  Output pixel (2i + py, 2j + px) sees the upsampled rows
// 2i+py-1 .. 2i+py+1, which are the source rows i+py-1 and i+py (two of the
// three kernel rows fall on the same source row), and likewise for columns.
// So each of the four output phases (py, px) is a 2x2 convolution of the
// zero-padded input with weights summed over the kernel taps that land on the
// same source pixel:
//   source offset a = 0, 1 takes kernel rows {0} and {1, 2} when py = 0,
//   and {0, 1} and {2} when py = 1 (the same for columns with px).
// k_upconv_prep forms the summed weights once per layer as fp32 sums and
// keeps each as a pair of bf16 values, hi = the sum rounded to bf16 and lo =
// the remainder rounded to bf16, which together carry it to about 2^-17 of
// its size: both are applied, so no rounding of the weights departs from the
// definition beyond fp32 accumulation.  That is 32 C_in C_out multiply-adds
// per input pixel (four phases, four taps, hi and lo) against the 36 of the
// convolution over the upsampled image.
//
// Each phase is an implicit GEMM: M = the phase's output pixels, N = C_out,
// K = 8 x C_in (the four taps with their hi weights, then the four taps with
// their lo weights), with the A rows gathered from the input by tap.  Tiling
// and pipeline follow k_gemm: 256 x 256 tiles, K steps of 64 channels of one
// tap, two LDS stages filled by buffer_load ... lds, eight waves of 32x32x16
// MFMAs.  A tap that falls outside the image (or a row past M) is issued at an
// offset with bit 31 set, beyond the buffer's range, so it reads zeros.  The
// four phases of a tile run next to each other on one XCD and share its L2.
//
// Determinism: every output element sums its taps in a fixed order (the hi
// taps, then the lo taps, tap-major, channels ascending, one MFMA per 16
// channels), whatever rows a call covers, so a stage computed in row bands
// equals the stage computed at once.
#include "device_common.h"
#include "kernels.h"

namespace xema {

namespace {

constexpr int UBM = 256, UBN = 256, UBK = 64;
constexpr int UKS = UBK / 16;             // MFMA k-steps per stage
constexpr int UROWB = UBK * 2;            // bytes of one operand row in a stage
constexpr int USLOTS = UBK / 8;           // 16-byte slots per row
constexpr int URPL = 1024 / UROWB;        // rows filled by one 1 KiB wave load
constexpr int UNWAVES = 8;
constexpr int UWN = UBN * 2 / UNWAVES;    // output columns per wave (64)
constexpr int UMI = UBM / 64, UNJ = UWN / 32;
constexpr int UA_BYTES = UBM * UBK * 2, UB_BYTES = UBN * UBK * 2;
constexpr int UA_LOADS = UBM / UNWAVES / URPL, UB_LOADS = UBN / UNWAVES / URPL;
constexpr int ULPS = UA_LOADS + UB_LOADS;
constexpr int UGROUP_M = 8;

__host__ __device__ constexpr int swz(int r) { return (r >> 1) & 7; }
constexpr int vm_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ void barrier_all() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(vm_imm(0));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

}  // namespace

// The phase-summed weights: s = the sum of w[o][ky][kx][c] over the kernel
// taps (ky, kx) of phase p = 2 py + px that land on source offset t = 2 a +
// b, in fp32 in ascending (ky, kx); wp[p][o][t][c] = hi = bf16(s) and
// wp[p][o][4 + t][c] = bf16(s - hi) (s - hi is exact in fp32).  One thread
// per (p, o, t, c) writes both.
__global__ void k_upconv_prep(const uint16_t* __restrict__ w, int ci, int co, uint16_t* __restrict__ wp) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)16 * co * ci;
  if (idx >= total) return;
  const int c = (int)(idx % ci);
  const int t = (int)((idx / ci) % 4);
  const int o = (int)((idx / ((int64_t)4 * ci)) % co);
  const int p = (int)(idx / ((int64_t)4 * ci * co));
  const int py = p >> 1, px = p & 1, a = t >> 1, b = t & 1;
  // kernel rows landing on source offset a: py = 0: {0} | {1, 2}; py = 1: {0, 1} | {2}
  const int r0 = (py == 0) ? (a == 0 ? 0 : 1) : (a == 0 ? 0 : 2);
  const int r1 = (py == 0) ? (a == 0 ? 0 : 2) : (a == 0 ? 1 : 2);
  const int c0 = (px == 0) ? (b == 0 ? 0 : 1) : (b == 0 ? 0 : 2);
  const int c1 = (px == 0) ? (b == 0 ? 0 : 2) : (b == 0 ? 1 : 2);
  float s = 0.f;
  for (int ky = r0; ky <= r1; ++ky)
    for (int kx = c0; kx <= c1; ++kx) s += bf16_bits_to_f32(w[(((int64_t)o * 3 + ky) * 3 + kx) * ci + c]);
  const bf16 hi = (bf16)s;
  const bf16 lo = (bf16)(s - (float)hi);
  uint16_t* row = wp + (((int64_t)p * co + o) * 8) * ci;
  row[(int64_t)t * ci + c] = __builtin_bit_cast(uint16_t, hi);
  row[(int64_t)(4 + t) * ci + c] = __builtin_bit_cast(uint16_t, lo);
}

__global__ __launch_bounds__(UNWAVES * 64, 1) void k_upconv(UpconvParams p) {
  typedef bf16x8 frag;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2][UA_BYTES + UB_BYTES];

  const int ci = p.ci, co = p.co, W = p.w, H = p.h;
  const int KT = 8 * ci / UBK;             // K steps: (4 hi + 4 lo taps) x ci / 64
  const int cpt = ci / UBK;                // K steps per tap
  const int64_t M = (int64_t)p.n * p.row_count * W;   // output pixels of one phase
  const int tiles_m = (int)((M + UBM - 1) / UBM);
  const int tiles_n = co / UBN;
  const int total = tiles_m * tiles_n * 4;
  // XCD-aware order: each XCD walks a contiguous range; the four phases of a
  // tile are consecutive, then tiles in groups of UGROUP_M tile-rows
  const int wg = blockIdx.x;
  const int xcd = wg & 7, slot = wg >> 3;
  const int per = total >> 3, rem = total & 7;
  const int t = xcd * per + min(xcd, rem) + slot;
  const int phase = t & 3, tile = t >> 2;
  const int group = tile / (UGROUP_M * tiles_n);
  const int first_m = group * UGROUP_M;
  const int gsize = min(tiles_m - first_m, UGROUP_M);
  const int in_group = tile - group * UGROUP_M * tiles_n;
  const int tm = first_m + in_group % gsize;
  const int tn = in_group / gsize;
  const int64_t m0 = (int64_t)tm * UBM;
  const int n0 = tn * UBN;
  const int py = phase >> 1, px = phase & 1;

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / (UBN / UWN), wn = wave % (UBN / UWN);

  const __amdgpu_buffer_rsrc_t ra = rsrc(p.x, (int64_t)p.n * H * W * ci * 2);
  const uint16_t* wph = p.wp + ((int64_t)phase * co + n0) * 8 * ci;
  const __amdgpu_buffer_rsrc_t rb = rsrc(wph, (int64_t)UBN * 8 * ci * 2);

  // A rows: load c of this wave fills tile rows (wave*UA_LOADS + c)*URPL +
  // lane/USLOTS; each row is one output pixel (frame f, source row i, column
  // j) of this phase.  a_base holds the byte offset of the lane's 16 bytes in
  // the source pixel of tap (0, 0), i.e. (i + py - 1, j + px - 1), taken
  // modulo 2^32 (it may sit before the buffer: only valid taps are used);
  // a_valid has bit t set when tap t = 2a + b lies inside the image.
  uint32_t a_base[UA_LOADS];
  uint32_t a_valid[UA_LOADS];
#pragma unroll
  for (int c = 0; c < UA_LOADS; ++c) {
    const int row = (wave * UA_LOADS + c) * URPL + lane / USLOTS;
    const int64_t m = m0 + row;
    const int64_t frame = m / ((int64_t)p.row_count * W);
    const int64_t r = m - frame * p.row_count * W;
    const int i = p.row_begin + (int)(r / W), j = (int)(r % W);
    uint32_t v = 0;
#pragma unroll
    for (int tap = 0; tap < 4; ++tap) {
      const int si = i + py + (tap >> 1) - 1, sj = j + px + (tap & 1) - 1;
      if (m < M && si >= 0 && si < H && sj >= 0 && sj < W) v |= 1u << tap;
    }
    a_valid[c] = v;
    const int64_t pix = ((int64_t)frame * H + (i + py - 1)) * W + (j + px - 1);
    a_base[c] = (uint32_t)(pix * ci * 2 + ((lane % USLOTS) ^ swz(row)) * 16);
  }
  uint32_t b_off[UB_LOADS];
#pragma unroll
  for (int c = 0; c < UB_LOADS; ++c) {
    const int row = (wave * UB_LOADS + c) * URPL + lane / USLOTS;
    b_off[c] = (uint32_t)(row * 8 * ci * 2 + ((lane % USLOTS) ^ swz(row)) * 16);
  }

  auto issue = [&](int kt, int idx) {
    uint8_t* st = smem[kt & 1];
    if (idx < UA_LOADS) {
      const int tap = kt / cpt;                       // 0-3 hi, 4-7 lo, >= 8 past the last step
      const int src = tap & 3;                        // the source offset both weights apply to
      const uint32_t cbyte = (uint32_t)((kt - tap * cpt) * UBK * 2);
      const uint32_t tdelta = (uint32_t)((((src >> 1) * W) + (src & 1)) * ci * 2);
      const uint32_t valid = tap < 8 ? (a_valid[idx] >> src) & 1u : 0u;
      const uint32_t oob = (valid ^ 1u) << 31;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(st + (wave * UA_LOADS + idx) * 1024), 16,
                                               (a_base[idx] + tdelta + cbyte) | oob, 0, 0, 0);
    } else {
      const int c = idx - UA_LOADS;
      const uint32_t oob = (uint32_t)((KT - 1 - kt) >> 31) << 31;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr_t)(st + UA_BYTES + (wave * UB_LOADS + c) * 1024),
                                               16, (b_off[c] + (uint32_t)(kt * UBK * 2)) | oob, 0, 0, 0);
    }
  };

  f32x16 acc[UMI][UNJ];
#pragma unroll
  for (int i = 0; i < UMI; ++i)
#pragma unroll
    for (int j = 0; j < UNJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int r32 = lane & 31, hi = lane >> 5, sw = swz(r32);
  const int a_row0 = (wm * (UBM / 2) + r32) * UROWB;
  const int b_row0 = (wn * UWN + r32) * UROWB;
  frag fx[2][UMI], fw[2][UNJ];
  auto read_one = [&](const uint8_t* st, int kk, int f, frag (&x)[UMI], frag (&wv)[UNJ]) {
    const int so = (((kk * 2 + hi) ^ sw) * 16);
    if (f < UMI)
      x[f] = *reinterpret_cast<const frag*>(st + a_row0 + f * 32 * UROWB + so);
    else
      wv[f - UMI] = *reinterpret_cast<const frag*>(st + UA_BYTES + b_row0 + (f - UMI) * 32 * UROWB + so);
  };
  auto mfma_step = [&](const frag (&x)[UMI], const frag (&wv)[UNJ]) {
#pragma unroll
    for (int i = 0; i < UMI; ++i)
#pragma unroll
      for (int j = 0; j < UNJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv[j], x[i], acc[i][j], 0, 0, 0);
  };
  constexpr int NR = UMI + UNJ, NM = UMI * UNJ;

  // The pipeline of k_gemm: step kt is consumed from stage kt & 1; the
  // barrier before its last k-step means step kt is fully read and step kt+1
  // has landed; a step's loads go out in two halves over the two k-steps
  // after the barrier that frees its stage.
  constexpr int H1 = ULPS / 2;
#pragma unroll
  for (int l = 0; l < ULPS; ++l) issue(0, l);
  barrier_all();
#pragma unroll
  for (int f = 0; f < NR; ++f) read_one(smem[0], 0, f, fx[0], fw[0]);
#pragma unroll
  for (int l = 0; l < H1; ++l) issue(1, l);
  for (int kt = 0; kt < KT; ++kt) {
    const uint8_t* st = smem[kt & 1];
#pragma unroll
    for (int kk = 0; kk < UKS - 1; ++kk) {
      const int nl = kk == 0 ? ULPS - H1 : 0;
      const int ne = NR > nl ? NR : nl;
#pragma unroll
      for (int e = 0; e < ne; ++e) {
        if (e < NR) read_one(st, kk + 1, e, fx[(kk + 1) & 1], fw[(kk + 1) & 1]);
        if (e < nl) issue(kt + 1, H1 + e);
      }
      mfma_step(fx[kk & 1], fw[kk & 1]);
      const int ng = NM > ne ? NM : ne;
#pragma unroll
      for (int g = 0; g < ng; ++g) {
        if (g < NM) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (g < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        if (g < nl) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    }
    barrier_all();
    const int ne = NR > H1 ? NR : H1;
#pragma unroll
    for (int e = 0; e < ne; ++e) {
      if (e < NR) read_one(smem[(kt + 1) & 1], 0, e, fx[UKS & 1], fw[UKS & 1]);
      if (e < H1) issue(kt + 2, e);
    }
    mfma_step(fx[(UKS - 1) & 1], fw[(UKS - 1) & 1]);
    const int ng = NM > ne ? NM : ne;
#pragma unroll
    for (int g = 0; g < ng; ++g) {
      if (g < NM) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (g < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (g < H1) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
  }
  __builtin_amdgcn_s_waitcnt(vm_imm(0));

  // Epilogue: acc[i][j][r] is output channel n0 + wn*64 + j*32 + 8*(r/4) +
  // 4*hi + r%4 of the phase's pixel m0 + wm*128 + i*32 + r32, which is output
  // pixel (frame, 2 i_src + py, 2 j_src + px).  Bias, one bf16 rounding, 8-byte stores.
  float bv[UNJ][4][4];
#pragma unroll
  for (int j = 0; j < UNJ; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const u32x2 u = *reinterpret_cast<const u32x2*>(p.bias + n0 + wn * UWN + j * 32 + 8 * q + 4 * hi);
      bv[j][q][0] = __uint_as_float(u[0] << 16);
      bv[j][q][1] = __uint_as_float(u[0] & 0xffff0000u);
      bv[j][q][2] = __uint_as_float(u[1] << 16);
      bv[j][q][3] = __uint_as_float(u[1] & 0xffff0000u);
    }
#pragma unroll
  for (int i = 0; i < UMI; ++i) {
    const int64_t m = m0 + wm * (UBM / 2) + i * 32 + r32;
    if (m >= M) continue;
    const int64_t frame = m / ((int64_t)p.row_count * W);
    const int64_t r = m - frame * p.row_count * W;
    const int64_t oy = 2 * (p.row_begin + r / W) + py, ox = 2 * (r % W) + px;
    uint16_t* yrow = p.y + ((frame * 2 * H + oy) * 2 * W + ox) * co;
#pragma unroll
    for (int j = 0; j < UNJ; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (bf16)(acc[i][j][4 * q + e] + bv[j][q][e]);
        *reinterpret_cast<bf16x4*>(yrow + n0 + wn * UWN + j * 32 + 8 * q + 4 * hi) = o;
      }
  }
}

hipError_t launch_upconv_prep(const uint16_t* w, int ci, int co, uint16_t* wp, hipStream_t s) {
  const int64_t total = (int64_t)16 * co * ci;
  hipLaunchKernelGGL(k_upconv_prep, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, w, ci, co, wp);
  return hipGetLastError();
}

hipError_t launch_upconv(const UpconvParams& p, hipStream_t s) {
  const int64_t M = (int64_t)p.n * p.row_count * p.w;
  const int64_t tiles = ((M + UBM - 1) / UBM) * (p.co / UBN) * 4;
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(k_upconv, dim3((unsigned)tiles), dim3(UNWAVES * 64), 0, s, p);
  return hipGetLastError();
}

}  // namespace xema
