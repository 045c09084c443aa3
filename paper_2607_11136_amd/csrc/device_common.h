// Device-side helpers for the gfx950 kernels of libxema.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xema {

typedef _Float16 f16;
typedef __bf16 bf16;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// LDS address-space pointer, as taken by the direct global->LDS load builtin.
typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(f16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }
template <>
__device__ __forceinline__ f16 from_f32<f16>(float x) { return (f16)x; }
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }

// x as an fp32 register value: the empty asm keeps the compiler from merging
// the operation that produced x into a following fp16 conversion (a mixed
// multiply-add rounds once, the operation then the conversion round twice),
// which it may do in one instantiation of a kernel and not in another.
__device__ __forceinline__ float as_rounded_f32(float x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Whether v rounds to a finite fp16 value: |v| < 65520 (values from 65504
// up round to 65504, from 65520 on to infinity); false for NaN.
__device__ __forceinline__ bool fits_f16(float v) { return __builtin_fabsf(v) < 65520.0f; }

// Range flag: the lanes that saw a value outside the fp16 range store 1 to
// the flag word (a plain vector store; every writer stores the same value).
__device__ __forceinline__ void raise_flag(uint32_t* flag, bool bad) {
  if (flag != nullptr && bad) *(volatile uint32_t*)flag = 1u;
}

// Butterfly sum over the 64 lanes of a wave (fixed pairing order, so every
// lane ends with the same, run-to-run reproducible value).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// GELU, tanh form: 0.5 u (1 + tanh(a (u + 0.044715 u^3))), a = sqrt(2/pi).
// Since 0.5 (1 + tanh(z)) = 1 / (1 + e^(-2z)), this is u / (1 + 2^(-2 z log2 e)),
// taken with the hardware exp2 and reciprocal (about 1 ulp each).  Large |u|
// gives 2^(+inf) -> 1/inf = 0 or 2^(-inf) -> 1/1 = 1, so no NaN appears.
__device__ __forceinline__ float gelu_tanh(float u) {
  const float c = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 a log2(e)
  const float e = __builtin_amdgcn_exp2f(c * fmaf(0.044715f * u, u * u, u));
  return u * __builtin_amdgcn_rcpf(1.0f + e);
}

}  // namespace xema
