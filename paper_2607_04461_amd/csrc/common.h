// Internal device/host helpers shared by the library's HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

namespace fb {

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// tanh-form GELU in fp32: 0.5 x (1 + tanh(u)), u = sqrt(2/pi) (x + 0.044715 x^3).  Since
// 0.5 (1 + tanh u) = 1 / (1 + exp(-2u)), it is x / (1 + 2^(-x (a + b x^2))) with
// a = 2 sqrt(2/pi) log2(e) and b = 0.044715 a: one hardware exp2 and one hardware reciprocal
// (about 1 ulp each) instead of an IEEE division.  Saturates cleanly: the exp2 overflows to +inf
// for large negative x (result -0) and underflows to 0 for large positive x (result x).
__device__ __forceinline__ float gelu_tanh(float x) {
  const float a = 2.302208198f;            // 2 sqrt(2/pi) / ln 2
  const float b = 0.1029432396f;           // 0.044715 a
  const float e = __builtin_amdgcn_exp2f(-x * fmaf(b, x * x, a));
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

// wave64 reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

}  // namespace fb
