// Shared device-side helpers for the gfx950 (CDNA4) kernels of the
// fine-tuning step: bf16 storage type, vector types for the MFMA operands,
// wavefront reductions and the launch-error plumbing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define SAT_WAVE 64

__device__ __forceinline__ float bf2f(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }

// Sum / max over the 64 lanes of a wavefront (butterfly through DPP-capable
// shuffles; every lane receives the result).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, SAT_WAVE);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, SAT_WAVE));
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, SAT_WAVE);
  return v;
}

// GELU, tanh approximation and exact erf form, and their derivatives.
// tanh(y) is evaluated as 1 - 2 / (exp(2y) + 1) with the hardware base-2
// exponential and reciprocal (about 1 ulp each), which saturates correctly at
// both ends (exp overflow gives 1, underflow gives -1).
__device__ __forceinline__ float tanh_fast(float y) {
  return 1.f - 2.f * __builtin_amdgcn_rcpf(__builtin_amdgcn_exp2f(2.8853900817779268f * y) + 1.f);
}
__device__ __forceinline__ float gelu_tanh_f(float x) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  float t = tanh_fast(c * (x + a * x * x * x));
  return 0.5f * x * (1.f + t);
}
__device__ __forceinline__ float gelu_tanh_grad_f(float x) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  float t = tanh_fast(c * (x + a * x * x * x));
  return 0.5f * (1.f + t) + 0.5f * x * (1.f - t * t) * c * (1.f + 3.f * a * x * x);
}
__device__ __forceinline__ float gelu_erf_f(float x) {
  return 0.5f * x * (1.f + erff(x * 0.7071067811865476f));
}
__device__ __forceinline__ float gelu_erf_grad_f(float x) {
  float cdf = 0.5f * (1.f + erff(x * 0.7071067811865476f));
  float pdf = 0.3989422804014327f * __expf(-0.5f * x * x);
  return cdf + x * pdf;
}
__device__ __forceinline__ float gelu_f(float x, int erf_form) {
  return erf_form ? gelu_erf_f(x) : gelu_tanh_f(x);
}
__device__ __forceinline__ float gelu_grad_f(float x, int erf_form) {
  return erf_form ? gelu_erf_grad_f(x) : gelu_tanh_grad_f(x);
}
template <int ERF>
__device__ __forceinline__ float gelu_t(float x) {
  return ERF ? gelu_erf_f(x) : gelu_tanh_f(x);
}
template <int ERF>
__device__ __forceinline__ float gelu_grad_t(float x) {
  return ERF ? gelu_erf_grad_f(x) : gelu_tanh_grad_f(x);
}

static inline int sat_cdiv(long a, long b) { return (int)((a + b - 1) / b); }
