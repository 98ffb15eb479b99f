// Shared device-side helpers for the gfx950 (CDNA4) kernels of the
// fine-tuning step: bf16 storage type, vector types for the MFMA operands,
// wavefront reductions, explicit waits and barriers, and the launch-error
// plumbing.
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

// Explicit waits.  A wave's vmcnt counts its vector loads, stores and LDS
// copies in issue order; the compiler's own waits are only as precise as its
// view of that order, so the pipelined kernels wait for exactly what they
// need.  The encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8.
// s_waitcnt vmcnt(VM) lgkmcnt(0): at most VM vector memory operations of the
// wave still in flight, every LDS and scalar memory operation done.
template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4));
}
// s_waitcnt lgkmcnt(0) only: vector memory operations may stay in flight.
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xF | (3 << 14) | (7 << 4)); }
// Workgroup barrier with no implied wait: __syncthreads' fence would also
// wait for every vector load in flight (the next block's copies, the next
// row's loads).  Callers wait for what the barrier publishes first; the
// scheduling barriers keep the compiler from moving work across it.
__device__ __forceinline__ void cta_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_sched_barrier(0);
}

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

// GELU, tanh approximation and erf form, and their derivatives.
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
// 1 + erf(z) for the erf-form GELU, from Abramowitz & Stegun 7.1.26
// (Hastings' rational approximation): erfc(|z|) ~= q = t P(t) exp(-z^2),
// t = 1 / (1 + p |z|), absolute error at most 1.5e-7.  For z < 0 the result
// is q itself, so the negative tail keeps its relative accuracy (no
// cancellation in 1 + erf).  exp(-z^2) is returned as well: at
// z = x / sqrt(2) it is the Gaussian density factor of GELU'.
__device__ __forceinline__ float one_plus_erf(float z, float& ez2) {
  const float az = fabsf(z);
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, az, 1.f));
  const float poly =
      t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  ez2 = __builtin_amdgcn_exp2f(-1.4426950408889634f * az * az);
  const float q = poly * ez2;
  return z >= 0.f ? 2.f - q : q;
}
__device__ __forceinline__ float gelu_erf_f(float x) {
  float e;
  return 0.5f * x * one_plus_erf(x * 0.7071067811865476f, e);
}
__device__ __forceinline__ float gelu_erf_grad_f(float x) {
  float e;
  const float cdf = 0.5f * one_plus_erf(x * 0.7071067811865476f, e);
  return cdf + x * (0.3989422804014327f * e);
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
