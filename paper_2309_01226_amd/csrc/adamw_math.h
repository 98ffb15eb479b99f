// One AdamW step on fp32 values (decoupled weight decay, bias-corrected
// moments), shared by the flat / segment-table AdamW kernels and the GEMM
// epilogue that applies the update to a weight as its gradient is formed.
// The constants are formed on the host in double precision (kernels.h).
#pragma once

#include "common.h"
#include "kernels.h"

// No contraction into fused multiply-adds: the separate pass and the GEMM
// epilogue must round identically, whatever code surrounds each call.
__device__ __forceinline__ void adamw_one(float& p, float g, float& m, float& v,
                                          const AdamWConsts& c) {
#pragma clang fp contract(off)
  p = p - c.lr_wd * p;
  m = c.b1 * m + c.omb1 * g;
  v = c.b2 * v + c.omb2 * g * g;
  p = p - c.step * m / (sqrtf(v) / c.bc2s + c.eps);
}

__device__ __forceinline__ void adamw_four(floatx4& p, floatx4 g, floatx4& m, floatx4& v,
                                           const AdamWConsts& c) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float pe = p[e], me = m[e], ve = v[e];
    adamw_one(pe, g[e], me, ve, c);
    p[e] = pe;
    m[e] = me;
    v[e] = ve;
  }
}
