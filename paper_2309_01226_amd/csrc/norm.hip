// LayerNorm forward / backward and deterministic column reductions.
//
// One wavefront owns one row (rows up to 8192 wide stay in registers as
// float4 chunks, 256 columns per chunk); mean and variance are two-pass
// wave reductions over the register copy, so x is read from HBM once.
// Gain / shift gradients are reduced without atomics: each wave accumulates
// the columns of a fixed, strided set of rows into a partial row, and a second
// kernel sums the partial rows in a fixed order (bitwise reproducible).
#include "common.h"
#include "kernels.h"

namespace {

constexpr int LN_MAXC = 32;  // float4 chunks per lane: d <= 64 * 4 * 32 = 8192

template <int NC>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const float* __restrict__ x, long ldx,
                                                     long row_stride, const float* __restrict__ g,
                                                     const float* __restrict__ b, bf16* __restrict__ y,
                                                     long ldy, float* __restrict__ mean,
                                                     float* __restrict__ rstd, int rows, int d,
                                                     float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float* xr = x + (long)row * row_stride * ldx;
  float4 v[NC];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    int col = (c * 64 + lane) * 4;
    if (col < d) v[c] = *reinterpret_cast<const float4*>(xr + col);
    else v[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    s += v[c].x + v[c].y + v[c].z + v[c].w;
  }
  const float mu = wave_sum(s) / d;
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    int col = (c * 64 + lane) * 4;
    if (col < d) {
      float a0 = v[c].x - mu, a1 = v[c].y - mu, a2 = v[c].z - mu, a3 = v[c].w - mu;
      q += a0 * a0 + a1 * a1 + a2 * a2 + a3 * a3;
    }
  }
  const float rs = rsqrtf(wave_sum(q) / d + eps);
  bf16* yr = y + (long)row * ldy;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    int col = (c * 64 + lane) * 4;
    if (col < d) {
      float4 gg = *reinterpret_cast<const float4*>(g + col);
      float4 bb = *reinterpret_cast<const float4*>(b + col);
      bf16x4 o;
      o[0] = f2bf((v[c].x - mu) * rs * gg.x + bb.x);
      o[1] = f2bf((v[c].y - mu) * rs * gg.y + bb.y);
      o[2] = f2bf((v[c].z - mu) * rs * gg.z + bb.z);
      o[3] = f2bf((v[c].w - mu) * rs * gg.w + bb.w);
      *reinterpret_cast<bf16x4*>(yr + col) = o;
    }
  }
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

// Each wave handles rows w, w + n_part, w + 2 n_part, ... (w = global wave id
// < n_part) and keeps per-column partial sums of dy * xhat and dy in registers.
// A row is read twice (row statistics, then dx); the second read hits cache.
template <int NC>
__global__ __launch_bounds__(256) void ln_bwd_kernel(
    const float* __restrict__ dy, long lddy, const float* __restrict__ x, long ldx,
    long row_stride, const float* __restrict__ g, const float* __restrict__ mean,
    const float* __restrict__ rstd, float* __restrict__ dres, long ldres,
    float* __restrict__ part_g, float* __restrict__ part_b, int rows, int d, int n_part) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= n_part) return;
  float4 pg[NC], pb[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    pg[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    pb[c] = pg[c];
  }
  for (int row = w; row < rows; row += n_part) {
    const float* dyr = dy + (long)row * lddy;
    const float* xr = x + (long)row * row_stride * ldx;
    float* dr = dres + (long)row * row_stride * ldres;
    const float mu = mean[row], rs = rstd[row];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      int col = (c * 64 + lane) * 4;
      if (col < d) {
        float4 dv = *reinterpret_cast<const float4*>(dyr + col);
        float4 xv = *reinterpret_cast<const float4*>(xr + col);
        float4 gg = *reinterpret_cast<const float4*>(g + col);
        float4 xh = make_float4((xv.x - mu) * rs, (xv.y - mu) * rs, (xv.z - mu) * rs, (xv.w - mu) * rs);
        float4 gy = make_float4(dv.x * gg.x, dv.y * gg.y, dv.z * gg.z, dv.w * gg.w);
        pg[c].x += dv.x * xh.x; pg[c].y += dv.y * xh.y;
        pg[c].z += dv.z * xh.z; pg[c].w += dv.w * xh.w;
        pb[c].x += dv.x; pb[c].y += dv.y; pb[c].z += dv.z; pb[c].w += dv.w;
        s1 += gy.x + gy.y + gy.z + gy.w;
        s2 += gy.x * xh.x + gy.y * xh.y + gy.z * xh.z + gy.w * xh.w;
      }
    }
    const float m1 = wave_sum(s1) / d, m2 = wave_sum(s2) / d;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      int col = (c * 64 + lane) * 4;
      if (col < d) {
        float4 dv = *reinterpret_cast<const float4*>(dyr + col);
        float4 xv = *reinterpret_cast<const float4*>(xr + col);
        float4 gg = *reinterpret_cast<const float4*>(g + col);
        float4 o = *reinterpret_cast<float4*>(dr + col);
        o.x += rs * (dv.x * gg.x - m1 - (xv.x - mu) * rs * m2);
        o.y += rs * (dv.y * gg.y - m1 - (xv.y - mu) * rs * m2);
        o.z += rs * (dv.z * gg.z - m1 - (xv.z - mu) * rs * m2);
        o.w += rs * (dv.w * gg.w - m1 - (xv.w - mu) * rs * m2);
        *reinterpret_cast<float4*>(dr + col) = o;
      }
    }
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    int col = (c * 64 + lane) * 4;
    if (col < d) {
      *reinterpret_cast<float4*>(part_g + (long)w * d + col) = pg[c];
      *reinterpret_cast<float4*>(part_b + (long)w * d + col) = pb[c];
    }
  }
}

__global__ void colsum_partials_kernel(const float* __restrict__ part, int n_part, int d,
                                       float* __restrict__ out) {
  int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= d) return;
  float s = 0.f;
  for (int p = 0; p < n_part; ++p) s += part[(long)p * d + c];
  out[c] = s;
}

// Block p sums rows [p * rpp, min(rows, (p+1) * rpp)) of every column.
template <typename T>
__global__ __launch_bounds__(256) void colsum_pass1(const T* __restrict__ X, long ldx, int rows,
                                                    int cols, int rpp, float* __restrict__ part) {
  const int p = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  const int r0 = p * rpp, r1 = min(rows, r0 + rpp);
  float s = 0.f;
  for (int r = r0; r < r1; ++r) s += (float)X[(long)r * ldx + c];
  part[(long)p * cols + c] = s;
}

template <int NC>
hipError_t ln_fwd_launch(const float* x, long ldx, long rs, const float* g, const float* b,
                         bf16* y, long ldy, float* mean, float* rstd, int rows, int d, float eps,
                         hipStream_t s) {
  hipLaunchKernelGGL(ln_fwd_kernel<NC>, dim3(sat_cdiv(rows, 4)), dim3(256), 0, s, x, ldx, rs, g,
                     b, y, ldy, mean, rstd, rows, d, eps);
  return hipGetLastError();
}

template <int NC>
hipError_t ln_bwd_launch(const float* dy, long lddy, const float* x, long ldx, long rs,
                         const float* g, const float* mean, const float* rstd, float* dres,
                         long ldres, float* pg, float* pb, int rows, int d, int n_part,
                         hipStream_t s) {
  hipLaunchKernelGGL(ln_bwd_kernel<NC>, dim3(sat_cdiv(n_part, 4)), dim3(256), 0, s, dy, lddy, x,
                     ldx, rs, g, mean, rstd, dres, ldres, pg, pb, rows, d, n_part);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_layernorm_fwd(const float* x, long ldx, long row_stride, const float* g,
                                const float* b, bf16* y, long ldy, float* mean, float* rstd,
                                int rows, int d, float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d % 4 != 0 || d > 64 * 4 * LN_MAXC || ldx % 4 != 0 || ldy % 4 != 0)
    return hipErrorInvalidValue;
  int nc = sat_cdiv(d, 256);
  if (nc <= 1) return ln_fwd_launch<1>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
  if (nc <= 2) return ln_fwd_launch<2>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
  if (nc <= 4) return ln_fwd_launch<4>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
  if (nc <= 8) return ln_fwd_launch<8>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
  if (nc <= 16) return ln_fwd_launch<16>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
  return ln_fwd_launch<32>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
}

hipError_t launch_layernorm_bwd(const float* dy, long lddy, const float* x, long ldx,
                                long row_stride, const float* g, const float* mean,
                                const float* rstd, float* dres, long ldres, float* part_g,
                                float* part_b, int rows, int d, int n_part, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d % 4 != 0 || d > 64 * 4 * 16 || lddy % 4 != 0 || ldx % 4 != 0 || ldres % 4 != 0 ||
      n_part <= 0)
    return hipErrorInvalidValue;
  int nc = sat_cdiv(d, 256);
#define LNB(NC) ln_bwd_launch<NC>(dy, lddy, x, ldx, row_stride, g, mean, rstd, dres, ldres, part_g, part_b, rows, d, n_part, s)
  if (nc <= 1) return LNB(1);
  if (nc <= 2) return LNB(2);
  if (nc <= 4) return LNB(4);
  if (nc <= 8) return LNB(8);
  return LNB(16);
#undef LNB
}

hipError_t launch_colsum_partials(const float* part, int n_part, int d, float* out,
                                  hipStream_t s) {
  if (d <= 0) return hipSuccess;
  hipLaunchKernelGGL(colsum_partials_kernel, dim3(sat_cdiv(d, 256)), dim3(256), 0, s, part,
                     n_part, d, out);
  return hipGetLastError();
}

template <typename T>
static hipError_t colsum_any(const T* X, long ldx, int rows, int cols, float* part, int n_part,
                             float* out, hipStream_t s) {
  if (cols <= 0) return hipSuccess;
  if (rows <= 0 || n_part <= 0) return hipErrorInvalidValue;
  int rpp = sat_cdiv(rows, n_part);
  int np = sat_cdiv(rows, rpp);
  hipLaunchKernelGGL(colsum_pass1<T>, dim3(sat_cdiv(cols, 256), np), dim3(256), 0, s, X, ldx,
                     rows, cols, rpp, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_colsum_partials(part, np, cols, out, s);
}

hipError_t launch_colsum_bf16(const bf16* X, long ldx, int rows, int cols, float* part,
                              int n_part, float* out, hipStream_t s) {
  return colsum_any<bf16>(X, ldx, rows, cols, part, n_part, out, s);
}
hipError_t launch_colsum_f32(const float* X, long ldx, int rows, int cols, float* part,
                             int n_part, float* out, hipStream_t s) {
  return colsum_any<float>(X, ldx, rows, cols, part, n_part, out, s);
}
