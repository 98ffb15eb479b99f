// Bandwidth-bound kernels of the bottleneck-ResNet step (the paper's second
// image workload, Table 3): im2col / col2im around the MFMA GEMMs that carry
// every convolution, training-mode batch norm (per-channel statistics over the
// N x H x W rows, forward and backward), ReLU masks, 3 x 3 / stride-2 max
// pooling, global average pooling and the stride-2 shortcut scatter.
//
// Activations are NHWC: a [N, H, W, C] tensor is the row-major matrix
// [N * H * W, C], the layout the convolution GEMMs read and write.  Every
// reduction is done in a fixed order (per-workgroup partials, then one pass
// over the partials), so results are run-to-run deterministic.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int NT = 256;

int grid_for(long n, int per_thread = 1) {
  long b = (n / per_thread + NT - 1) / NT;
  if (b < 1) b = 1;
  return (int)(b < 65536 ? b : 65536);
}

// ---------------------------------------------------------------- im2col

// col[p, (a k + b) C + c] = x[n, i s - pad + a, j s - pad + b, c] (zero
// outside the image), p = (n Ho + i) Wo + j.  Eight channels per thread
// (16-byte loads and stores); C % 8 == 0.
__global__ void im2col8_kernel(const bf16* __restrict__ x, bf16* __restrict__ col, int N, int H,
                               int W, int C, int k, int s, int pad, int Ho, int Wo, long ldc) {
  const int C8 = C / 8;
  const long per_p = (long)k * k * C8;
  const long total = (long)N * Ho * Wo * per_p;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const long p = t / per_p;
    const int r = (int)(t - p * per_p);
    const int ab = r / C8, c8 = r - ab * C8;
    const int a = ab / k, b = ab - a * k;
    const int j = (int)(p % Wo);
    const long q = p / Wo;
    const int i = (int)(q % Ho);
    const int n = (int)(q / Ho);
    const int hi = i * s - pad + a, wi = j * s - pad + b;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (hi >= 0 && hi < H && wi >= 0 && wi < W)
      v = *reinterpret_cast<const u32x4*>(x + (((long)n * H + hi) * W + wi) * C + 8 * c8);
    *reinterpret_cast<u32x4*>(col + p * ldc + (long)ab * C + 8 * c8) = v;
  }
}

// The im2col matrix transposed, colT[(a k + b) C + c, p] (row stride ldt >=
// P = N Ho Wo), which the weight-gradient product reads token-contiguous:
// im2col and the transpose in one pass.  A lane gathers eight consecutive
// output pixels' 16-byte pieces (8 channels of one tap, zeros outside the
// image), transposes the 8 x 8 block with byte permutes (element j of pixels
// 2e and 2e + 1 into one dword) and stores eight 16-byte rows of 8 pixels.
// A workgroup covers 128 pixels x 512 columns; TB column blocks per lane
// keep 8 TB loads in flight.  P % 8 == 0 and C % 8 == 0.
constexpr int I2T_TB = 4;
__global__ __launch_bounds__(NT) void im2col_t_kernel(const bf16* __restrict__ x, bf16* __restrict__ colT,
                                                      long ldt, int N, int H, int W, int C, int k,
                                                      int s, int pad, int Ho, int Wo) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long P = (long)N * Ho * Wo;
  const int cols = k * k * C;
  const long p0 = (long)blockIdx.y * 128 + (wave >> 1) * 64 + (lane >> 3) * 8;
  const int cb = blockIdx.x * 128 * I2T_TB + (wave & 1) * 64 * I2T_TB + (lane & 7) * 8;
  if (p0 >= P) return;
  // the eight pixels' image row / column origins and image offsets
  int hi0[8], wi0[8];
  long nb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const long p = p0 + i;
    const int j = (int)(p % Wo);
    const long q = p / Wo;
    const int ii = (int)(q % Ho);
    const int n = (int)(q / Ho);
    hi0[i] = ii * s - pad;
    wi0[i] = j * s - pad;
    nb[i] = (long)n * H;
  }
  u32x4 v[I2T_TB][8];
#pragma unroll
  for (int bk = 0; bk < I2T_TB; ++bk) {
    const int c0 = cb + 64 * bk;
    if (c0 < cols) {
      const int tap = c0 / C, c = c0 - tap * C;
      const int a = tap / k, b = tap - a * k;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int hi = hi0[i] + a, wi = wi0[i] + b;
        u32x4 z = {0u, 0u, 0u, 0u};
        if (hi >= 0 && hi < H && wi >= 0 && wi < W)
          z = *reinterpret_cast<const u32x4*>(x + ((nb[i] + hi) * W + wi) * C + c);
        v[bk][i] = z;
      }
    }
  }
#pragma unroll
  for (int bk = 0; bk < I2T_TB; ++bk) {
    const int c0 = cb + 64 * bk;
    if (c0 >= cols) break;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = __builtin_amdgcn_perm(v[bk][2 * e + 1][j >> 1], v[bk][2 * e][j >> 1], sel);
      *reinterpret_cast<u32x4*>(colT + (long)(c0 + j) * ldt + p0) = o;
    }
  }
}

// The stem: fp32 NCHW images -> bf16 columns, K = k k C (taps ordered a, b,
// c as above), zero columns K .. ldc - 1.
__global__ void im2col_nchw_kernel(const float* __restrict__ img, bf16* __restrict__ col, int N,
                                   int C, int H, int W, int k, int s, int pad, int Ho, int Wo,
                                   long ldc) {
  const long total = (long)N * Ho * Wo * ldc;
  const int K = k * k * C;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const long p = t / ldc;
    const int kc = (int)(t - p * ldc);
    float v = 0.f;
    if (kc < K) {
      const int ab = kc / C, c = kc - ab * C;
      const int a = ab / k, b = ab - a * k;
      const int j = (int)(p % Wo);
      const long q = p / Wo;
      const int i = (int)(q % Ho);
      const int n = (int)(q / Ho);
      const int hi = i * s - pad + a, wi = j * s - pad + b;
      if (hi >= 0 && hi < H && wi >= 0 && wi < W) v = img[(((long)n * C + c) * H + hi) * W + wi];
    }
    col[t] = f2bf(v);
  }
}

// dx[n, h, w, c] (+)= sum over taps (a, b) with (h + pad - a) / s = i and
// (w + pad - b) / s = j whole and in range of dcol[(n Ho + i) Wo + j,
// (a k + b) C + c], taps in increasing (a, b) order.  Four channels per
// thread; C % 4 == 0.
__global__ void col2im4_kernel(const float* __restrict__ dcol, long ldc, float* __restrict__ dx,
                               int N, int H, int W, int C, int k, int s, int pad, int Ho, int Wo,
                               int accumulate) {
  const int C4 = C / 4;
  const long total = (long)N * H * W * C4;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const int c4 = (int)(t % C4);
    const long q = t / C4;
    const int w = (int)(q % W);
    const long q2 = q / W;
    const int h = (int)(q2 % H);
    const int n = (int)(q2 / H);
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int a = 0; a < k; ++a) {
      const int hh = h + pad - a;
      if (hh < 0 || hh % s) continue;
      const int i = hh / s;
      if (i >= Ho) continue;
      for (int b = 0; b < k; ++b) {
        const int ww = w + pad - b;
        if (ww < 0 || ww % s) continue;
        const int j = ww / s;
        if (j >= Wo) continue;
        acc += *reinterpret_cast<const floatx4*>(dcol + (((long)n * Ho + i) * Wo + j) * ldc +
                                                 (long)(a * k + b) * C + 4 * c4);
      }
    }
    floatx4* o = reinterpret_cast<floatx4*>(dx + q * C + 4 * c4);
    if (accumulate) *o += acc;
    else *o = acc;
  }
}

// ---------------------------------------------------------------- batch norm

// Column slab of a [P, C] reduction in groups of four columns (C % 4 == 0):
// a slab is up to 4 NT columns; thread t owns columns c .. c + 3 with
// c = c0 + 4 (t % cs4) and rows of phase t / cs4, cs4 = the slab's column
// groups (at most NT), all NT / cs4 phases busy when cs4 divides NT, else one.
struct Slab4 {
  int c, phase, phases, cs4;
  __device__ Slab4(int C) {
    const int c0 = blockIdx.y * 4 * NT;
    cs4 = min((C - c0) / 4, NT);
    phases = (NT % cs4 == 0) ? NT / cs4 : 1;
    const int t = threadIdx.x;
    phase = t / cs4;
    c = (phase < phases) ? c0 + 4 * (t % cs4) : -1;
  }
};

// Sum of v over the phases of each column group, in phase order; the result
// is valid in the threads of phase 0.
__device__ floatx4 phase_sum4(floatx4 v, const Slab4& sl, floatx4* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  floatx4 s = {0.f, 0.f, 0.f, 0.f};
  if (sl.phase == 0 && sl.c >= 0)
    for (int ph = 0; ph < sl.phases; ++ph) s += red[ph * sl.cs4 + threadIdx.x];
  __syncthreads();
  return s;
}

constexpr int BN_U = 8;  // rows whose loads a thread has in flight together

// Per-channel partial sums of (x - K_c) and (x - K_c)^2 over the rows of
// workgroup x's block, with the shift K_c = x[0, c] (the shifted-data form of
// the variance: no cancellation when the mean is large next to the spread).
// Each thread adds its rows in increasing order.
__global__ void bn_stats_partial_kernel(const float* __restrict__ x, long P, int C, long rpb,
                                        float* __restrict__ part) {
  __shared__ floatx4 red[NT];
  const Slab4 sl(C);
  floatx4 s1 = {0.f, 0.f, 0.f, 0.f}, s2 = s1;
  if (sl.c >= 0) {
    const floatx4 K = *reinterpret_cast<const floatx4*>(x + sl.c);
    const long r0 = (long)blockIdx.x * rpb;
    const long r1 = min(P, r0 + rpb);
    for (long rb = r0 + sl.phase; rb < r1; rb += (long)BN_U * sl.phases) {
      floatx4 v[BN_U];
#pragma unroll
      for (int i = 0; i < BN_U; ++i) {
        const long r = rb + (long)i * sl.phases;
        if (r < r1) v[i] = *reinterpret_cast<const floatx4*>(x + r * C + sl.c);
      }
#pragma unroll
      for (int i = 0; i < BN_U; ++i)
        if (rb + (long)i * sl.phases < r1) {
          const floatx4 d = v[i] - K;
          s1 += d;
          s2 += d * d;
        }
    }
  }
  s1 = phase_sum4(s1, sl, red);
  s2 = phase_sum4(s2, sl, red);
  if (sl.phase == 0 && sl.c >= 0) {
    *reinterpret_cast<floatx4*>(part + (long)blockIdx.x * C + sl.c) = s1;
    *reinterpret_cast<floatx4*>(part + ((long)gridDim.x + blockIdx.x) * C + sl.c) = s2;
  }
}

// The final reductions over the nb partial rows: a workgroup of FL_T
// threads owns FL_C consecutive columns; lane group l (of FL_L) sums rows
// l, l + FL_L, ..., then the lane groups are added in order.
constexpr int FL_C = 64, FL_L = 16, FL_T = FL_C * FL_L;

template <typename T>
__device__ void final_sums(const float* __restrict__ part, int nb, int C, T& s1, T& s2) {
  __shared__ T r1[FL_T], r2[FL_T];
  const int t = threadIdx.x, cl = t % FL_C, l = t / FL_C;
  const int c = blockIdx.x * FL_C + cl;
  T a = 0, b2 = 0;
  if (c < C) {
#pragma unroll 4
    for (int b = l; b < nb; b += FL_L) {
      a += (T)part[(long)b * C + c];
      b2 += (T)part[((long)nb + b) * C + c];
    }
  }
  r1[t] = a;
  r2[t] = b2;
  __syncthreads();
  s1 = 0;
  s2 = 0;
  if (l == 0)
    for (int k = 0; k < FL_L; ++k) {
      s1 += r1[k * FL_C + cl];
      s2 += r2[k * FL_C + cl];
    }
}

__global__ __launch_bounds__(FL_T) void bn_stats_final_kernel(const float* __restrict__ x,
                                                              const float* __restrict__ part, int nb,
                                                              long P, int C, float eps,
                                                              float* __restrict__ mean,
                                                              float* __restrict__ rstd) {
  double s1, s2;
  final_sums<double>(part, nb, C, s1, s2);
  const int c = blockIdx.x * FL_C + threadIdx.x % FL_C;
  if (threadIdx.x >= FL_C || c >= C) return;
  const double m1 = s1 / (double)P;
  double var = s2 / (double)P - m1 * m1;
  if (var < 0.0) var = 0.0;
  mean[c] = (float)(x[c] + m1);
  rstd[c] = (float)(1.0 / sqrt(var + (double)eps));
}

// Four consecutive per-channel values p[c .. c + 3] (c % 4 == 0): one
// 16-byte load when the arrays are 16-byte aligned (V), else four.  The
// elementwise kernels read up to ten such parameters per four elements, so
// their instruction count, not their bytes, set their time with scalar loads.
template <bool V>
__device__ __forceinline__ floatx4 ld4(const float* __restrict__ p, int c) {
  if constexpr (V) return *reinterpret_cast<const floatx4*>(p + c);
  floatx4 r = {p[c], p[c + 1], p[c + 2], p[c + 3]};
  return r;
}

__host__ __device__ inline bool a16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15) == 0;
}

// y = (x - mean) rstd g + b, ReLU when relu, as bf16 (when y) and fp32 (when yf).
template <bool V>
__global__ void bn_apply_kernel(const float* __restrict__ x, long n4, int C,
                                const float* __restrict__ mean, const float* __restrict__ rstd,
                                const float* __restrict__ g, const float* __restrict__ b, int relu,
                                bf16* __restrict__ y, float* __restrict__ yf) {
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < n4; t += (long)gridDim.x * NT) {
    const int c = (int)((4 * t) % C);
    const floatx4 v = reinterpret_cast<const floatx4*>(x)[t];
    const floatx4 m4 = ld4<V>(mean, c), r4 = ld4<V>(rstd, c), g4 = ld4<V>(g, c), b4 = ld4<V>(b, c);
    floatx4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float z = (v[e] - m4[e]) * r4[e] * g4[e] + b4[e];
      o[e] = relu ? fmaxf(z, 0.f) : z;
    }
    if (y) {
      bf16x4 ob = {f2bf(o[0]), f2bf(o[1]), f2bf(o[2]), f2bf(o[3])};
      reinterpret_cast<bf16x4*>(y)[t] = ob;
    }
    if (yf) reinterpret_cast<floatx4*>(yf)[t] = o;
  }
}

// out = ReLU(BN_a(xa) + (xs2 ? BN_s(xs) : xs)), fp32 and bf16.
template <bool V>
__global__ void bn_add_relu_kernel(const float* __restrict__ xa, const float* __restrict__ ma,
                                   const float* __restrict__ ra, const float* __restrict__ ga,
                                   const float* __restrict__ ba, const float* __restrict__ xs,
                                   const float* __restrict__ ms, const float* __restrict__ rs,
                                   const float* __restrict__ gs, const float* __restrict__ bs,
                                   long n4, int C, float* __restrict__ out,
                                   bf16* __restrict__ outb) {
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < n4; t += (long)gridDim.x * NT) {
    const int c = (int)((4 * t) % C);
    const floatx4 a = reinterpret_cast<const floatx4*>(xa)[t];
    const floatx4 sv = reinterpret_cast<const floatx4*>(xs)[t];
    const floatx4 ma4 = ld4<V>(ma, c), ra4 = ld4<V>(ra, c), ga4 = ld4<V>(ga, c), ba4 = ld4<V>(ba, c);
    floatx4 o;
    if (ms) {
      const floatx4 ms4 = ld4<V>(ms, c), rs4 = ld4<V>(rs, c), gs4 = ld4<V>(gs, c), bs4 = ld4<V>(bs, c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float za = (a[e] - ma4[e]) * ra4[e] * ga4[e] + ba4[e];
        const float zs = (sv[e] - ms4[e]) * rs4[e] * gs4[e] + bs4[e];
        o[e] = fmaxf(za + zs, 0.f);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float za = (a[e] - ma4[e]) * ra4[e] * ga4[e] + ba4[e];
        o[e] = fmaxf(za + sv[e], 0.f);
      }
    }
    reinterpret_cast<floatx4*>(out)[t] = o;
    bf16x4 ob = {f2bf(o[0]), f2bf(o[1]), f2bf(o[2]), f2bf(o[3])};
    reinterpret_cast<bf16x4*>(outb)[t] = ob;
  }
}

// Gradient through a ReLU: g = dy where the mask source is positive.
// MASK 0: none; 1: bf16 activation a > 0; 2: fp32 activation > 0.
template <int MASK>
__device__ __forceinline__ float masked(float dy, const void* m, long i) {
  if (MASK == 1) return bf2f(reinterpret_cast<const bf16*>(m)[i]) > 0.f ? dy : 0.f;
  if (MASK == 2) return reinterpret_cast<const float*>(m)[i] > 0.f ? dy : 0.f;
  return dy;
}

// The same for four consecutive elements 4 t .. 4 t + 3 (one vector load of
// the mask when V, i.e. when the mask is aligned for it).
template <int MASK, bool V>
__device__ __forceinline__ floatx4 masked4(floatx4 dy, const void* m, long t) {
  if constexpr (!V) {
#pragma unroll
    for (int e = 0; e < 4; ++e) dy[e] = masked<MASK>(dy[e], m, 4 * t + e);
  } else if constexpr (MASK == 1) {
    const bf16x4 a = reinterpret_cast<const bf16x4*>(m)[t];
#pragma unroll
    for (int e = 0; e < 4; ++e) dy[e] = bf2f(a[e]) > 0.f ? dy[e] : 0.f;
  } else if constexpr (MASK == 2) {
    const floatx4 a = reinterpret_cast<const floatx4*>(m)[t];
#pragma unroll
    for (int e = 0; e < 4; ++e) dy[e] = a[e] > 0.f ? dy[e] : 0.f;
  }
  return dy;
}

// Per-channel partial sums of g and g * xhat, xhat = (x - mean) rstd, each
// thread over its rows in increasing order.
template <int MASK>
__global__ void bn_bwd_partial_kernel(const float* __restrict__ dy, const void* __restrict__ msk,
                                      const float* __restrict__ x, const float* __restrict__ mean,
                                      const float* __restrict__ rstd, long P, int C, long rpb,
                                      float* __restrict__ part) {
  __shared__ floatx4 red[NT];
  const Slab4 sl(C);
  floatx4 s1 = {0.f, 0.f, 0.f, 0.f}, s2 = s1;
  if (sl.c >= 0) {
    const floatx4 mu = *reinterpret_cast<const floatx4*>(mean + sl.c);
    const floatx4 rs = *reinterpret_cast<const floatx4*>(rstd + sl.c);
    const long r0 = (long)blockIdx.x * rpb;
    const long r1 = min(P, r0 + rpb);
    for (long rb = r0 + sl.phase; rb < r1; rb += (long)BN_U * sl.phases) {
      floatx4 gv[BN_U], xv[BN_U];
#pragma unroll
      for (int i = 0; i < BN_U; ++i) {
        const long r = rb + (long)i * sl.phases;
        if (r < r1) {
          const long i4 = (r * C + sl.c) / 4;
          gv[i] = masked4<MASK, true>(reinterpret_cast<const floatx4*>(dy)[i4], msk, i4);
          xv[i] = reinterpret_cast<const floatx4*>(x)[i4];
        }
      }
#pragma unroll
      for (int i = 0; i < BN_U; ++i)
        if (rb + (long)i * sl.phases < r1) {
          s1 += gv[i];
          s2 += gv[i] * ((xv[i] - mu) * rs);
        }
    }
  }
  s1 = phase_sum4(s1, sl, red);
  s2 = phase_sum4(s2, sl, red);
  if (sl.phase == 0 && sl.c >= 0) {
    *reinterpret_cast<floatx4*>(part + (long)blockIdx.x * C + sl.c) = s1;
    *reinterpret_cast<floatx4*>(part + ((long)gridDim.x + blockIdx.x) * C + sl.c) = s2;
  }
}

// dbeta = sum g, dgamma = sum g xhat (written to the gradient arena).
__global__ __launch_bounds__(FL_T) void bn_bwd_final_kernel(const float* __restrict__ part, int nb,
                                                            int C, float* __restrict__ dg,
                                                            float* __restrict__ db) {
  float s1, s2;
  final_sums<float>(part, nb, C, s1, s2);
  const int c = blockIdx.x * FL_C + threadIdx.x % FL_C;
  if (threadIdx.x >= FL_C || c >= C) return;
  db[c] = s1;
  dg[c] = s2;
}

// dx = rstd g_c (g - dbeta / P - xhat dgamma / P), as bf16.
template <int MASK, bool V>
__global__ void bn_bwd_apply_kernel(const float* __restrict__ dy, const void* __restrict__ msk,
                                    const float* __restrict__ x, const float* __restrict__ mean,
                                    const float* __restrict__ rstd, const float* __restrict__ gam,
                                    const float* __restrict__ dg, const float* __restrict__ db,
                                    long n4, int C, float inv_p, bf16* __restrict__ dx) {
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < n4; t += (long)gridDim.x * NT) {
    const int c = (int)((4 * t) % C);
    const floatx4 d = masked4<MASK, V>(reinterpret_cast<const floatx4*>(dy)[t], msk, t);
    const floatx4 v = reinterpret_cast<const floatx4*>(x)[t];
    const floatx4 m4 = ld4<V>(mean, c), r4 = ld4<V>(rstd, c), g4 = ld4<V>(gam, c);
    const floatx4 dg4 = ld4<V>(dg, c), db4 = ld4<V>(db, c);
    bf16x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float xh = (v[e] - m4[e]) * r4[e];
      o[e] = f2bf(r4[e] * g4[e] * (d[e] - db4[e] * inv_p - xh * dg4[e] * inv_p));
    }
    reinterpret_cast<bf16x4*>(dx)[t] = o;
  }
}

// do = dy where out > 0 (the ReLU after a block's shortcut add).
__global__ void relu_mask_kernel(const float* __restrict__ dy, const float* __restrict__ out,
                                 long n4, float* __restrict__ dz) {
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < n4; t += (long)gridDim.x * NT) {
    const floatx4 d = reinterpret_cast<const floatx4*>(dy)[t];
    const floatx4 o = reinterpret_cast<const floatx4*>(out)[t];
    floatx4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = o[e] > 0.f ? d[e] : 0.f;
    reinterpret_cast<floatx4*>(dz)[t] = r;
  }
}

// ---------------------------------------------------------------- pooling

// 3 x 3 max pool, stride 2, padding 1 (padding never wins; ties go to the
// first tap in row-major order): fp32 and bf16 outputs and the winning tap.
__global__ void maxpool_fwd_kernel(const float* __restrict__ x, int N, int H, int W, int C, int Ho,
                                   int Wo, float* __restrict__ y, bf16* __restrict__ yb,
                                   uint8_t* __restrict__ arg) {
  const long total = (long)N * Ho * Wo * C;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const int c = (int)(t % C);
    const long q = t / C;
    const int j = (int)(q % Wo);
    const long q2 = q / Wo;
    const int i = (int)(q2 % Ho);
    const int n = (int)(q2 / Ho);
    float best = -INFINITY;
    int bi = 0;
    for (int a = 0; a < 3; ++a) {
      const int h = 2 * i - 1 + a;
      if (h < 0 || h >= H) continue;
      for (int b = 0; b < 3; ++b) {
        const int w = 2 * j - 1 + b;
        if (w < 0 || w >= W) continue;
        const float v = x[(((long)n * H + h) * W + w) * C + c];
        if (v > best) {
          best = v;
          bi = 3 * a + b;
        }
      }
    }
    y[t] = best;
    yb[t] = f2bf(best);
    arg[t] = (uint8_t)bi;
  }
}

// dx[n, h, w, c] = sum of dy over the windows whose winning tap is (h, w),
// windows in increasing (i, j) order.
__global__ void maxpool_bwd_kernel(const float* __restrict__ dy, const uint8_t* __restrict__ arg,
                                   int N, int H, int W, int C, int Ho, int Wo,
                                   float* __restrict__ dx) {
  const long total = (long)N * H * W * C;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const int c = (int)(t % C);
    const long q = t / C;
    const int w = (int)(q % W);
    const long q2 = q / W;
    const int h = (int)(q2 % H);
    const int n = (int)(q2 / H);
    float acc = 0.f;
    const int i0 = h / 2, j0 = w / 2;  // windows i with 2i - 1 <= h <= 2i + 1
    for (int i = i0; i <= min(Ho - 1, (h + 1) / 2); ++i) {
      if (2 * i - 1 > h) continue;
      for (int j = j0; j <= min(Wo - 1, (w + 1) / 2); ++j) {
        if (2 * j - 1 > w) continue;
        const long o = (((long)n * Ho + i) * Wo + j) * C + c;
        if (arg[o] == 3 * (h - 2 * i + 1) + (w - 2 * j + 1)) acc += dy[o];
      }
    }
    dx[t] = acc;
  }
}

// feat[n, c] = mean over the HW rows of image n (bf16), in row order.
__global__ void avgpool_fwd_kernel(const float* __restrict__ x, int N, int HW, int C,
                                   bf16* __restrict__ feat) {
  const long total = (long)N * C;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const int c = (int)(t % C);
    const long n = t / C;
    float s = 0.f;
    for (int r = 0; r < HW; ++r) s += x[(n * HW + r) * C + c];
    feat[t] = f2bf(s / (float)HW);
  }
}

__global__ void avgpool_bwd_kernel(const float* __restrict__ dfeat, int N, int HW, int C,
                                   float* __restrict__ dx) {
  const long total = (long)N * HW * C;
  const float inv = 1.f / (float)HW;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const int c = (int)(t % C);
    const long n = t / ((long)HW * C);
    dx[t] = dfeat[n * C + c] * inv;
  }
}

// dx[n, 2i, 2j, c] += dsub[n, i, j, c]: the input gradient of a stride-2
// 1 x 1 convolution (every other row and column of the input), four
// channels per thread.
__global__ void stride2_add_kernel(const float* __restrict__ dsub, int N, int Ho, int Wo, int C,
                                   int H, int W, float* __restrict__ dx) {
  const int C4 = C / 4;
  const long total = (long)N * Ho * Wo * C4;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const int c4 = (int)(t % C4);
    const long q = t / C4;
    const int j = (int)(q % Wo);
    const long q2 = q / Wo;
    const int i = (int)(q2 % Ho);
    const int n = (int)(q2 / Ho);
    floatx4* o = reinterpret_cast<floatx4*>(dx + (((long)n * H + 2 * i) * W + 2 * j) * C + 4 * c4);
    *o += *reinterpret_cast<const floatx4*>(dsub + q * C + 4 * c4);
  }
}

__global__ void pad_cols_kernel(const bf16* __restrict__ src, int rows, int cols,
                                bf16* __restrict__ dst, long ldd) {
  const long total = (long)rows * ldd;
  for (long t = (long)blockIdx.x * NT + threadIdx.x; t < total; t += (long)gridDim.x * NT) {
    const long r = t / ldd;
    const int c = (int)(t - r * ldd);
    dst[t] = c < cols ? src[r * cols + c] : f2bf(0.f);
  }
}

}  // namespace

hipError_t launch_pad_cols_bf16(const bf16* src, int rows, int cols, bf16* dst, long ldd,
                                hipStream_t st) {
  if (ldd < cols) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pad_cols_kernel, dim3(grid_for((long)rows * ldd)), dim3(NT), 0, st, src, rows,
                     cols, dst, ldd);
  return hipGetLastError();
}

// Row blocks of the batch-norm reductions: about 1024 workgroups in all,
// at least 32 rows each.
int bn_parts(long P, int C) {
  const int slabs = (C + 4 * NT - 1) / (4 * NT);
  long nb = 1024 / slabs;
  nb = nb < 1 ? 1 : nb;
  const long by_rows = (P + 31) / 32;
  return (int)(nb < by_rows ? nb : (by_rows < 1 ? 1 : by_rows));
}

hipError_t launch_im2col(const bf16* x, bf16* col, long ldc, int N, int H, int W, int C, int k,
                         int s, int pad, int Ho, int Wo, hipStream_t st) {
  if (C % 8 || ldc != (long)k * k * C) return hipErrorInvalidValue;
  const long total = (long)N * Ho * Wo * k * k * (C / 8);
  hipLaunchKernelGGL(im2col8_kernel, dim3(grid_for(total)), dim3(NT), 0, st, x, col, N, H, W, C, k,
                     s, pad, Ho, Wo, ldc);
  return hipGetLastError();
}

hipError_t launch_im2col_t(const bf16* x, bf16* colT, long ldt, int N, int H, int W, int C, int k,
                           int s, int pad, int Ho, int Wo, hipStream_t st) {
  const long P = (long)N * Ho * Wo;
  if (C % 8 || P % 8 || ldt < P || ldt % 8 ||
      ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(colT)) & 15))
    return hipErrorInvalidValue;
  const int cols = k * k * C;
  dim3 grid((unsigned)((cols + 128 * I2T_TB - 1) / (128 * I2T_TB)), (unsigned)((P + 127) / 128));
  hipLaunchKernelGGL(im2col_t_kernel, grid, dim3(NT), 0, st, x, colT, ldt, N, H, W, C, k, s, pad, Ho,
                     Wo);
  return hipGetLastError();
}

hipError_t launch_im2col_nchw(const float* img, bf16* col, long ldc, int N, int C, int H, int W,
                              int k, int s, int pad, int Ho, int Wo, hipStream_t st) {
  if (ldc < (long)k * k * C) return hipErrorInvalidValue;
  const long total = (long)N * Ho * Wo * ldc;
  hipLaunchKernelGGL(im2col_nchw_kernel, dim3(grid_for(total)), dim3(NT), 0, st, img, col, N, C, H,
                     W, k, s, pad, Ho, Wo, ldc);
  return hipGetLastError();
}

hipError_t launch_col2im(const float* dcol, long ldc, float* dx, int N, int H, int W, int C, int k,
                         int s, int pad, int Ho, int Wo, int accumulate, hipStream_t st) {
  if (C % 4 || ldc % 4) return hipErrorInvalidValue;
  const long total = (long)N * H * W * (C / 4);
  hipLaunchKernelGGL(col2im4_kernel, dim3(grid_for(total)), dim3(NT), 0, st, dcol, ldc, dx, N, H,
                     W, C, k, s, pad, Ho, Wo, accumulate);
  return hipGetLastError();
}

hipError_t launch_bn_stats(const float* x, long P, int C, float eps, float* part, float* mean,
                           float* rstd, hipStream_t st) {
  if (P <= 0 || C <= 0) return hipErrorInvalidValue;
  const int nb = bn_parts(P, C);
  const long rpb = (P + nb - 1) / nb;
  hipLaunchKernelGGL(bn_stats_partial_kernel, dim3(nb, (C + 4 * NT - 1) / (4 * NT)), dim3(NT), 0, st, x, P,
                     C, rpb, part);
  hipLaunchKernelGGL(bn_stats_final_kernel, dim3((C + FL_C - 1) / FL_C), dim3(FL_T), 0, st, x, part,
                     nb, P, C, eps, mean, rstd);
  return hipGetLastError();
}

hipError_t launch_bn_apply(const float* x, long P, int C, const float* mean, const float* rstd,
                           const float* g, const float* b, int relu, bf16* y, float* yf,
                           hipStream_t st) {
  if (C % 4) return hipErrorInvalidValue;
  const long n4 = P * C / 4;
  if (a16(mean) && a16(rstd) && a16(g) && a16(b))
    hipLaunchKernelGGL(bn_apply_kernel<true>, dim3(grid_for(n4)), dim3(NT), 0, st, x, n4, C, mean, rstd,
                       g, b, relu, y, yf);
  else
    hipLaunchKernelGGL(bn_apply_kernel<false>, dim3(grid_for(n4)), dim3(NT), 0, st, x, n4, C, mean, rstd,
                       g, b, relu, y, yf);
  return hipGetLastError();
}

hipError_t launch_bn_add_relu(const float* xa, const float* ma, const float* ra, const float* ga,
                              const float* ba, const float* xs, const float* ms, const float* rs,
                              const float* gs, const float* bs, long P, int C, float* out,
                              bf16* outb, hipStream_t st) {
  if (C % 4) return hipErrorInvalidValue;
  const long n4 = P * C / 4;
  const bool v = a16(ma) && a16(ra) && a16(ga) && a16(ba) &&
                 (ms == nullptr || (a16(ms) && a16(rs) && a16(gs) && a16(bs)));
  if (v)
    hipLaunchKernelGGL(bn_add_relu_kernel<true>, dim3(grid_for(n4)), dim3(NT), 0, st, xa, ma, ra, ga,
                       ba, xs, ms, rs, gs, bs, n4, C, out, outb);
  else
    hipLaunchKernelGGL(bn_add_relu_kernel<false>, dim3(grid_for(n4)), dim3(NT), 0, st, xa, ma, ra, ga,
                       ba, xs, ms, rs, gs, bs, n4, C, out, outb);
  return hipGetLastError();
}

hipError_t launch_bn_bwd(const float* dy, int mask_kind, const void* mask, const float* x,
                         const float* mean, const float* rstd, const float* gam, long P, int C,
                         float* part, float* dg, float* db, bf16* dx, hipStream_t st) {
  if (C % 4 || P <= 0 || mask_kind < 0 || mask_kind > 2) return hipErrorInvalidValue;
  const int nb = bn_parts(P, C);
  const long rpb = (P + nb - 1) / nb;
  const dim3 g2(nb, (C + 4 * NT - 1) / (4 * NT));
  if (mask_kind == 0)
    hipLaunchKernelGGL(bn_bwd_partial_kernel<0>, g2, dim3(NT), 0, st, dy, mask, x, mean, rstd, P, C,
                       rpb, part);
  else if (mask_kind == 1)
    hipLaunchKernelGGL(bn_bwd_partial_kernel<1>, g2, dim3(NT), 0, st, dy, mask, x, mean, rstd, P, C,
                       rpb, part);
  else
    hipLaunchKernelGGL(bn_bwd_partial_kernel<2>, g2, dim3(NT), 0, st, dy, mask, x, mean, rstd, P, C,
                       rpb, part);
  hipLaunchKernelGGL(bn_bwd_final_kernel, dim3((C + FL_C - 1) / FL_C), dim3(FL_T), 0, st, part, nb, C,
                     dg, db);
  const long n4 = P * C / 4;
  const float inv_p = (float)(1.0 / (double)P);
  const dim3 g1(grid_for(n4));
  const bool v = a16(mean) && a16(rstd) && a16(gam) && a16(dg) && a16(db) &&
                 (mask_kind != 1 || (reinterpret_cast<uintptr_t>(mask) & 7) == 0) &&
                 (mask_kind != 2 || a16(mask));
#define BNB(M, VV)                                                                              \
  hipLaunchKernelGGL((bn_bwd_apply_kernel<M, VV>), g1, dim3(NT), 0, st, dy, mask, x, mean, rstd, \
                     gam, dg, db, n4, C, inv_p, dx)
  if (mask_kind == 0) {
    if (v) BNB(0, true); else BNB(0, false);
  } else if (mask_kind == 1) {
    if (v) BNB(1, true); else BNB(1, false);
  } else {
    if (v) BNB(2, true); else BNB(2, false);
  }
#undef BNB
  return hipGetLastError();
}

hipError_t launch_relu_mask(const float* dy, const float* out, long n, float* dz, hipStream_t st) {
  if (n % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(relu_mask_kernel, dim3(grid_for(n / 4)), dim3(NT), 0, st, dy, out, n / 4, dz);
  return hipGetLastError();
}

hipError_t launch_maxpool_fwd(const float* x, int N, int H, int W, int C, int Ho, int Wo, float* y,
                              bf16* yb, uint8_t* arg, hipStream_t st) {
  const long total = (long)N * Ho * Wo * C;
  hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(grid_for(total)), dim3(NT), 0, st, x, N, H, W, C, Ho,
                     Wo, y, yb, arg);
  return hipGetLastError();
}

hipError_t launch_maxpool_bwd(const float* dy, const uint8_t* arg, int N, int H, int W, int C,
                              int Ho, int Wo, float* dx, hipStream_t st) {
  const long total = (long)N * H * W * C;
  hipLaunchKernelGGL(maxpool_bwd_kernel, dim3(grid_for(total)), dim3(NT), 0, st, dy, arg, N, H, W,
                     C, Ho, Wo, dx);
  return hipGetLastError();
}

hipError_t launch_avgpool_fwd(const float* x, int N, int HW, int C, bf16* feat, hipStream_t st) {
  hipLaunchKernelGGL(avgpool_fwd_kernel, dim3(grid_for((long)N * C)), dim3(NT), 0, st, x, N, HW, C,
                     feat);
  return hipGetLastError();
}

hipError_t launch_avgpool_bwd(const float* dfeat, int N, int HW, int C, float* dx, hipStream_t st) {
  hipLaunchKernelGGL(avgpool_bwd_kernel, dim3(grid_for((long)N * HW * C)), dim3(NT), 0, st, dfeat,
                     N, HW, C, dx);
  return hipGetLastError();
}

hipError_t launch_stride2_add(const float* dsub, int N, int Ho, int Wo, int C, int H, int W,
                              float* dx, hipStream_t st) {
  if (C % 4) return hipErrorInvalidValue;
  const long total = (long)N * Ho * Wo * (C / 4);
  hipLaunchKernelGGL(stride2_add_kernel, dim3(grid_for(total)), dim3(NT), 0, st, dsub, N, Ho, Wo, C,
                     H, W, dx);
  return hipGetLastError();
}
