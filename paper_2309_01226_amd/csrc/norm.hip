// LayerNorm forward / backward and deterministic column reductions.
//
// One wavefront owns one row (rows up to 8192 wide stay in registers as
// float4 chunks, 256 columns per chunk); mean and variance are two-pass
// wave reductions over the register copy, so x is read from HBM once.
// Gain / shift gradients are reduced without atomics: each workgroup of the
// backward accumulates the columns of a fixed block of rows into a partial
// row, and a second kernel sums the partial rows in a fixed order (bitwise
// reproducible).
#include "common.h"
#include "kernels.h"

namespace {

constexpr int LN_MAXC = 32;  // float4 chunks per lane: d <= 64 * 4 * 32 = 8192
#ifndef LN_FWD_GRID
#define LN_FWD_GRID 1024
#endif

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

// s_waitcnt lgkmcnt(0) only: vector loads may stay in flight across it.
// Raw buffer resource over `bytes` bytes at p: accesses past the end read 0
// and write nothing.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}
__device__ __forceinline__ float4 bload4(__amdgpu_buffer_rsrc_t r, int vo, int so) {
  const floatx4 v = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(r, vo, so, 0));
  return make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void bstore4(float4 v, __amdgpu_buffer_rsrc_t r, int vo, int so) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, floatx4{v.x, v.y, v.z, v.w}), r, vo,
                                         so, 0);
}
// N stores into an empty buffer range (dropped by the range check, counted by
// the vector-memory counter).  Issued between the first row's loads and the
// loop, they give the loop's entry the same count of operations after those
// loads as its back edge has (the previous row's stores), so the compiler's
// wait at the loop head does not also wait for the previous row's stores.
template <int N>
__device__ __forceinline__ void vm_pad(const void* any) {
  const auto r = rsrc(any, 0);
  // volatile (bit 31 of the auxiliary argument): kept one by one, never merged
#pragma unroll
  for (int i = 0; i < N; ++i) __builtin_amdgcn_raw_buffer_store_b32(0u, r, 4 * i, 0, (int)0x80000000u);
}

// Wide rows (d >= 1024): workgroup w walks the rows w, w + gridDim.x, ...,
// each thread holding NCH float4 chunks of a row (columns (c * 256 + tid) * 4
// .. +3).  The loop is software pipelined like the backward's: the next row
// is loaded into the other of two register sets before the current one is
// reduced and written (unrolled by two, so no set is copied), and every row
// access is a buffer instruction, so columns past d need no branch (reads give
// 0, writes are dropped) and the compiler's wait counts stay exact.  Mean and
// variance are two passes over the register copy (x is read from HBM once);
// the row sums are combined across the four waves through LDS in a fixed
// order, with barriers that do not wait for the next row's loads.  The gain
// and shift chunks are loaded once per workgroup.
template <int NCH>
__global__ __launch_bounds__(256) void ln_fwd_wg_kernel(const float* __restrict__ x, long ldx,
                                                        long row_stride,
                                                        const float* __restrict__ g,
                                                        const float* __restrict__ b,
                                                        bf16* __restrict__ y, long ldy,
                                                        float* __restrict__ mean,
                                                        float* __restrict__ rstd, int rows, int d,
                                                        float eps) {
  __shared__ float red[2][2][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int vo = 16 * tid;  // byte offset of the thread's columns; chunk c adds 4096 c
  float4 gg[NCH], bb[NCH];
  bool in[NCH];
  {
    const auto rg = rsrc(g, 4 * d), rb = rsrc(b, 4 * d);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      gg[c] = bload4(rg, vo, 4096 * c);
      bb[c] = bload4(rb, vo, 4096 * c);
      in[c] = (c * 256 + tid) * 4 < d;
    }
  }
  auto load = [&](int row, bool ok, float4* v) {
    const auto rx = rsrc(x + (long)(ok ? row : 0) * row_stride * ldx, ok ? 4 * d : 0);
#pragma unroll
    for (int c = 0; c < NCH; ++c) v[c] = bload4(rx, vo, 4096 * c);
  };
  auto process = [&](int row, int par, const float4* v) {
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) s += v[c].x + v[c].y + v[c].z + v[c].w;  // 0 past d
    s = wave_sum(s);
    if (lane == 0) red[par][0][wave] = s;
    wait_lgkm0();
    cta_barrier();
    const float mu = (red[par][0][0] + red[par][0][1] + red[par][0][2] + red[par][0][3]) / d;
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const float a0 = v[c].x - mu, a1 = v[c].y - mu, a2 = v[c].z - mu, a3 = v[c].w - mu;
      q += in[c] ? a0 * a0 + a1 * a1 + a2 * a2 + a3 * a3 : 0.f;
    }
    q = wave_sum(q);
    if (lane == 0) red[par][1][wave] = q;
    wait_lgkm0();
    cta_barrier();
    const float rs = rsqrtf((red[par][1][0] + red[par][1][1] + red[par][1][2] + red[par][1][3]) / d + eps);
    const auto ry = rsrc(y + (long)row * ldy, 2 * d);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const bf16x4 o = {f2bf((v[c].x - mu) * rs * gg[c].x + bb[c].x),
                        f2bf((v[c].y - mu) * rs * gg[c].y + bb[c].y),
                        f2bf((v[c].z - mu) * rs * gg[c].z + bb[c].z),
                        f2bf((v[c].w - mu) * rs * gg[c].w + bb[c].w)};
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, o), ry, 8 * tid, 2048 * c, 0);
    }
    // the statistics: every lane stores, all but thread 0 past the 4-byte range
    const int so = tid == 0 ? 0 : 4;
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, mu), rsrc(mean + row, 4), so, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, rs), rsrc(rstd + row, 4), so, 0, 0);
  };
  const int step = gridDim.x;
  float4 A[NCH], B[NCH];
  int row = blockIdx.x;
  if (row < rows) load(row, true, A);
  vm_pad<NCH + 2>(y);  // a row's stores: NCH chunks of y, mean, rstd
  for (; row < rows; row += 2 * step) {
    load(row + step, row + step < rows, B);
    process(row, 0, A);
    if (row + step >= rows) break;
    load(row + 2 * step, row + 2 * step < rows, A);
    process(row + step, 1, B);
  }
}

// One row of the backward's operands: dy, x and the residual gradient for
// the thread's columns (j * 256 + tid) * 4 .. +3, with the row's statistics.
template <int NC4>
struct LnBwdRow {
  float4 dy[NC4], x[NC4], res[NC4];
  float mu, rs;
};

// Backward: workgroup p owns rows [p * rpb, (p + 1) * rpb); each thread owns
// the columns (j * 256 + tid) * 4 .. +3 and keeps their dg / db partial sums
// in registers, so the workgroup writes one partial row per tensor and needs
// no cross-wave reduction of the columns.  The row loop is software
// pipelined: the next row's dy, x and residual gradient are loaded before the
// current row is reduced and written, into the other of two register sets
// (the loop is unrolled by two, so no set is ever copied and no wait for the
// next row is implied).  Every row access is a buffer instruction, so columns
// past d and a next row that does not exist need no branch (their reads give
// 0, their writes are dropped) and the wait counts stay exact.  The two row
// sums go through LDS in a fixed order (lane tree, then waves 0..3), one
// barrier per row.  dy, x and the residual gradient are read once.  BIAS: a
// third partial row at part_o, the column sums of the updated residual
// gradient (the bias gradient of the product that last fed the residual).
template <int NC4, bool BIAS>
__global__ __launch_bounds__(256) void ln_bwd_kernel(
    const float* __restrict__ dy, long lddy, const float* __restrict__ x, long ldx,
    long row_stride, const float* __restrict__ g, const float* __restrict__ mean,
    const float* __restrict__ rstd, float* __restrict__ dres, long ldres,
    float* __restrict__ part_g, float* __restrict__ part_b, int rows, int d, int rpb,
    bf16* __restrict__ dres_bf, long ldbf, float* __restrict__ part_o) {
  __shared__ float red[2][2][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r0 = blockIdx.x * rpb, r1 = min(rows, r0 + rpb);
  const int vo = 16 * tid;  // byte offset of the thread's columns; column block j adds 4096 j
  float4 gg[NC4], pg[NC4], pb[NC4], po[NC4];
  {
    const auto rg = rsrc(g, 4 * d);
#pragma unroll
    for (int j = 0; j < NC4; ++j) {
      gg[j] = bload4(rg, vo, 4096 * j);
      pg[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      pb[j] = pg[j];
      po[j] = pg[j];
    }
  }
  // row rr's operands, or zeros when !ok (the statistics then come from row
  // r0, an existing row, and are not used)
  auto load = [&](int rr, bool ok, LnBwdRow<NC4>& o) {
    const int rc = ok ? rr : r0;
    o.mu = mean[rc];
    o.rs = rstd[rc];
    const int nb = ok ? 4 * d : 0;
    const auto rd = rsrc(dy + (long)rc * lddy, nb);
    const auto rx = rsrc(x + (long)rc * row_stride * ldx, nb);
    const auto rr_ = rsrc(dres + (long)rc * row_stride * ldres, nb);
#pragma unroll
    for (int j = 0; j < NC4; ++j) {
      o.dy[j] = bload4(rd, vo, 4096 * j);
      o.x[j] = bload4(rx, vo, 4096 * j);
      o.res[j] = bload4(rr_, vo, 4096 * j);
    }
  };
  auto process = [&](int row, int par, const LnBwdRow<NC4>& c) {
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int j = 0; j < NC4; ++j) {
      const float4 v = c.dy[j], xv = c.x[j];
      const float4 h = make_float4((xv.x - c.mu) * c.rs, (xv.y - c.mu) * c.rs,
                                   (xv.z - c.mu) * c.rs, (xv.w - c.mu) * c.rs);
      const float4 gy = make_float4(v.x * gg[j].x, v.y * gg[j].y, v.z * gg[j].z, v.w * gg[j].w);
      s0 += gy.x + gy.y + gy.z + gy.w;  // columns past d: dy = 0, g = 0
      s1 += gy.x * h.x + gy.y * h.y + gy.z * h.z + gy.w * h.w;
    }
    s0 = wave_sum(s0);
    s1 = wave_sum(s1);
    if (lane == 0) {
      red[par][0][wave] = s0;
      red[par][1][wave] = s1;
    }
    wait_lgkm0();
    cta_barrier();
    const float m1 = (red[par][0][0] + red[par][0][1] + red[par][0][2] + red[par][0][3]) / d;
    const float m2 = (red[par][1][0] + red[par][1][1] + red[par][1][2] + red[par][1][3]) / d;
    const auto rw = rsrc(dres + (long)row * row_stride * ldres, 4 * d);
    const auto rb = dres_bf != nullptr ? rsrc(dres_bf + (long)row * ldbf, 2 * d) : rsrc(dres, 0);
#pragma unroll
    for (int j = 0; j < NC4; ++j) {
      const float4 v = c.dy[j], xv = c.x[j];
      const float4 h = make_float4((xv.x - c.mu) * c.rs, (xv.y - c.mu) * c.rs,
                                   (xv.z - c.mu) * c.rs, (xv.w - c.mu) * c.rs);
      float4 o = c.res[j];
      o.x += c.rs * (v.x * gg[j].x - m1 - h.x * m2);
      o.y += c.rs * (v.y * gg[j].y - m1 - h.y * m2);
      o.z += c.rs * (v.z * gg[j].z - m1 - h.z * m2);
      o.w += c.rs * (v.w * gg[j].w - m1 - h.w * m2);
      bstore4(o, rw, vo, 4096 * j);
      const bf16x4 ob = {f2bf(o.x), f2bf(o.y), f2bf(o.z), f2bf(o.w)};
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, ob), rb, 8 * tid, 2048 * j, 0);
      // columns past d: dy = 0, so the partial sums gain nothing there (the
      // sums of o there are not stored)
      pg[j].x += v.x * h.x; pg[j].y += v.y * h.y; pg[j].z += v.z * h.z; pg[j].w += v.w * h.w;
      pb[j].x += v.x; pb[j].y += v.y; pb[j].z += v.z; pb[j].w += v.w;
      if (BIAS) {
        po[j].x += o.x; po[j].y += o.y; po[j].z += o.z; po[j].w += o.w;
      }
    }
  };
  LnBwdRow<NC4> A, B;
  if (r0 < r1) load(r0, true, A);
  vm_pad<2 * NC4>(dres);  // a row's stores: NC4 chunks of the residual gradient and its bf16 copy
  for (int row = r0; row < r1; row += 2) {
    load(row + 1, row + 1 < r1, B);
    process(row, 0, A);
    if (row + 1 >= r1) break;
    load(row + 2, row + 2 < r1, A);
    process(row + 1, 1, B);
  }
  // every workgroup writes its partial rows (zeros when it owns no row)
  const auto rpg = rsrc(part_g + (long)blockIdx.x * d, 4 * d);
  const auto rpb_ = rsrc(part_b + (long)blockIdx.x * d, 4 * d);
#pragma unroll
  for (int j = 0; j < NC4; ++j) {
    bstore4(pg[j], rpg, vo, 4096 * j);
    bstore4(pb[j], rpb_, vo, 4096 * j);
  }
  if (BIAS) {
    const auto rpo = rsrc(part_o + (long)blockIdx.x * d, 4 * d);
#pragma unroll
    for (int j = 0; j < NC4; ++j) bstore4(po[j], rpo, vo, 4096 * j);
  }
}

// out[c] = sum over p of part[p * d + c].  A workgroup owns 16 columns: 64
// row lanes of 4 threads (4 columns each, one 16-byte load per row), then a
// fixed-order tree over the row lanes, so the sum does not depend on timing.
// blockIdx.y = 1 and 2 sum the next arrays of partials, part + y n_part d,
// into out1 and out2 (the LayerNorm backward's partials in one launch).
template <bool VEC>
__global__ __launch_bounds__(256) void colsum_partials_kernel(const float* __restrict__ part0,
                                                              int n_part, int d,
                                                              float* __restrict__ out0,
                                                              float* __restrict__ out1,
                                                              float* __restrict__ out2) {
  __shared__ float4 red[64][4];
  const float* part = part0 + (long)blockIdx.y * n_part * d;
  float* out = blockIdx.y == 0 ? out0 : blockIdx.y == 1 ? out1 : out2;
  const int c4 = threadIdx.x & 3, rl = threadIdx.x >> 2;
  const int c = blockIdx.x * 16 + 4 * c4;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (VEC) {
    if (c < d)
      for (int p = rl; p < n_part; p += 64) {
        const float4 v = *reinterpret_cast<const float4*>(part + (long)p * d + c);
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
      }
  } else {
    for (int p = rl; p < n_part; p += 64) {
      const float* r = part + (long)p * d;
      if (c < d) s.x += r[c];
      if (c + 1 < d) s.y += r[c + 1];
      if (c + 2 < d) s.z += r[c + 2];
      if (c + 3 < d) s.w += r[c + 3];
    }
  }
  red[rl][c4] = s;
  __syncthreads();
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) {
    if (rl < w) {
      const float4 o = red[rl + w][c4];
      float4& t = red[rl][c4];
      t.x += o.x; t.y += o.y; t.z += o.z; t.w += o.w;
    }
    __syncthreads();
  }
  if (rl == 0) {
    const float4 t = red[0][c4];
    if (VEC) {
      if (c < d) *reinterpret_cast<float4*>(out + c) = t;
    } else {
      if (c < d) out[c] = t.x;
      if (c + 1 < d) out[c + 1] = t.y;
      if (c + 2 < d) out[c + 2] = t.z;
      if (c + 3 < d) out[c + 3] = t.w;
    }
  }
}

// Block (x, p) sums rows [p * rpp, min(rows, (p+1) * rpp)) of columns
// [x * 256 * V, (x + 1) * 256 * V), V consecutive columns per thread (one
// 16-byte load per row when VEC, else V = 1).
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void colsum_pass1(const T* __restrict__ X, long ldx, int rows,
                                                    int cols, int rpp, float* __restrict__ part) {
  constexpr int V = VEC ? 16 / (int)sizeof(T) : 1;
  const int p = blockIdx.y;
  const int c = (blockIdx.x * 256 + threadIdx.x) * V;
  if (c >= cols) return;
  const int r0 = p * rpp, r1 = min(rows, r0 + rpp);
  float s[V];
#pragma unroll
  for (int v = 0; v < V; ++v) s[v] = 0.f;
  auto add = [&](const T* src) {
    if constexpr (VEC) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(src);
      const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
      for (int v = 0; v < V; ++v) s[v] += (float)e[v];
    } else {
      s[0] += (float)src[0];
    }
  };
  int r = r0;
  // eight rows' loads issued together (one row at a time waited for each
  // load's full latency); the rows are still added in order
  for (; r + 8 <= r1; r += 8) {
    u32x4 raw[8];
    if constexpr (VEC) {
#pragma unroll
      for (int u = 0; u < 8; ++u) raw[u] = *reinterpret_cast<const u32x4*>(X + (long)(r + u) * ldx + c);
#pragma unroll
      for (int u = 0; u < 8; ++u) add(reinterpret_cast<const T*>(&raw[u]));
    } else {
      T x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = X[(long)(r + u) * ldx + c];
#pragma unroll
      for (int u = 0; u < 8; ++u) s[0] += (float)x[u];
    }
  }
  for (; r < r1; ++r) add(X + (long)r * ldx + c);
#pragma unroll
  for (int v = 0; v < V; ++v) part[(long)p * cols + c + v] = s[v];
}

template <int NC>
hipError_t ln_fwd_launch(const float* x, long ldx, long rs, const float* g, const float* b,
                         bf16* y, long ldy, float* mean, float* rstd, int rows, int d, float eps,
                         hipStream_t s) {
  hipLaunchKernelGGL(ln_fwd_kernel<NC>, dim3(sat_cdiv(rows, 4)), dim3(256), 0, s, x, ldx, rs, g,
                     b, y, ldy, mean, rstd, rows, d, eps);
  return hipGetLastError();
}

template <int NCH>
hipError_t ln_fwd_wg_launch(const float* x, long ldx, long rs, const float* g, const float* b,
                            bf16* y, long ldy, float* mean, float* rstd, int rows, int d, float eps,
                            hipStream_t s) {
  // workgroups that walk rows / grid rows each, two rows in flight per workgroup
  const int grid = rows < LN_FWD_GRID ? rows : LN_FWD_GRID;
  hipLaunchKernelGGL(ln_fwd_wg_kernel<NCH>, dim3(grid), dim3(256), 0, s, x, ldx, rs, g, b, y, ldy,
                     mean, rstd, rows, d, eps);
  return hipGetLastError();
}

template <int NC4>
hipError_t ln_bwd_launch(const float* dy, long lddy, const float* x, long ldx, long rs,
                         const float* g, const float* mean, const float* rstd, float* dres,
                         long ldres, float* pg, float* pb, int rows, int d, int n_part,
                         hipStream_t s, bf16* dres_bf, long ldbf, float* po) {
  // exactly n_part workgroups, so every partial row is written (zeros past the last row)
  const int rpb = sat_cdiv(rows, n_part);
  if (po != nullptr)
    hipLaunchKernelGGL((ln_bwd_kernel<NC4, true>), dim3(n_part), dim3(256), 0, s, dy, lddy, x,
                       ldx, rs, g, mean, rstd, dres, ldres, pg, pb, rows, d, rpb, dres_bf, ldbf, po);
  else
    hipLaunchKernelGGL((ln_bwd_kernel<NC4, false>), dim3(n_part), dim3(256), 0, s, dy, lddy, x,
                       ldx, rs, g, mean, rstd, dres, ldres, pg, pb, rows, d, rpb, dres_bf, ldbf, po);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_layernorm_fwd(const float* x, long ldx, long row_stride, const float* g,
                                const float* b, bf16* y, long ldy, float* mean, float* rstd,
                                int rows, int d, float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d % 4 != 0 || d > 64 * 4 * LN_MAXC || ldx % 4 != 0 || ldy % 4 != 0)
    return hipErrorInvalidValue;
  if (d >= 1024) {
    const int nch = sat_cdiv(d, 1024);
    if (nch <= 1) return ln_fwd_wg_launch<1>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
    if (nch <= 2) return ln_fwd_wg_launch<2>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
    if (nch <= 4) return ln_fwd_wg_launch<4>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
    return ln_fwd_wg_launch<8>(x, ldx, row_stride, g, b, y, ldy, mean, rstd, rows, d, eps, s);
  }
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
                                float* part_b, int rows, int d, int n_part, hipStream_t s,
                                bf16* dres_bf, long ldbf, float* part_o) {
  if (rows <= 0) return hipSuccess;
  if (dres_bf != nullptr && (row_stride != 1 || ldbf % 4 != 0 ||
                             (reinterpret_cast<uintptr_t>(dres_bf) & 7) != 0))
    return hipErrorInvalidValue;
  if (d % 4 != 0 || d > 64 * 4 * 16 || lddy % 4 != 0 || ldx % 4 != 0 || ldres % 4 != 0 ||
      n_part <= 0)
    return hipErrorInvalidValue;
  const int nc = sat_cdiv(d, 1024);
#define LNB(NC) ln_bwd_launch<NC>(dy, lddy, x, ldx, row_stride, g, mean, rstd, dres, ldres, part_g, part_b, rows, d, n_part, s, dres_bf, ldbf, part_o)
  if (nc <= 1) return LNB(1);
  if (nc <= 2) return LNB(2);
  return LNB(4);
#undef LNB
}

// Workgroups (and partial rows) of the backward: 512 for rows wider than 1024
// (two per CU, each with two rows of 3 x 4 d bytes in flight), 1024 for
// narrower rows, which need more workgroups for the same bytes in flight.
// Fewer partial rows also shorten the column sums that follow.
int ln_bwd_parts(int rows, int d) {
  const int cap = d > 1024 ? 512 : 1024;
  return rows < cap ? rows : cap;
}

static hipError_t colsum_partials(const float* part, int n_part, int d, float* out0, float* out1,
                                  float* out2, int n_arrays, hipStream_t s) {
  if (d <= 0) return hipSuccess;
  auto a16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  const bool vec = d % 4 == 0 && a16(part) && a16(out0) && a16(out1) && a16(out2);
  const dim3 grid(sat_cdiv(d, 16), n_arrays);
  if (vec)
    hipLaunchKernelGGL(colsum_partials_kernel<true>, grid, dim3(256), 0, s, part, n_part, d, out0,
                       out1, out2);
  else
    hipLaunchKernelGGL(colsum_partials_kernel<false>, grid, dim3(256), 0, s, part, n_part, d, out0,
                       out1, out2);
  return hipGetLastError();
}

hipError_t launch_colsum_partials(const float* part, int n_part, int d, float* out,
                                  hipStream_t s) {
  return colsum_partials(part, n_part, d, out, out, out, 1, s);
}

hipError_t launch_ln_bwd_colsums(const float* part, int n_part, int d, float* dg, float* db,
                                 hipStream_t s, float* dbias) {
  return colsum_partials(part, n_part, d, dg, db, dbias ? dbias : db, dbias ? 3 : 2, s);
}

template <typename T>
static hipError_t colsum_any(const T* X, long ldx, int rows, int cols, float* part, int n_part,
                             float* out, hipStream_t s) {
  if (cols <= 0) return hipSuccess;
  if (rows <= 0 || n_part <= 0) return hipErrorInvalidValue;
  const int rpp = sat_cdiv(rows, n_part);
  const int np = sat_cdiv(rows, rpp);
  constexpr int V = 16 / (int)sizeof(T);
  const bool vec = cols % V == 0 && ldx % V == 0 && reinterpret_cast<uintptr_t>(X) % 16 == 0;
  if (vec)
    hipLaunchKernelGGL((colsum_pass1<T, true>), dim3(sat_cdiv(cols, 256 * V), np), dim3(256), 0, s, X,
                       ldx, rows, cols, rpp, part);
  else
    hipLaunchKernelGGL((colsum_pass1<T, false>), dim3(sat_cdiv(cols, 256), np), dim3(256), 0, s, X, ldx,
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
