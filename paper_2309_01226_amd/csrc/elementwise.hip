// Bandwidth-bound kernels of the fine-tuning step: rotary embedding, token
// embedding forward / deterministic backward, ViT patch extraction and token
// assembly, softmax cross-entropy, the fused AdamW update, the counter-based
// parameter initialisation and small helpers.  All reductions run in a fixed
// order (no floating-point atomics), so every step is bitwise reproducible.
#include <math.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "adamw_math.h"

namespace {

// ---------------------------------------------------------------- rotary
// Angle of pair i at position pos: pos * 10000^(-2i/rd), in double precision,
// rounded to float cos / sin once.
__device__ __forceinline__ void rope_cs(int pos, int i, int rd, float& c, float& sn) {
  const double ang = (double)pos * pow(10000.0, -2.0 * i / (double)rd);
  double sd, cd;
  sincos(ang, &sd, &cd);
  c = (float)cd;
  sn = (float)sd;
}

__global__ void rope_table_kernel(float2* __restrict__ cs, int S, int rd) {
  const int half = rd / 2;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)S * half) return;
  float c, sn;
  rope_cs((int)(idx / half), (int)(idx % half), rd, c, sn);
  cs[idx] = make_float2(c, sn);
}

// One thread per (token, q or k head, 8 dims = 4 pairs) of the rotated part:
// one 16-byte load and store, the 2x2 rotation (or its transpose for
// backward) of each pair with cos / sin from the table cs[pos][i] when given
// (the same values computed inline otherwise).  Needs rd % 8 == 0, dh and ld
// multiples of 8 and a 16-byte aligned buffer (launch_rotary checks).
__global__ void rotary8_kernel(bf16* __restrict__ qk, long ld, int T, int S, int H, int dh, int rd,
                               int inverse, const float2* __restrict__ cs) {
  const int c8 = rd / 8;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)T * 2 * H * c8) return;
  const int c = idx % c8;
  const long th = idx / c8;
  const int hh = th % (2 * H);  // q heads, then k heads
  const int t = (int)(th / (2 * H));
  const int pos = t % S;
  u32x4* p = reinterpret_cast<u32x4*>(qk + (long)t * ld + (long)hh * dh + 8 * c);
  u32x4 w = *p;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = 4 * c + j;
    float cc, sn;
    if (cs != nullptr) {
      const float2 v = cs[(long)pos * (rd / 2) + i];
      cc = v.x;
      sn = v.y;
    } else {
      rope_cs(pos, i, rd, cc, sn);
    }
    const float s = inverse ? -sn : sn;
    const float x0 = __uint_as_float(w[j] << 16), x1 = __uint_as_float(w[j] & 0xFFFF0000u);
    const bf16 y0 = f2bf(x0 * cc - x1 * s), y1 = f2bf(x0 * s + x1 * cc);
    w[j] = (uint32_t)__builtin_bit_cast(uint16_t, y0) | ((uint32_t)__builtin_bit_cast(uint16_t, y1) << 16);
  }
  *p = w;
}

// General form (any even rd): one thread per (token, pair i), all heads,
// with the same arithmetic.  Consecutive threads take consecutive pairs, so
// each head's rotated part is read and written as one contiguous piece (a
// pair is one 4-byte word).
__global__ void rotary_kernel(bf16* __restrict__ qk, long ld, int T, int S, int H, int dh, int rd,
                              int inverse, const float2* __restrict__ cs) {
  const int half = rd / 2;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)T * half) return;
  const int i = idx % half;
  const int t = (int)(idx / half);
  const int pos = t % S;
  float c, sn;
  if (cs != nullptr) {
    const float2 v = cs[(long)pos * half + i];
    c = v.x;
    sn = v.y;
  } else {
    rope_cs(pos, i, rd, c, sn);
  }
  const float s = inverse ? -sn : sn;
  bf16* row = qk + (long)t * ld + 2 * i;
  for (int hh = 0; hh < 2 * H; ++hh) {  // q heads, then k heads
    uint32_t* p = reinterpret_cast<uint32_t*>(row + (long)hh * dh);
    const uint32_t w = *p;
    const float x0 = __uint_as_float(w << 16), x1 = __uint_as_float(w & 0xFFFF0000u);
    const bf16 y0 = f2bf(x0 * c - x1 * s), y1 = f2bf(x0 * s + x1 * c);
    *p = (uint32_t)__builtin_bit_cast(uint16_t, y0) |
         ((uint32_t)__builtin_bit_cast(uint16_t, y1) << 16);
  }
}

// ---------------------------------------------------------------- embedding
__global__ void embed_fwd_kernel(const int32_t* __restrict__ tok, const float* __restrict__ wte,
                                 const float* __restrict__ wpe, float* __restrict__ h, int T,
                                 int S, int d) {
  const int d4 = d / 4;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)T * d4) return;
  int t = idx / d4, c = (idx % d4) * 4;
  float4 v = *reinterpret_cast<const float4*>(wte + (long)tok[t] * d + c);
  if (wpe != nullptr) {
    float4 w = *reinterpret_cast<const float4*>(wpe + (long)(t % S) * d + c);
    v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
  }
  *reinterpret_cast<float4*>(h + (long)t * d + c) = v;
}

// Sorts the keys (token << 15 | position) of T <= 16384 tokens with a bitonic
// network in LDS (one workgroup); keys are unique, so the order is unique.
// Longer inputs are processed in chunks of this many positions.
constexpr int EMB_MAXT = 16384;
__global__ __launch_bounds__(1024) void embed_sort_kernel(const int32_t* __restrict__ tok, int T,
                                                          int32_t* __restrict__ sorted) {
  __shared__ uint32_t key[EMB_MAXT];
  int n = 1;
  while (n < T) n <<= 1;
  for (int i = threadIdx.x; i < n; i += blockDim.x)
    key[i] = (i < T) ? (((uint32_t)tok[i] << 15) | (uint32_t)i) : 0xFFFFFFFFu;
  __syncthreads();
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n; i += blockDim.x) {
        int ixj = i ^ j;
        if (ixj > i) {
          uint32_t a = key[i], b = key[ixj];
          bool up = (i & k) == 0;
          if ((a > b) == up) {
            key[i] = b;
            key[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int i = threadIdx.x; i < T; i += blockDim.x) sorted[i] = (int32_t)key[i];
}

// One wavefront per vocabulary row v: binary-search v's run in the sorted
// keys, sum the matching dh rows in increasing position order, write the row
// (zeros when v does not occur).
// Row v of dwte = the sum, in position order, of dh over the positions holding
// token v (ACC: added to the row's current value, for the chunks after the first).
template <bool ACC>
__global__ __launch_bounds__(256) void embed_bwd_rows_kernel(const int32_t* __restrict__ sorted,
                                                             int T, const float* __restrict__ dh,
                                                             float* __restrict__ dwte, int d,
                                                             int V) {
  const int lane = threadIdx.x & 63;
  const int v = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (v >= V) return;
  const uint32_t lo_key = (uint32_t)v << 15;
  int lo = 0, hi = T;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if ((uint32_t)sorted[mid] < lo_key) lo = mid + 1;
    else hi = mid;
  }
  int end = lo;
  while (end < T && ((uint32_t)sorted[end] >> 15) == (uint32_t)v) ++end;
  float* out = dwte + (long)v * d;
  for (int c = lane * 4; c < d; c += 256) {
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = lo; j < end; ++j) {
      int t = sorted[j] & 0x7FFF;
      float4 x = *reinterpret_cast<const float4*>(dh + (long)t * d + c);
      s.x += x.x; s.y += x.y; s.z += x.z; s.w += x.w;
    }
    if (ACC) {
      const float4 o = *reinterpret_cast<const float4*>(out + c);
      s.x = o.x + s.x; s.y = o.y + s.y; s.z = o.z + s.z; s.w = o.w + s.w;
    }
    *reinterpret_cast<float4*>(out + c) = s;
  }
}

// ---------------------------------------------------------------- ViT
// Rows of pitch ldo >= pd; the padding columns pd .. ldo - 1 are written as 0.
__global__ void patchify_kernel(const float* __restrict__ img, bf16* __restrict__ out, int B,
                                int C, int I, int p, int ldo) {
  const int g = I / p, np = g * g, pd = C * p * p;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)B * np * ldo) return;
  int col = idx % ldo;
  long row = idx / ldo;
  if (col >= pd) {
    out[idx] = f2bf(0.f);
    return;
  }
  int i = row % np, b = row / np;
  int c = col / (p * p), kh = (col / p) % p, kw = col % p;
  int pr = i / g, pc = i % g;
  out[idx] = f2bf(img[(((long)b * C + c) * I + pr * p + kh) * I + pc * p + kw]);
}

__global__ void vit_assemble_kernel(const float* __restrict__ z, const float* __restrict__ cls,
                                    const float* __restrict__ pos, float* __restrict__ h, int B,
                                    int np, int d) {
  const int S = np + 1;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)B * S * d) return;
  int c = idx % d;
  long r = idx / d;
  int s = r % S, b = r / S;
  float base = (s == 0) ? cls[c] : z[((long)b * np + s - 1) * d + c];
  h[idx] = base + pos[(long)s * d + c];
}

// dz[b*np + i, :] = bf16(dh[b*S + 1 + i, :])
__global__ void vit_patch_grad_kernel(const float* __restrict__ dh, bf16* __restrict__ dz, int B,
                                      int np, int d) {
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)B * np * d) return;
  int c = idx % d;
  long r = idx / d;
  int i = r % np, b = r / np;
  dz[idx] = f2bf(dh[((long)b * (np + 1) + 1 + i) * d + c]);
}

__global__ void f32_to_bf16_kernel(const float* __restrict__ x, long ldx, bf16* __restrict__ y,
                                   long ldy, int rows, int cols) {
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)rows * cols) return;
  int c = idx % cols;
  long r = idx / cols;
  y[r * ldy + c] = f2bf(x[r * ldx + c]);
}

// dst[c, r] = src[r, c] for a bf16 [rows, cols] matrix, rows and cols
// multiples of 8.  Each lane moves 8 x 8 blocks: eight 16-byte row loads, a
// transpose by byte permutes (element j of rows 2e and 2e + 1 into one
// dword), eight 16-byte column stores; eight lanes cover 128 contiguous bytes
// on both sides.  TNB blocks per lane along the columns (a workgroup covers
// 128 x 128 TNB): four (32 loads in flight per lane) measured up to 20%
// faster than one on [4096, 28672] and [4096, 4096] activations; matrices of
// at most 3072 columns take two, which gives them twice the workgroups
// ([8192, 768]: 8.9 -> 6.5 us; [8192, 3072]: 24.3 -> 20.8 us).
template <int TNB>
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const bf16* __restrict__ src,
                                                             long lds, bf16* __restrict__ dst,
                                                             long ldd, int rows, int cols) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.y * 128 + (wave >> 1) * 64 + (lane >> 3) * 8;
  const int cb = blockIdx.x * 128 * TNB + (wave & 1) * 64 * TNB + (lane & 7) * 8;
  if (r0 >= rows) return;
  u32x4 v[TNB][8];
#pragma unroll
  for (int b = 0; b < TNB; ++b) {
    const int c0 = cb + 64 * b;
    if (c0 < cols) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        v[b][i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + (long)(r0 + i) * lds + c0));
    }
  }
#pragma unroll
  for (int b = 0; b < TNB; ++b) {
    const int c0 = cb + 64 * b;
    if (c0 >= cols) break;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = __builtin_amdgcn_perm(v[b][2 * e + 1][j >> 1], v[b][2 * e][j >> 1], sel);
      __builtin_nontemporal_store(o, reinterpret_cast<u32x4*>(dst + (long)(c0 + j) * ldd + r0));
    }
  }
}

// out[s, c] = sum_b dh[(b*S + s) * d + c]
__global__ void sum_rows_batched_kernel(const float* __restrict__ dh, float* __restrict__ out,
                                        int B, int S, int d) {
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)S * d) return;
  float s = 0.f;
  for (int b = 0; b < B; ++b) s += dh[(long)b * S * d + idx];
  out[idx] = s;
}

// ---------------------------------------------------------------- cross-entropy
__device__ __forceinline__ float block_reduce_sum_256(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return sh[0] + sh[1] + sh[2] + sh[3];
}
__device__ __forceinline__ float block_reduce_max_256(float v, float* sh) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3]));
}

// One 256-thread block per row: online (max, sum exp) in one pass, block
// combine, then dz = (exp(z - lse) - onehot) * inv_n in a second pass.
__global__ __launch_bounds__(256) void xent_kernel(const float* __restrict__ z, long ldz,
                                                   const int32_t* __restrict__ labels, int V,
                                                   float* __restrict__ row_loss,
                                                   bf16* __restrict__ dz, long lddz,
                                                   const float* __restrict__ inv_n_p) {
  __shared__ float sh[4];
  const int row = blockIdx.x;
  const float* zr = z + (long)row * ldz;
  const int y = labels[row];
  float m = -INFINITY, s = 0.f;
  for (int c = threadIdx.x; c < V; c += 256) {
    float x = zr[c];
    if (x > m) {
      s = s * __expf(m - x) + 1.f;
      m = x;
    } else {
      s += __expf(x - m);
    }
  }
  const float M = block_reduce_max_256(m, sh);
  float sl = (m == -INFINITY) ? 0.f : s * __expf(m - M);
  const float tot = block_reduce_sum_256(sl, sh);
  const float lse = M + __logf(tot);
  bf16* dr = dz + (long)row * lddz;
  if (y < 0) {
    const int cend = min((long)((V + 7) & ~7), lddz);
    for (int c = threadIdx.x; c < cend; c += 256) dr[c] = f2bf(0.f);
    if (threadIdx.x == 0) row_loss[row] = 0.f;
    return;
  }
  const float inv_n = *inv_n_p;
  for (int c = threadIdx.x; c < V; c += 256) {
    float pr = __expf(zr[c] - lse);
    dr[c] = f2bf((pr - (c == y ? 1.f : 0.f)) * inv_n);
  }
  // zero the row padding up to the next multiple of 8 columns (within lddz)
  const int cpad = min((long)((V + 7) & ~7), lddz);
  for (int c = V + threadIdx.x; c < cpad; c += 256) dr[c] = f2bf(0.f);
  if (threadIdx.x == 0) row_loss[row] = lse - zr[y];
}

// Rows that fit in the registers of one workgroup (NT threads, thread t
// holding columns 4 t + 4 NT g .. + 3 for g < NV4): the logits are read once
// and exp is taken once per element: p = exp(z - max), lse = max + log(sum p),
// dz = (p / sum p - onehot) * inv_n.  Block max and sum go through LDS in a
// fixed order.  Row reads and writes are buffer instructions (one VGPR offset
// per thread, the group offset in the scalar offset, so the row's addresses
// take no registers) with the non-temporal hint: the logits are read once and
// the gradient is consumed by the next kernel from HBM.  At 512 threads two
// workgroups share a CU, so one row's reads overlap the other's writes.
// FULL: the host has checked that every group but the last lies inside the
// row (4 NT (NV4 - 1) <= V), so only the last one is tested.
template <int NT, int NV4, bool FULL>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(4, 4)))
void xent_reg_kernel(const float* __restrict__ z, long ldz, const int32_t* __restrict__ labels,
                     int V, float* __restrict__ row_loss, bf16* __restrict__ dz, long lddz,
                     const float* __restrict__ inv_n_p) {
  constexpr int NW = NT / 64, GS = 4 * NT;  // waves, columns per group
  constexpr int NT_HINT = 2;                 // buffer cache policy: non-temporal
  __shared__ float red[2][NW];
  const int row = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* zr = z + (long)row * ldz;
  bf16* dr = dz + (long)row * lddz;
  const int y = labels[row];
  const int cpad = (int)min((long)((V + 7) & ~7), lddz);  // zero the row padding too
  const __amdgpu_buffer_rsrc_t rz =
      __builtin_amdgcn_make_buffer_rsrc((void*)zr, (short)0, V * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rd =
      __builtin_amdgcn_make_buffer_rsrc((void*)dr, (short)0, cpad * 2, 0x00020000);
  floatx4 v[NV4];
#pragma unroll
  for (int g = 0; g < NV4; ++g) {
    const int c = 4 * t + GS * g;
    v[g] = floatx4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    // the first two tests are uniform: the whole group lies in the row
    if ((FULL && g < NV4 - 1) || GS * (g + 1) <= V || c + 3 < V) {
      v[g] = __builtin_bit_cast(
          floatx4, __builtin_amdgcn_raw_buffer_load_b128(rz, 16 * t, 4 * GS * g, NT_HINT));
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (c + e < V)
          v[g][e] = __builtin_bit_cast(
              float, __builtin_amdgcn_raw_buffer_load_b32(rz, 16 * t + 4 * e, 4 * GS * g, NT_HINT));
    }
  }
  // the label's logit, read while the row is still arriving
  const float zy = (t == 0 && y >= 0)
                       ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rz, 4 * y, 0, 0))
                       : 0.f;
  float m = -INFINITY;
#pragma unroll
  for (int g = 0; g < NV4; ++g)
#pragma unroll
    for (int e = 0; e < 4; ++e) m = fmaxf(m, v[g][e]);
  m = wave_max(m);
  if (lane == 0) red[0][wave] = m;
  __syncthreads();
  float M = red[0][0];
#pragma unroll
  for (int w = 1; w < NW; ++w) M = fmaxf(M, red[0][w]);
  float s = 0.f;
#pragma unroll
  for (int g = 0; g < NV4; ++g)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[g][e] = __expf(v[g][e] - M);  // exp(-inf) = 0 past V
      s += v[g][e];
    }
  s = wave_sum(s);
  if (lane == 0) red[1][wave] = s;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) tot += red[1][w];
  const float lse = M + __logf(tot);
  const float inv_n = y < 0 ? 0.f : *inv_n_p;
  const float rt = 1.f / tot;
#pragma unroll
  for (int g = 0; g < NV4; ++g) {
    const int c = 4 * t + GS * g;
    if (c >= cpad) continue;
    bf16x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float pr = c + e < V ? v[g][e] * rt : 0.f;
      o[e] = f2bf((pr - (c + e == y ? 1.f : 0.f)) * inv_n);
    }
    if ((FULL && g < NV4 - 1) || GS * (g + 1) <= cpad || c + 3 < cpad) {
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, o), rd, 8 * t, 2 * GS * g,
                                            NT_HINT);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (c + e < cpad)
          __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, o[e]), rd,
                                                8 * t + 2 * e, 2 * GS * g, NT_HINT);
    }
  }
  if (t == 0) row_loss[row] = y < 0 ? 0.f : lse - zy;
}

// Single block: out[0] = (sum of row_loss in a fixed tree order) * inv_n.
__global__ __launch_bounds__(256) void loss_finalize_kernel(const float* __restrict__ row_loss,
                                                            int n, const float* __restrict__ inv_n,
                                                            float* __restrict__ out) {
  __shared__ float sh[4];
  double acc = 0.0;
  for (int i = threadIdx.x; i < n; i += 256) acc += row_loss[i];
  float v = block_reduce_sum_256((float)acc, sh);
  if (threadIdx.x == 0) out[0] = v * inv_n[0];
}

__global__ __launch_bounds__(256) void count_valid_kernel(const int32_t* __restrict__ labels,
                                                          int n, float* __restrict__ inv_n) {
  __shared__ float sh[4];
  float c = 0.f;
  for (int i = threadIdx.x; i < n; i += 256) c += (labels[i] >= 0) ? 1.f : 0.f;
  float tot = block_reduce_sum_256(c, sh);
  if (threadIdx.x == 0) inv_n[0] = 1.f / fmaxf(tot, 1.f);
}

// ---------------------------------------------------------------- AdamW
// Grid-stride over float4 groups, two groups per iteration with all eight
// loads issued first.  Every byte is touched once per step, so loads and
// stores are non-temporal (they stream past the caches).
__global__ __launch_bounds__(256) void adamw_kernel(float* __restrict__ p,
                                                    const float* __restrict__ g,
                                                    float* __restrict__ m, float* __restrict__ v,
                                                    bf16* __restrict__ shadow, long n4, long n,
                                                    AdamWConsts c) {
  const long stride = (long)gridDim.x * blockDim.x;
  floatx4* P = reinterpret_cast<floatx4*>(p);
  const floatx4* G = reinterpret_cast<const floatx4*>(g);
  floatx4* Mo = reinterpret_cast<floatx4*>(m);
  floatx4* Vo = reinterpret_cast<floatx4*>(v);
  bf16x4* Sh = reinterpret_cast<bf16x4*>(shadow);
  long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + stride < n4; i += 2 * stride) {
    floatx4 pp[2], gg[2], mm[2], vv[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const long j = i + u * stride;
      pp[u] = __builtin_nontemporal_load(P + j);
      gg[u] = __builtin_nontemporal_load(G + j);
      mm[u] = __builtin_nontemporal_load(Mo + j);
      vv[u] = __builtin_nontemporal_load(Vo + j);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const long j = i + u * stride;
      adamw_four(pp[u], gg[u], mm[u], vv[u], c);
      __builtin_nontemporal_store(pp[u], P + j);
      __builtin_nontemporal_store(mm[u], Mo + j);
      __builtin_nontemporal_store(vv[u], Vo + j);
      if (shadow != nullptr) {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = f2bf(pp[u][e]);
        __builtin_nontemporal_store(o, Sh + j);
      }
    }
  }
  for (; i < n4; i += stride) {
    floatx4 pp = P[i], mm = Mo[i], vv = Vo[i];
    adamw_four(pp, G[i], mm, vv, c);
    P[i] = pp;
    Mo[i] = mm;
    Vo[i] = vv;
    if (shadow != nullptr) {
      bf16x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = f2bf(pp[e]);
      Sh[i] = o;
    }
  }
  // scalar tail (n not a multiple of 4, or unaligned pointers)
  long t = n4 * 4 + (long)blockIdx.x * blockDim.x + threadIdx.x;
  for (; t < n; t += stride) {
    float pp = p[t], mm = m[t], vv = v[t];
    adamw_one(pp, g[t], mm, vv, c);
    p[t] = pp; m[t] = mm; v[t] = vv;
    if (shadow != nullptr) shadow[t] = f2bf(pp);
  }
}

// ---------------------------------------------------------------- init
// Philox4x32-10 (Salmon et al., SC'11) keyed by the seed, counter =
// (pair index, tensor id); Box-Muller turns its outputs into two normals.
__device__ __forceinline__ void philox_round(uint32_t& c0, uint32_t& c1, uint32_t& c2,
                                             uint32_t& c3, uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  uint32_t hi0 = __umulhi(M0, c0), lo0 = M0 * c0;
  uint32_t hi1 = __umulhi(M1, c2), lo1 = M1 * c2;
  uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
  c0 = n0; c1 = n1; c2 = n2; c3 = n3;
}
__device__ __forceinline__ void philox4x32_10(uint32_t ctr[4], uint32_t k0, uint32_t k1) {
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    philox_round(ctr[0], ctr[1], ctr[2], ctr[3], k0, k1);
    k0 += W0;
    k1 += W1;
  }
}

__global__ void init_normal_kernel(float* __restrict__ p, bf16* __restrict__ shadow, long n,
                                   uint32_t k0, uint32_t k1, uint32_t stream_id, float std) {
  long pair = (long)blockIdx.x * blockDim.x + threadIdx.x;
  long i0 = pair * 2;
  if (i0 >= n) return;
  uint32_t c[4] = {(uint32_t)pair, (uint32_t)(pair >> 32), stream_id, 0x5A17u};
  philox4x32_10(c, k0, k1);
  // uniforms in (0, 1]: (x + 1) * 2^-32 with 24-bit mantissa safety
  float u1 = ((c[0] >> 8) + 1) * (1.0f / 16777216.0f);
  float u2 = (c[1] >> 8) * (1.0f / 16777216.0f);
  float r = sqrtf(-2.f * __logf(u1));
  float sn, cs;
  __sincosf(6.283185307179586f * u2, &sn, &cs);
  float z0 = r * cs * std, z1 = r * sn * std;
  p[i0] = z0;
  if (shadow) shadow[i0] = f2bf(z0);
  if (i0 + 1 < n) {
    p[i0 + 1] = z1;
    if (shadow) shadow[i0 + 1] = f2bf(z1);
  }
}

__global__ void fill_kernel(float* __restrict__ p, bf16* __restrict__ shadow, long n, float v) {
  long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  p[i] = v;
  if (shadow) shadow[i] = f2bf(v);
}

__global__ void zero_kernel(uint32_t* __restrict__ p, long n) {
  const long stride = (long)gridDim.x * blockDim.x;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0u;
}

inline unsigned blocks_for(long n, int bs = 256) { return (unsigned)((n + bs - 1) / bs); }

}  // namespace

hipError_t launch_rope_table(float2* cs, int S, int rd, hipStream_t s) {
  if (rd <= 0 || S <= 0) return hipSuccess;
  if (rd % 2) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks_for((long)S * (rd / 2))), dim3(256), 0, s, cs, S, rd);
  return hipGetLastError();
}

hipError_t launch_rotary(bf16* qk, long ld, int B, int S, int H, int dh, int rd, int inverse,
                         hipStream_t s, const float2* cs) {
  if (rd <= 0) return hipSuccess;
  if (rd % 2 || rd > dh || ld % 2 || dh % 2 || (reinterpret_cast<uintptr_t>(qk) & 3))
    return hipErrorInvalidValue;
  if (rd % 8 == 0 && dh % 8 == 0 && ld % 8 == 0 && (reinterpret_cast<uintptr_t>(qk) & 15) == 0) {
    const long total = (long)B * S * 2 * H * (rd / 8);
    hipLaunchKernelGGL(rotary8_kernel, dim3(blocks_for(total)), dim3(256), 0, s, qk, ld, B * S, S, H,
                       dh, rd, inverse, cs);
    return hipGetLastError();
  }
  long total = (long)B * S * (rd / 2);
  hipLaunchKernelGGL(rotary_kernel, dim3(blocks_for(total)), dim3(256), 0, s, qk, ld, B * S, S, H,
                     dh, rd, inverse, cs);
  return hipGetLastError();
}

hipError_t launch_embed_fwd(const int32_t* tok, const float* wte, const float* wpe, float* h,
                            int T, int S, int d, int V, hipStream_t s) {
  (void)V;
  if (T <= 0) return hipSuccess;
  if (d % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_fwd_kernel, dim3(blocks_for((long)T * d / 4)), dim3(256), 0, s, tok,
                     wte, wpe, h, T, S, d);
  return hipGetLastError();
}

// Positions are taken in chunks of EMB_MAXT, in order, one after the other on
// the stream: the first chunk writes every row's sum, later chunks add theirs.
// work holds one chunk's sorted keys (min(T, EMB_MAXT) entries).
hipError_t launch_embed_bwd(const int32_t* tok, const float* dh, float* dwte, int T, int d, int V,
                            int32_t* work, hipStream_t s) {
  if (T <= 0 || d % 4 || V <= 0 || V >= (1 << 16)) return hipErrorInvalidValue;
  for (int t0 = 0; t0 < T; t0 += EMB_MAXT) {
    const int n = T - t0 < EMB_MAXT ? T - t0 : EMB_MAXT;
    hipLaunchKernelGGL(embed_sort_kernel, dim3(1), dim3(1024), 0, s, tok + t0, n, work);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const float* dhc = dh + (long)t0 * d;
    if (t0 == 0)
      hipLaunchKernelGGL(embed_bwd_rows_kernel<false>, dim3(sat_cdiv(V, 4)), dim3(256), 0, s, work,
                         n, dhc, dwte, d, V);
    else
      hipLaunchKernelGGL(embed_bwd_rows_kernel<true>, dim3(sat_cdiv(V, 4)), dim3(256), 0, s, work,
                         n, dhc, dwte, d, V);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_patchify(const float* img, bf16* out, int B, int C, int I, int p, int ldo,
                           hipStream_t s) {
  if (ldo < C * p * p) return hipErrorInvalidValue;
  long total = (long)B * (I / p) * (I / p) * ldo;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(patchify_kernel, dim3(blocks_for(total)), dim3(256), 0, s, img, out, B, C, I,
                     p, ldo);
  return hipGetLastError();
}

hipError_t launch_vit_assemble(const float* z, const float* cls, const float* pos, float* h,
                               int B, int np, int d, hipStream_t s) {
  long total = (long)B * (np + 1) * d;
  hipLaunchKernelGGL(vit_assemble_kernel, dim3(blocks_for(total)), dim3(256), 0, s, z, cls, pos,
                     h, B, np, d);
  return hipGetLastError();
}

hipError_t launch_vit_patch_grad(const float* dh, bf16* dz, int B, int np, int d, hipStream_t s) {
  long total = (long)B * np * d;
  hipLaunchKernelGGL(vit_patch_grad_kernel, dim3(blocks_for(total)), dim3(256), 0, s, dh, dz, B,
                     np, d);
  return hipGetLastError();
}

hipError_t launch_f32_to_bf16(const float* x, long ldx, bf16* y, long ldy, int rows, int cols,
                              hipStream_t s) {
  long total = (long)rows * cols;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(blocks_for(total)), dim3(256), 0, s, x, ldx, y, ldy,
                     rows, cols);
  return hipGetLastError();
}

hipError_t launch_transpose_bf16(const bf16* src, long lds, bf16* dst, long ldd, int rows,
                                int cols, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (rows % 8 || cols % 8 || lds % 8 || ldd % 8 || lds < cols || ldd < rows ||
      (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16)
    return hipErrorInvalidValue;
  if (cols <= 3072) {
    dim3 grid((unsigned)((cols + 255) / 256), (unsigned)((rows + 127) / 128));
    hipLaunchKernelGGL(transpose_bf16_kernel<2>, grid, dim3(256), 0, s, src, lds, dst, ldd, rows, cols);
  } else {
    dim3 grid((unsigned)((cols + 511) / 512), (unsigned)((rows + 127) / 128));
    hipLaunchKernelGGL(transpose_bf16_kernel<4>, grid, dim3(256), 0, s, src, lds, dst, ldd, rows, cols);
  }
  return hipGetLastError();
}

hipError_t launch_sum_rows_batched(const float* dh, float* out, int B, int S, int d,
                                   hipStream_t s) {
  long total = (long)S * d;
  hipLaunchKernelGGL(sum_rows_batched_kernel, dim3(blocks_for(total)), dim3(256), 0, s, dh, out,
                     B, S, d);
  return hipGetLastError();
}

hipError_t launch_xent(const float* z, long ldz, const int32_t* labels, int N, int V,
                       float* row_loss, bf16* dz, long lddz, const float* inv_n, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  // rows in registers: 512 threads (two workgroups per CU) for up to 12
  // groups of 2048 logits and for exactly 25 (the GPT vocabularies), 1024
  // threads for up to 13 groups of 4096
  const bool reg = V <= 13 * 4096 && ldz % 4 == 0 && lddz % 4 == 0 &&
                   (reinterpret_cast<uintptr_t>(z) & 15) == 0 && (reinterpret_cast<uintptr_t>(dz) & 7) == 0;
  const int g512 = (V + 2047) / 2048;
#define XREG(NT, NV, FULL) hipLaunchKernelGGL((xent_reg_kernel<NT, NV, FULL>), dim3(N), dim3(NT), 0, s, \
                                              z, ldz, labels, V, row_loss, dz, lddz, inv_n)
  if (reg && g512 <= 1) XREG(512, 1, false);
  else if (reg && g512 <= 4) XREG(512, 4, false);
  else if (reg && g512 <= 8) XREG(512, 8, false);
  else if (reg && g512 <= 12) XREG(512, 12, false);
  else if (reg && g512 == 25) XREG(512, 25, true);
  else if (reg) XREG(1024, 13, false);
  else
    hipLaunchKernelGGL(xent_kernel, dim3(N), dim3(256), 0, s, z, ldz, labels, V, row_loss, dz, lddz,
                       inv_n);
#undef XREG
  return hipGetLastError();
}

hipError_t launch_loss_finalize(const float* row_loss, int n, const float* inv_n, float* out,
                                hipStream_t s) {
  hipLaunchKernelGGL(loss_finalize_kernel, dim3(1), dim3(256), 0, s, row_loss, n, inv_n, out);
  return hipGetLastError();
}

// Synthetic batches for profiling runs: a 32-bit integer hash (the finaliser
// of MurmurHash3) of (seed, index) gives uniform tokens, labels and image
// values; token stream b is hashed at positions 0 .. S, inputs take 0 .. S-1
// and labels 1 .. S (the next token).
__device__ __forceinline__ uint32_t mix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}
__device__ __forceinline__ uint32_t hash2(uint32_t seed, uint32_t i) {
  return mix32(mix32(seed ^ 0x9E3779B9u) + i);
}

__global__ void synth_tokens_kernel(int32_t* __restrict__ x, int32_t* __restrict__ y, int B, int S,
                                    int V, uint32_t seed) {
  const long n = (long)B * S;
  for (long t = (long)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += (long)gridDim.x * blockDim.x) {
    const long b = t / S, s = t % S;
    const uint32_t base = (uint32_t)(b * (S + 1) + s);
    x[t] = (int32_t)(hash2(seed, base) % (uint32_t)V);
    y[t] = (int32_t)(hash2(seed, base + 1) % (uint32_t)V);
  }
}

__global__ void synth_images_kernel(float* __restrict__ img, long n, int32_t* __restrict__ y, int B,
                                    int classes, uint32_t seed) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    img[i] = (float)(hash2(seed, (uint32_t)i) >> 8) * (2.f / 16777216.f) - 1.f;  // uniform [-1, 1)
  const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < B) y[t] = (int32_t)(hash2(seed ^ 0x5bd1e995u, (uint32_t)t) % (uint32_t)classes);
}

hipError_t launch_synth_tokens(int32_t* x, int32_t* y, int B, int S, int V, uint32_t seed,
                               hipStream_t s) {
  if ((long)B * S <= 0) return hipSuccess;
  hipLaunchKernelGGL(synth_tokens_kernel, dim3(blocks_for((long)B * S)), dim3(256), 0, s, x, y, B, S,
                     V, seed);
  return hipGetLastError();
}

hipError_t launch_synth_images(float* img, long n, int32_t* y, int B, int classes, uint32_t seed,
                               hipStream_t s) {
  hipLaunchKernelGGL(synth_images_kernel, dim3(blocks_for(n > B ? n : B)), dim3(256), 0, s, img, n, y,
                     B, classes, seed);
  return hipGetLastError();
}

hipError_t launch_count_valid(const int32_t* labels, int n, float* inv_n, hipStream_t s) {
  hipLaunchKernelGGL(count_valid_kernel, dim3(1), dim3(256), 0, s, labels, n, inv_n);
  return hipGetLastError();
}

AdamWConsts adamw_consts(double lr, double beta1, double beta2, double eps, double wd, long t) {
  AdamWConsts c;
  c.lr_wd = (float)(lr * wd);
  c.b1 = (float)beta1;
  c.omb1 = (float)(1.0 - beta1);
  c.b2 = (float)beta2;
  c.omb2 = (float)(1.0 - beta2);
  c.step = (float)(lr / (1.0 - pow(beta1, (double)t)));
  c.bc2s = (float)sqrt(1.0 - pow(beta2, (double)t));
  c.eps = (float)eps;
  return c;
}

hipError_t launch_adamw(float* p, const float* g, float* m, float* v, bf16* shadow, long n,
                        const AdamWConsts& c, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  bool al = ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(g) |
              reinterpret_cast<uintptr_t>(m) | reinterpret_cast<uintptr_t>(v)) & 15) == 0 &&
            (shadow == nullptr || (reinterpret_cast<uintptr_t>(shadow) & 7) == 0);
  long n4 = al ? n / 4 : 0;
  long work = n4 > 0 ? n4 : n;
  unsigned grid = (unsigned)std::min<long>(blocks_for(work), 256L * 64);
  hipLaunchKernelGGL(adamw_kernel, dim3(grid), dim3(256), 0, s, p, g, m, v, shadow, n4, n, c);
  return hipGetLastError();
}

// AdamW over a table of segments, one launch per step.  A workgroup finds its
// segment by binary search on first_block.  Flat segments: 8192 elements per
// workgroup, float4 groups (offsets are multiples of 64 elements) and a scalar
// tail.  Matrix segments: a 64 x 64 tile; thread (ty, tx) updates rows
// 4 ty .. 4 ty + 3, columns 4 tx .. 4 tx + 3, stages the bf16 values
// transposed in LDS, and the tile is written to shadow_t as 64 rows of 128
// contiguous bytes.
__global__ __launch_bounds__(256) void adamw_seg_kernel(float* __restrict__ p,
                                                        const float* __restrict__ g,
                                                        float* __restrict__ m,
                                                        float* __restrict__ v,
                                                        bf16* __restrict__ shadow,
                                                        bf16* __restrict__ shadow_t,
                                                        const AdamWSeg* __restrict__ segs, int nseg,
                                                        AdamWConsts c) {
  __shared__ __attribute__((aligned(16))) bf16 tt[64 * 72];  // [column][row], pitch 72
  const int b = blockIdx.x;
  int lo = 0, hi = nseg - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (segs[mid].first_block <= b) lo = mid;
    else hi = mid - 1;
  }
  const AdamWSeg sg = segs[lo];
  const int local = b - sg.first_block;
  const int t = threadIdx.x;
  if (sg.toff < 0) {
    const long n = sg.rows;
    const long base = sg.off + (long)local * kAdamWChunk;
    const long cnt = min((long)kAdamWChunk, n - (long)local * kAdamWChunk);
    const long c4 = cnt / 4;
    for (long i = t; i < c4; i += 256) {
      const long j = base + 4 * i;
      floatx4 pp = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p + j));
      const floatx4 gg = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(g + j));
      floatx4 mm = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(m + j));
      floatx4 vv = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(v + j));
      adamw_four(pp, gg, mm, vv, c);
      __builtin_nontemporal_store(pp, reinterpret_cast<floatx4*>(p + j));
      __builtin_nontemporal_store(mm, reinterpret_cast<floatx4*>(m + j));
      __builtin_nontemporal_store(vv, reinterpret_cast<floatx4*>(v + j));
      bf16x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = f2bf(pp[e]);
      __builtin_nontemporal_store(o, reinterpret_cast<bf16x4*>(shadow + j));
    }
    for (long i = 4 * c4 + t; i < cnt; i += 256) {
      const long j = base + i;
      float pp = p[j], mm = m[j], vv = v[j];
      adamw_one(pp, g[j], mm, vv, c);
      p[j] = pp;
      m[j] = mm;
      v[j] = vv;
      shadow[j] = f2bf(pp);
    }
    return;
  }
  const int tiles_n = (sg.cols + 63) / 64;
  const int r0 = (local / tiles_n) * 64, c0 = (local % tiles_n) * 64;
  const int ty = t >> 4, tx = t & 15;
  const int col = c0 + 4 * tx;
  bf16x4 o[4];  // o[i]: row 4 ty + i, columns 4 tx .. 4 tx + 3
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = r0 + 4 * ty + i;
    o[i] = bf16x4{f2bf(0.f), f2bf(0.f), f2bf(0.f), f2bf(0.f)};
    if (r < sg.rows && col < sg.cols) {
      const long j = sg.off + (long)r * sg.cols + col;
      floatx4 pp = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p + j));
      const floatx4 gg = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(g + j));
      floatx4 mm = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(m + j));
      floatx4 vv = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(v + j));
      adamw_four(pp, gg, mm, vv, c);
      __builtin_nontemporal_store(pp, reinterpret_cast<floatx4*>(p + j));
      __builtin_nontemporal_store(mm, reinterpret_cast<floatx4*>(m + j));
      __builtin_nontemporal_store(vv, reinterpret_cast<floatx4*>(v + j));
#pragma unroll
      for (int e = 0; e < 4; ++e) o[i][e] = f2bf(pp[e]);
      __builtin_nontemporal_store(o[i], reinterpret_cast<bf16x4*>(shadow + j));
    }
  }
  // column 4 tx + e of the tile gets rows 4 ty .. 4 ty + 3
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bf16x4 w = {o[0][e], o[1][e], o[2][e], o[3][e]};
    *reinterpret_cast<bf16x4*>(tt + (4 * tx + e) * 72 + 4 * ty) = w;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int idx = t + 256 * k;
    const int cc = idx >> 3, q = idx & 7;  // column of the tile, 8-row piece
    if (c0 + cc < sg.cols && r0 + 8 * q < sg.trows) {
      const bf16x8 w = *reinterpret_cast<const bf16x8*>(tt + cc * 72 + 8 * q);
      __builtin_nontemporal_store(
          w, reinterpret_cast<bf16x8*>(shadow_t + sg.toff + (long)(c0 + cc) * sg.trows + r0 + 8 * q));
    }
  }
}

int adamw_seg_blocks(const AdamWSeg& g) {
  if (g.toff < 0) return (int)((g.rows + kAdamWChunk - 1) / kAdamWChunk);
  return ((g.trows + 63) / 64) * ((g.cols + 63) / 64);
}

hipError_t launch_adamw_segments(float* p, const float* g, float* m, float* v, bf16* shadow,
                                 bf16* shadow_t, const AdamWSeg* segs, int nseg,
                                 int total_blocks, const AdamWConsts& c, hipStream_t s) {
  if (nseg <= 0 || total_blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(adamw_seg_kernel, dim3((unsigned)total_blocks), dim3(256), 0, s, p, g, m, v,
                     shadow, shadow_t, segs, nseg, c);
  return hipGetLastError();
}

hipError_t launch_init_normal(float* p, bf16* shadow, long n, uint64_t seed, uint32_t stream_id,
                              float std, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  long pairs = (n + 1) / 2;
  hipLaunchKernelGGL(init_normal_kernel, dim3(blocks_for(pairs)), dim3(256), 0, s, p, shadow, n,
                     (uint32_t)seed, (uint32_t)(seed >> 32), stream_id, std);
  return hipGetLastError();
}

hipError_t launch_fill(float* p, bf16* shadow, long n, float value, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, dim3(blocks_for(n)), dim3(256), 0, s, p, shadow, n, value);
  return hipGetLastError();
}

hipError_t launch_zero(void* p, long bytes, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  if (bytes % 4) return hipErrorInvalidValue;
  long n = bytes / 4;
  unsigned grid = (unsigned)std::min<long>(blocks_for(n), 256L * 64);
  hipLaunchKernelGGL(zero_kernel, dim3(grid), dim3(256), 0, s, (uint32_t*)p, n);
  return hipGetLastError();
}
