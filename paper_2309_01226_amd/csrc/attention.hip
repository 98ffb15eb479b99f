// Flash-style attention forward and backward on gfx950 MFMA (bf16 operands,
// fp32 accumulation), causal (decoders) or bidirectional (ViT).
//
// Per head: P = softmax(scale * q k^T + mask), o = P v, saved per query:
// lse = log sum_j exp(scale * q.k_j).  The S x S matrix never touches HBM:
// key/value (or query/gradient) blocks are staged through LDS and the softmax
// runs online.
//
// Layout trick.  With v_mfma_f32_32x32x16_bf16 a lane of the 32 x 32
// accumulator owns one column and 16 rows.  The forward and the dQ kernel
// compute the transposed score tile S^T = K Q^T, so each lane owns one query
// (column) and its running max / sum / rescale are per-lane scalars; its 16
// probabilities are then already an MFMA operand for O^T += V^T P^T, provided
// V^T is read from LDS with the same key permutation.  The dK/dV kernel owns
// keys instead and computes S = Q K^T the other way round.
//
// Backward without atomics: one kernel accumulates dK and dV per key block
// over all query blocks, a second accumulates dQ per query block over all key
// blocks (the score and dP tiles are recomputed in both).
//
// This file serves head dims 16, 32 (first-generation kernels, whose output
// may be split into head-dim slices) and 128 (the pipelined *_fast kernels);
// head dims 64 and 80 run in attn_small.hip and 256 in attn256.hip.
#include "common.h"
#include "kernels.h"

namespace {

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr int NT = 256;  // 4 waves
constexpr int WROWS = 32;  // rows (queries or keys) owned by each wave
constexpr int WG_ROWS = 4 * WROWS;

__device__ __forceinline__ floatx16 zero16() {
  floatx16 z;
#pragma unroll
  for (int r = 0; r < 16; ++r) z[r] = 0.f;
  return z;
}

// Copy rows [row0, row0 + ROWS) x cols [0, DH) of a bf16 matrix (row r at
// src + r * ld) into LDS dst[r][c] (pitch P), zero for rows >= nvalid.
template <int ROWS, int DH, int P>
__device__ __forceinline__ void stage_rows(const bf16* __restrict__ src, long ld, int row0,
                                           int nvalid, bf16* dst) {
  constexpr int VPR = DH / 8;
  constexpr int NV = ROWS * VPR;
  for (int v = threadIdx.x; v < NV; v += NT) {
    int r = v / VPR, c = (v % VPR) * 8;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (row0 + r < nvalid) x = *reinterpret_cast<const u32x4*>(src + (long)(row0 + r) * ld + c);
    *reinterpret_cast<u32x4*>(dst + r * P + c) = x;
  }
}

// Transposed copy: dst[c][r] = src[row0 + r][col0 + c] for r < ROWS, c < COLS
// (zero for rows >= nvalid or columns >= DH), via 8 x 8 register transposes.
template <int ROWS, int COLS, int DH, int P>
__device__ __forceinline__ void stage_rows_T(const bf16* __restrict__ src, long ld, int row0,
                                             int nvalid, int col0, bf16* dst) {
  constexpr int RB = ROWS / 8, CB = COLS / 8, NB = RB * CB;
  for (int b = threadIdx.x; b < NB; b += NT) {
    int rb = b % RB, cb = b / RB;
    int c = col0 + cb * 8;
    u32x4 x[8];
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      int r = row0 + rb * 8 + kk;
      u32x4 z = {0u, 0u, 0u, 0u};
      x[kk] = (r < nvalid && c < DH) ? *reinterpret_cast<const u32x4*>(src + (long)r * ld + c) : z;
    }
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      u32x4 lo, hi;
#pragma unroll
      for (int w2 = 0; w2 < 4; ++w2) {
        uint32_t a = x[2 * w2][w], e = x[2 * w2 + 1][w];
        lo[w2] = __builtin_amdgcn_perm(e, a, 0x05040100u);
        hi[w2] = __builtin_amdgcn_perm(e, a, 0x07060302u);
      }
      *reinterpret_cast<u32x4*>(dst + (cb * 8 + 2 * w) * P + rb * 8) = lo;
      *reinterpret_cast<u32x4*>(dst + (cb * 8 + 2 * w + 1) * P + rb * 8) = hi;
    }
  }
}

// MFMA operand of 8 consecutive bf16 from LDS.
__device__ __forceinline__ bf16x8 lds8(const bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
// Operand in the accumulator's row permutation: for lane group g the 16-wide
// chunk starting at `base` contributes elements base + 4g + {0..3} and
// base + 8 + 4g + {0..3}.
__device__ __forceinline__ bf16x8 lds8_perm(const bf16* row, int base, int g) {
  bf16x4 a = *reinterpret_cast<const bf16x4*>(row + base + 4 * g);
  bf16x4 b = *reinterpret_cast<const bf16x4*>(row + base + 8 + 4 * g);
  bf16x8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}
// Eight accumulator values r = 8h .. 8h+7 as a bf16 operand.
__device__ __forceinline__ bf16x8 acc_to_bf16(const floatx16& x, int h) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = f2bf(x[8 * h + e]);
  return r;
}
// Row (within a 32 x 32 tile) held by accumulator register r of lane group g.
__device__ __forceinline__ int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// Load a 32-row x DH operand slice for this lane (row = lane % 32) from global.
template <int DH>
__device__ __forceinline__ void load_row_operand(const bf16* __restrict__ base, long ld, int row,
                                                 int nvalid, int g, bf16x8* out) {
#pragma unroll
  for (int c = 0; c < DH / 16; ++c) {
    u32x4 z = {0u, 0u, 0u, 0u};
    u32x4 x = (row < nvalid) ? *reinterpret_cast<const u32x4*>(base + (long)row * ld + c * 16 + 8 * g) : z;
    out[c] = *reinterpret_cast<bf16x8*>(&x);
  }
}

constexpr int round32(int x) { return (x + 31) / 32 * 32; }

// Heavy (late) causal blocks first.
__device__ __forceinline__ int block_index(int nblk, int causal) {
  return causal ? (nblk - 1 - (int)blockIdx.x) : (int)blockIdx.x;
}

// ================================================================ forward
template <int DH, int BKV>
__global__ __launch_bounds__(NT) void attn_fwd_kernel(AttnArgs a) {
  constexpr int DHP = round32(DH);
  constexpr int PK = DH + 8;    // K tile pitch
  constexpr int PV = BKV + 8;   // V^T tile pitch
  __shared__ __attribute__((aligned(16))) bf16 Ks[BKV * PK];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DHP * PV];

  const int S = a.S;
  const int nqb = (S + WG_ROWS - 1) / WG_ROWS;
  const int qb = block_index(nqb, a.causal);
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5;
  const int q0 = qb * WG_ROWS;
  const int q = q0 + wave * WROWS + (lane & 31);

  const bf16* Qb = a.q + (long)b * S * a.ldq + (long)h * DH;
  const bf16* Kb = a.k + (long)b * S * a.ldk + (long)h * DH;
  const bf16* Vb = a.v + (long)b * S * a.ldv + (long)h * DH;

  bf16x8 qf[DH / 16];
  load_row_operand<DH>(Qb, a.ldq, q, S, g, qf);

  floatx16 o[DHP / 32];
#pragma unroll
  for (int t = 0; t < DHP / 32; ++t) o[t] = zero16();
  float m = -INFINITY, l = 0.f;
  const float sc = a.scale * LOG2E;
  const int wave_qmax = q0 + wave * WROWS + WROWS - 1;

  const int kv_end = a.causal ? min(S, q0 + WG_ROWS) : S;
  for (int kv0 = 0; kv0 < kv_end; kv0 += BKV) {
    __syncthreads();
    stage_rows<BKV, DH, PK>(Kb, a.ldk, kv0, S, Ks);
    stage_rows_T<BKV, DHP, DH, PV>(Vb, a.ldv, kv0, S, 0, Vt);
    __syncthreads();
    if (a.causal && kv0 > wave_qmax) continue;

    floatx16 s[BKV / 32];
#pragma unroll
    for (int t = 0; t < BKV / 32; ++t) {
      s[t] = zero16();
#pragma unroll
      for (int c = 0; c < DH / 16; ++c)
        s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            lds8(Ks + (t * 32 + (lane & 31)) * PK + c * 16 + 8 * g), qf[c], s[t], 0, 0, 0);
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < BKV / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int key = kv0 + t * 32 + acc_row(r, g);
        float x = s[t][r] * sc;
        if (key >= S || (a.causal && key > q)) x = -INFINITY;
        s[t][r] = x;
        mloc = fmaxf(mloc, x);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float mnew = fmaxf(m, mloc);
    const float alpha = (mnew == -INFINITY) ? 1.f : exp2f(m - mnew);
    float lsum = 0.f;
#pragma unroll
    for (int t = 0; t < BKV / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = (mnew == -INFINITY) ? 0.f : exp2f(s[t][r] - mnew);
        s[t][r] = p;
        lsum += p;
      }
    lsum += __shfl_xor(lsum, 32, 64);
    l = l * alpha + lsum;
    m = mnew;
#pragma unroll
    for (int t = 0; t < DHP / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
#pragma unroll
    for (int t = 0; t < BKV / 32; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8 pb = acc_to_bf16(s[t], hh);
#pragma unroll
        for (int ot = 0; ot < DHP / 32; ++ot)
          o[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              lds8_perm(Vt + (ot * 32 + (lane & 31)) * PV, t * 32 + hh * 16, g), pb, o[ot], 0, 0, 0);
      }
  }
  if (q < S) {
    const float inv = (l > 0.f) ? 1.f / l : 0.f;
    bf16* Ob = a.o + ((long)b * S + q) * a.ldo + (long)h * DH;
#pragma unroll
    for (int ot = 0; ot < DHP / 32; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int j = ot * 32 + acc_row(r, g);
        if (j < DH) Ob[j] = f2bf(o[ot][r] * inv);
      }
    if (g == 0) a.lse[((long)b * a.H + h) * S + q] = (m + log2f(l)) * LN2;
  }
}

// ================================================================ forward, pipelined
// For head dims 64, 128 and 256: 64-key blocks in two LDS stages.  K rows go
// HBM -> LDS with buffer_load ... lds into a swizzled layout (16-byte chunk c
// of row r at position c ^ swz(r), conflict-free for the 16 lanes a 128-bit
// read serves); V is loaded one block ahead into registers and stored
// transposed (V^T, keys contiguous).  The copies of block j + 1 are in flight
// while block j is computed.

#define LDS_PTR(p) ((void __attribute__((address_space(3)))*)(p))
constexpr uint32_t OOB = 0x80000000u;
constexpr int FBKV = 64;  // keys per block

template <int ROWS, int DH>
struct RowTile {  // ROWS rows of DH bf16 in LDS, swizzled 16-byte chunks, filled by DMA
  static constexpr int CPR = DH / 8;
  __device__ __forceinline__ static int swz(int row) { return CPR >= 16 ? (row & 15) : ((row >> 1) & 7); }
  __device__ __forceinline__ static int off(int row, int chunk) {
    return row * DH + ((chunk ^ swz(row)) << 3);
  }
  static constexpr int NI = ROWS * CPR / 64 / 4;  // DMA instructions per wave
  static_assert(ROWS * CPR % 256 == 0, "tile must be a whole number of 1 KB wave copies");
  __device__ __forceinline__ static void copy(__amdgpu_buffer_rsrc_t rs, long ld, int nvalid,
                                              bf16* __restrict__ S, int wave) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = (i * 4 + wave) * 64 + lane;
      const int row = q / CPR, pos = q % CPR;
      const int c = pos ^ swz(row);
      const uint32_t o = row < nvalid ? (uint32_t)(((long)row * ld + c * 8) * 2) : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, LDS_PTR(S + (i * 4 + wave) * 512), 16, o, 0, 0, 0);
    }
  }
};

// Transposed tile: DH rows (head dims) x ROWS columns (keys or queries) in
// LDS, pitch ROWS + 4 (for 32 columns: 72-byte rows, so the 8-byte operand
// reads of 32 consecutive rows hit distinct banks).  Built from ROWS x DH
// row-major data in 4 x 8 pieces: a thread loads 4 rows x 8 columns (four
// 16-byte loads) and writes 8 transposed rows of 4 values.
template <int ROWS, int DH>
struct TransTile {
  static constexpr int PITCH = ROWS + 4;
  static constexpr int SIZE = DH * PITCH;
  static constexpr int NP = (ROWS / 4) * (DH / 8);  // pieces
  __device__ __forceinline__ static void load(__amdgpu_buffer_rsrc_t rs, long ld, int nvalid, int p,
                                              u32x4* regs) {
    const int rq = p / (DH / 8), db = p % (DH / 8);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int r = rq * 4 + kk;
      const uint32_t o = r < nvalid ? (uint32_t)(((long)r * ld + db * 8) * 2) : OOB;
      regs[kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, o, 0, 0));
    }
  }
  __device__ __forceinline__ static void store(bf16* __restrict__ S, int p, const u32x4* x) {
    const int rq = p / (DH / 8), db = p % (DH / 8);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      u32x2 lo, hi;
#pragma unroll
      for (int w2 = 0; w2 < 2; ++w2) {
        const uint32_t a0 = x[2 * w2][w], a1 = x[2 * w2 + 1][w];
        lo[w2] = __builtin_amdgcn_perm(a1, a0, 0x05040100u);
        hi[w2] = __builtin_amdgcn_perm(a1, a0, 0x07060302u);
      }
      *reinterpret_cast<u32x2*>(S + (db * 8 + 2 * w) * PITCH + rq * 4) = lo;
      *reinterpret_cast<u32x2*>(S + (db * 8 + 2 * w + 1) * PITCH + rq * 4) = hi;
    }
  }
  // MFMA operand of row `row` in the accumulator permutation (lds8_perm)
  __device__ __forceinline__ static bf16x8 read_perm(const bf16* __restrict__ S, int row, int base, int g) {
    return lds8_perm(S + row * PITCH, base, g);
  }
};

template <int DH>
struct KTile {  // K block in LDS: FBKV rows of DH bf16
  static constexpr int CPR = DH / 8;  // 16-byte chunks per row
  __device__ __forceinline__ static int swz(int row) { return CPR >= 16 ? (row & 15) : ((row >> 1) & 7); }
  __device__ __forceinline__ static int off(int row, int chunk) {
    return row * DH + ((chunk ^ swz(row)) << 3);
  }
  // DMA of rows [0, FBKV) of the block starting at key kv0 (rows >= nvalid read 0)
  __device__ __forceinline__ static void copy(__amdgpu_buffer_rsrc_t rs, long ld, int nvalid,
                                              bf16* __restrict__ S, int wave) {
    const int lane = threadIdx.x & 63;
    constexpr int NI = FBKV * CPR / 64 / 4;  // instructions per wave
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = (i * 4 + wave) * 64 + lane;
      const int row = q / CPR, pos = q % CPR;
      const int c = pos ^ swz(row);
      const uint32_t o = row < nvalid ? (uint32_t)(((long)row * ld + c * 8) * 2) : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, LDS_PTR(S + (i * 4 + wave) * 512), 16, o, 0, 0, 0);
    }
  }
};

template <int DH>
struct VtTile {  // V^T block in LDS: DH rows (head dims) of FBKV keys
  static constexpr int KB = FBKV / 8;       // key blocks of 8
  static constexpr int NB = KB * (DH / 8);  // 8 x 8 blocks
  static constexpr int NPT = (NB + NT - 1) / NT;
  __device__ __forceinline__ static int swz(int row) { return (row >> 1) & 7; }
  __device__ __forceinline__ static int off(int row, int chunk) {
    return row * FBKV + ((chunk ^ swz(row)) << 3);
  }
  __device__ __forceinline__ static int loads(int wave) {
    int n = 0;
#pragma unroll
    for (int j = 0; j < NPT; ++j)
      if (wave * 64 + j * NT < NB) n += 8;
    return n;
  }
  // 8 keys x 8 dims per block; block b = key block b / (DH/8), dim block b % (DH/8)
  __device__ __forceinline__ static void load(__amdgpu_buffer_rsrc_t rs, long ld, int nvalid,
                                              u32x4* regs) {
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      const int b = threadIdx.x + j * NT;
      if (b >= NB) break;
      const int kb = b / (DH / 8), db = b % (DH / 8);
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const int key = kb * 8 + kk;
        const uint32_t o = key < nvalid ? (uint32_t)(((long)key * ld + db * 8) * 2) : OOB;
        regs[8 * j + kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, o, 0, 0));
      }
    }
  }
  __device__ __forceinline__ static void store(bf16* __restrict__ S, const u32x4* regs) {
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      const int b = threadIdx.x + j * NT;
      if (b >= NB) break;
      const int kb = b / (DH / 8), db = b % (DH / 8);
      const u32x4* x = regs + 8 * j;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        u32x4 lo, hi;
#pragma unroll
        for (int w2 = 0; w2 < 4; ++w2) {
          uint32_t a0 = x[2 * w2][w], a1 = x[2 * w2 + 1][w];
          lo[w2] = __builtin_amdgcn_perm(a1, a0, 0x05040100u);
          hi[w2] = __builtin_amdgcn_perm(a1, a0, 0x07060302u);
        }
        *reinterpret_cast<u32x4*>(S + off(db * 8 + 2 * w, kb)) = lo;
        *reinterpret_cast<u32x4*>(S + off(db * 8 + 2 * w + 1, kb)) = hi;
      }
    }
  }
};

// Wait until at most n' vector loads of this wave are in flight (and all LDS
// operations are done), n' the largest of {0, 2, 4, 6, 8, 10, 12, 16} not
// above `n` (wave-uniform).
__device__ __forceinline__ void wait_loads_upto(int n) {
  if (n >= 16) wait_vm_lgkm0<16>();
  else if (n >= 12) wait_vm_lgkm0<12>();
  else if (n >= 10) wait_vm_lgkm0<10>();
  else if (n >= 8) wait_vm_lgkm0<8>();
  else if (n >= 6) wait_vm_lgkm0<6>();
  else if (n >= 4) wait_vm_lgkm0<4>();
  else if (n >= 2) wait_vm_lgkm0<2>();
  else wait_vm_lgkm0<0>();
}

// One forward block: S^T = K Q^T, online softmax, O^T += V^T P^T.  `kt` and
// `vt` are the resident stage; `nxt` receives the copies of the next block.
template <int DH>
__device__ __forceinline__ void fwd_block(const bf16* __restrict__ kt, const bf16* __restrict__ vt,
                                          bf16* __restrict__ nxt, bool copy_next,
                                          __amdgpu_buffer_rsrc_t rsK, long ldk, int nvalid_next,
                                          const bf16x8 (&qf)[DH / 16], floatx16 (&o)[DH / 32],
                                          float& m, float& l, int kv0, int q, int S, int causal,
                                          float sc, bool active, int wave, int lane) {
  if (copy_next) KTile<DH>::copy(rsK, ldk, nvalid_next, nxt, wave);
  if (!active) return;
  const int g = lane >> 5;
  floatx16 s[FBKV / 32];
#pragma unroll
  for (int t = 0; t < FBKV / 32; ++t) {
    s[t] = zero16();
    const int row = t * 32 + (lane & 31);
#pragma unroll
    for (int c = 0; c < DH / 16; ++c)
      s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          *reinterpret_cast<const bf16x8*>(kt + KTile<DH>::off(row, 2 * c + g)), qf[c], s[t], 0, 0, 0);
  }
  float mloc = -INFINITY;
#pragma unroll
  for (int t = 0; t < FBKV / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = kv0 + t * 32 + acc_row(r, g);
      float x = s[t][r] * sc;
      if (key >= S || (causal && key > q)) x = -INFINITY;
      s[t][r] = x;
      mloc = fmaxf(mloc, x);
    }
  mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
  const float mnew = fmaxf(m, mloc);
  const float alpha = (mnew == -INFINITY) ? 1.f : exp2f(m - mnew);
  float lsum = 0.f;
#pragma unroll
  for (int t = 0; t < FBKV / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float pr = (mnew == -INFINITY) ? 0.f : exp2f(s[t][r] - mnew);
      s[t][r] = pr;
      lsum += pr;
    }
  lsum += __shfl_xor(lsum, 32, 64);
  l = l * alpha + lsum;
  m = mnew;
#pragma unroll
  for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[ot][r] *= alpha;
#pragma unroll
  for (int t = 0; t < FBKV / 32; ++t)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const bf16x8 pb = acc_to_bf16(s[t], hh);
      const int c0 = (t * 32 + hh * 16) / 8;  // first 8-key chunk of this 16-key step
#pragma unroll
      for (int ot = 0; ot < DH / 32; ++ot) {
        const int row = ot * 32 + (lane & 31);
        const bf16x4 a0 = *reinterpret_cast<const bf16x4*>(vt + VtTile<DH>::off(row, c0) + 4 * g);
        const bf16x4 a1 = *reinterpret_cast<const bf16x4*>(vt + VtTile<DH>::off(row, c0 + 1) + 4 * g);
        bf16x8 av;
        av[0] = a0[0]; av[1] = a0[1]; av[2] = a0[2]; av[3] = a0[3];
        av[4] = a1[0]; av[5] = a1[1]; av[6] = a1[2]; av[7] = a1[3];
        o[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb, o[ot], 0, 0, 0);
      }
    }
}

template <int DH>
__global__ __launch_bounds__(NT) void attn_fwd_fast(AttnArgs a) {
  constexpr int KSZ = FBKV * DH, VSZ = DH * FBKV, STG = KSZ + VSZ;
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * STG];
  const int S = a.S;
  const int nqb = (S + WG_ROWS - 1) / WG_ROWS;
  const int qb = block_index(nqb, a.causal);
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int q0 = qb * WG_ROWS;
  const int q = q0 + wave * WROWS + (lane & 31);
  const bf16* Qb = a.q + (long)b * S * a.ldq + (long)h * DH;
  const bf16* Kb = a.k + (long)b * S * a.ldk + (long)h * DH;
  const bf16* Vb = a.v + (long)b * S * a.ldv + (long)h * DH;

  bf16x8 qf[DH / 16];
  load_row_operand<DH>(Qb, a.ldq, q, S, g, qf);
  floatx16 o[DH / 32];
#pragma unroll
  for (int t = 0; t < DH / 32; ++t) o[t] = zero16();
  float m = -INFINITY, l = 0.f;
  const float sc = a.scale * LOG2E;
  const int wave_qmax = q0 + wave * WROWS + WROWS - 1;
  const int kv_end = a.causal ? min(S, q0 + WG_ROWS) : S;
  const int nblk = (kv_end + FBKV - 1) / FBKV;
  const int nvl = VtTile<DH>::loads(wave);
  auto rsrc = [&](const bf16* base, int kv0, long ld) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)(base + (long)kv0 * ld), (short)0, 0x7FFFFFFF,
                                             0x00020000);
  };

  // prologue: block 0 resident in stage 0, V of block 1 requested
  u32x4 vr[8 * VtTile<DH>::NPT];
  KTile<DH>::copy(rsrc(Kb, 0, a.ldk), a.ldk, S, smem, wave);
  VtTile<DH>::load(rsrc(Vb, 0, a.ldv), a.ldv, S, vr);
  VtTile<DH>::store(smem + KSZ, vr);
  if (nblk > 1) VtTile<DH>::load(rsrc(Vb, FBKV, a.ldv), a.ldv, S - FBKV, vr);
  wait_loads_upto(nblk > 1 ? nvl : 0);
  cta_barrier();

  for (int j = 0; j < nblk; ++j) {
    const int kv0 = j * FBKV;
    bf16* cur = smem + (j & 1) * STG;
    bf16* nxt = smem + ((j + 1) & 1) * STG;
    const bool next = j + 1 < nblk;
    fwd_block<DH>(cur, cur + KSZ, nxt, next, rsrc(Kb, kv0 + FBKV, a.ldk), a.ldk, S - kv0 - FBKV,
                  qf, o, m, l, kv0, q, S, a.causal, sc, !(a.causal && kv0 > wave_qmax), wave, lane);
    if (next) {
      VtTile<DH>::store(nxt + KSZ, vr);
      if (j + 2 < nblk) VtTile<DH>::load(rsrc(Vb, kv0 + 2 * FBKV, a.ldv), a.ldv, S - kv0 - 2 * FBKV, vr);
      wait_loads_upto(j + 2 < nblk ? nvl : 0);
      cta_barrier();
    }
  }
  if (q < S) {
    const float inv = (l > 0.f) ? 1.f / l : 0.f;
    bf16* Ob = a.o + ((long)b * S + q) * a.ldo + (long)h * DH;
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) Ob[ot * 32 + acc_row(r, g)] = f2bf(o[ot][r] * inv);
    if (g == 0) a.lse[((long)b * a.H + h) * S + q] = (m + log2f(l)) * LN2;
  }
}

// ================================================================ backward
// delta[b, h, s] = sum_j dO[s, j] * O[s, j]; one wave per (b, s, h).
__global__ __launch_bounds__(256) void attn_delta_kernel(AttnBwdArgs a) {
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const long total = (long)a.f.B * a.f.S * a.f.H;
  if (row >= total) return;
  const int h = row % a.f.H;
  const long bs = row / a.f.H;
  const int dh = a.f.dh;
  const bf16* o = a.f.o + bs * a.f.ldo + (long)h * dh;
  const bf16* d = a.dout + bs * a.lddo + (long)h * dh;
  float acc = 0.f;
  for (int j = lane; j < dh; j += 64) acc += bf2f(o[j]) * bf2f(d[j]);
  acc = wave_sum(acc);
  const int b = bs / a.f.S, s = bs % a.f.S;
  if (lane == 0) a.delta[((long)b * a.f.H + h) * a.f.S + s] = acc;
}

// dQ: workgroup = 128 queries of one (b, h); grid.z = output dh slice.
template <int DH, int DHS, int BKV>
__global__ __launch_bounds__(NT) void attn_bwd_dq_kernel(AttnBwdArgs a) {
  constexpr int PK = DH + 8;
  constexpr int PT = BKV + 8;
  __shared__ __attribute__((aligned(16))) bf16 Ks[BKV * PK];
  __shared__ __attribute__((aligned(16))) bf16 Vs[BKV * PK];
  __shared__ __attribute__((aligned(16))) bf16 Kt[DHS * PT];

  const int S = a.f.S;
  const int nqb = (S + WG_ROWS - 1) / WG_ROWS;
  const int qb = block_index(nqb, a.f.causal);
  const int bh = blockIdx.y, b = bh / a.f.H, h = bh % a.f.H;
  const int col0 = blockIdx.z * DHS;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5;
  const int q0 = qb * WG_ROWS;
  const int q = q0 + wave * WROWS + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;

  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;

  bf16x8 qf[DH / 16], df[DH / 16];
  load_row_operand<DH>(Qb, a.f.ldq, q, S, g, qf);
  load_row_operand<DH>(dOb, a.lddo, q, S, g, df);
  const float sc = a.f.scale * LOG2E;
  const float lse2 = (q < S) ? a.f.lse[hs + q] * LOG2E : 0.f;
  const float dlt = (q < S) ? a.delta[hs + q] : 0.f;

  floatx16 dq[DHS / 32];
#pragma unroll
  for (int t = 0; t < DHS / 32; ++t) dq[t] = zero16();
  const int wave_qmax = q0 + wave * WROWS + WROWS - 1;
  const int kv_end = a.f.causal ? min(S, q0 + WG_ROWS) : S;
  for (int kv0 = 0; kv0 < kv_end; kv0 += BKV) {
    __syncthreads();
    stage_rows<BKV, DH, PK>(Kb, a.f.ldk, kv0, S, Ks);
    stage_rows<BKV, DH, PK>(Vb, a.f.ldv, kv0, S, Vs);
    stage_rows_T<BKV, DHS, DH, PT>(Kb, a.f.ldk, kv0, S, col0, Kt);
    __syncthreads();
    if (a.f.causal && kv0 > wave_qmax) continue;
#pragma unroll
    for (int t = 0; t < BKV / 32; ++t) {
      floatx16 s = zero16(), dp = zero16();
#pragma unroll
      for (int c = 0; c < DH / 16; ++c) {
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            lds8(Ks + (t * 32 + (lane & 31)) * PK + c * 16 + 8 * g), qf[c], s, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            lds8(Vs + (t * 32 + (lane & 31)) * PK + c * 16 + 8 * g), df[c], dp, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int key = kv0 + t * 32 + acc_row(r, g);
        bool ok = key < S && q < S && !(a.f.causal && key > q);
        float p = ok ? exp2f(s[r] * sc - lse2) : 0.f;
        s[r] = p * (dp[r] - dlt);
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8 db = acc_to_bf16(s, hh);
#pragma unroll
        for (int ot = 0; ot < DHS / 32; ++ot)
          dq[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              lds8_perm(Kt + (ot * 32 + (lane & 31)) * PT, t * 32 + hh * 16, g), db, dq[ot], 0, 0, 0);
      }
    }
  }
  if (q < S) {
    bf16* out = a.dq + ((long)b * S + q) * a.lddq + (long)h * DH;
#pragma unroll
    for (int ot = 0; ot < DHS / 32; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int j = col0 + ot * 32 + acc_row(r, g);
        if (j < DH && j < col0 + DHS) out[j] = f2bf(dq[ot][r] * a.f.scale);
      }
  }
}

// dK, dV: workgroup = 128 keys of one (b, h); grid.z = output dh slice.
template <int DH, int DHS, int BQ>
__global__ __launch_bounds__(NT) void attn_bwd_dkdv_kernel(AttnBwdArgs a) {
  constexpr int PK = DH + 8;
  constexpr int PT = BQ + 8;
  __shared__ __attribute__((aligned(16))) bf16 Qs[BQ * PK];
  __shared__ __attribute__((aligned(16))) bf16 dOs[BQ * PK];
  __shared__ __attribute__((aligned(16))) bf16 Qt[DHS * PT];
  __shared__ __attribute__((aligned(16))) bf16 dOt[DHS * PT];
  __shared__ float lse_s[BQ], dlt_s[BQ];

  const int S = a.f.S;
  const int nkb = (S + WG_ROWS - 1) / WG_ROWS;
  // causal: early key blocks see the most queries; schedule them first
  const int kb = (int)blockIdx.x;
  (void)nkb;
  const int bh = blockIdx.y, b = bh / a.f.H, h = bh % a.f.H;
  const int col0 = blockIdx.z * DHS;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5;
  const int k0 = kb * WG_ROWS;
  const int key = k0 + wave * WROWS + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;

  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;

  bf16x8 kf[DH / 16], vf[DH / 16];
  load_row_operand<DH>(Kb, a.f.ldk, key, S, g, kf);
  load_row_operand<DH>(Vb, a.f.ldv, key, S, g, vf);
  const float sc = a.f.scale * LOG2E;

  floatx16 dk[DHS / 32], dv[DHS / 32];
#pragma unroll
  for (int t = 0; t < DHS / 32; ++t) {
    dk[t] = zero16();
    dv[t] = zero16();
  }
  const int wave_kmin = k0 + wave * WROWS;
  const int q_start = a.f.causal ? (k0 / BQ) * BQ : 0;
  for (int qs0 = q_start; qs0 < S; qs0 += BQ) {
    __syncthreads();
    stage_rows<BQ, DH, PK>(Qb, a.f.ldq, qs0, S, Qs);
    stage_rows<BQ, DH, PK>(dOb, a.lddo, qs0, S, dOs);
    stage_rows_T<BQ, DHS, DH, PT>(Qb, a.f.ldq, qs0, S, col0, Qt);
    stage_rows_T<BQ, DHS, DH, PT>(dOb, a.lddo, qs0, S, col0, dOt);
    for (int i = threadIdx.x; i < BQ; i += NT) {
      int qq = qs0 + i;
      lse_s[i] = (qq < S) ? a.f.lse[hs + qq] * LOG2E : 0.f;
      dlt_s[i] = (qq < S) ? a.delta[hs + qq] : 0.f;
    }
    __syncthreads();
    if (a.f.causal && qs0 + BQ - 1 < wave_kmin) continue;
#pragma unroll
    for (int t = 0; t < BQ / 32; ++t) {
      floatx16 s = zero16(), dp = zero16();
#pragma unroll
      for (int c = 0; c < DH / 16; ++c) {
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            lds8(Qs + (t * 32 + (lane & 31)) * PK + c * 16 + 8 * g), kf[c], s, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            lds8(dOs + (t * 32 + (lane & 31)) * PK + c * 16 + 8 * g), vf[c], dp, 0, 0, 0);
      }
      // s, dp: rows = queries (acc_row), column = this lane's key
      floatx16 p;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int qi = t * 32 + acc_row(r, g);
        int qq = qs0 + qi;
        bool ok = qq < S && key < S && !(a.f.causal && key > qq);
        float pr = ok ? exp2f(s[r] * sc - lse_s[qi]) : 0.f;
        p[r] = pr;
        s[r] = pr * (dp[r] - dlt_s[qi]);
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8 pb = acc_to_bf16(p, hh);
        bf16x8 db = acc_to_bf16(s, hh);
#pragma unroll
        for (int ot = 0; ot < DHS / 32; ++ot) {
          dv[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              lds8_perm(dOt + (ot * 32 + (lane & 31)) * PT, t * 32 + hh * 16, g), pb, dv[ot], 0, 0, 0);
          dk[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              lds8_perm(Qt + (ot * 32 + (lane & 31)) * PT, t * 32 + hh * 16, g), db, dk[ot], 0, 0, 0);
        }
      }
    }
  }
  if (key < S) {
    bf16* ok_ = a.dk + ((long)b * S + key) * a.lddk + (long)h * DH;
    bf16* ov = a.dv + ((long)b * S + key) * a.lddv + (long)h * DH;
#pragma unroll
    for (int ot = 0; ot < DHS / 32; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int j = col0 + ot * 32 + acc_row(r, g);
        if (j < DH && j < col0 + DHS) {
          ok_[j] = f2bf(dk[ot][r] * a.f.scale);
          ov[j] = f2bf(dv[ot][r]);
        }
      }
  }
}

// ================================================================ backward, pipelined
// Both kernels loop over 32-row blocks of the other operand in two LDS
// stages: the rows arrive by direct HBM-to-LDS copies issued at the start of
// the previous block, the transposed tiles through registers loaded two
// blocks ahead; one barrier per block.
constexpr int BQB = 32;  // query rows per block (dK/dV kernels)
constexpr int BKB = 32;  // key rows per block (dQ kernel)

// dK/dV stage: Q rows, dO rows, Q^T, dO^T, lse * log2(e) and delta of 32 queries.
template <int DH>
struct KVStage {
  using RT = RowTile<BQB, DH>;
  using TT = TransTile<BQB, DH>;
  static constexpr int RQ = BQB * DH;
  static constexpr int SIZE = 2 * RQ + 2 * TT::SIZE + 2 * 2 * BQB;  // in bf16 units
  __device__ __forceinline__ static const bf16* rows(const bf16* st, int which) { return st + which * RQ; }
  __device__ __forceinline__ static const bf16* trans(const bf16* st, int which) {
    return st + 2 * RQ + which * TT::SIZE;
  }
  __device__ __forceinline__ static const float* lse(const bf16* st) {
    return reinterpret_cast<const float*>(st + 2 * RQ + 2 * TT::SIZE);
  }
};

// Register-staged half of a stage: the transposed pieces a thread loads for
// block q0 (Q^T pieces first, then dO^T), plus lse and delta on 32 threads.
template <int DH, int NTH>
struct KVTrans {
  using S = KVStage<DH>;
  using TT = typename S::TT;
  static constexpr int PER = (2 * TT::NP + NTH - 1) / NTH;
  u32x4 r[4 * PER];
  float lse = 0.f, dlt = 0.f;
  __device__ __forceinline__ static int loads(int wave) {  // vector loads per wave and call
    int n = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (wave * 64 + j * NTH < 2 * TT::NP) n += 4;
    return wave == 0 ? n + 2 : n;
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rsQ, __amdgpu_buffer_rsrc_t rsO, long ldq,
                                       long ldo, int nvalid, const float* lse_g, const float* dlt_g) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int p = tid + j * NTH;
      if (p < TT::NP) TT::load(rsQ, ldq, nvalid, p, r + 4 * j);
      else if (p < 2 * TT::NP) TT::load(rsO, ldo, nvalid, p - TT::NP, r + 4 * j);
    }
    if (tid < BQB) {
      lse = tid < nvalid ? lse_g[tid] * LOG2E : 0.f;
      dlt = tid < nvalid ? dlt_g[tid] : 0.f;
    }
  }
  __device__ __forceinline__ void store(bf16* __restrict__ st) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int p = tid + j * NTH;
      if (p < TT::NP) TT::store(st + 2 * S::RQ, p, r + 4 * j);
      else if (p < 2 * TT::NP) TT::store(st + 2 * S::RQ + TT::SIZE, p - TT::NP, r + 4 * j);
    }
    if (tid < BQB) {
      float* f = reinterpret_cast<float*>(st + 2 * S::RQ + 2 * TT::SIZE);
      f[tid] = lse;
      f[BQB + tid] = dlt;
    }
  }
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const bf16* base, int r0, long ld) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)(base + (long)r0 * ld), (short)0, 0x7FFFFFFF, 0x00020000);
}

// One query block of the dK/dV kernel for a wave owning 32 keys (full head
// dim): S = Q K^T and dP = dO V^T, P = exp(S - lse), dS = P (dP - delta),
// dV^T += dO^T P, dK^T += Q^T dS.
template <int DH>
__device__ __forceinline__ void kv_block(const bf16* __restrict__ cur, bf16* __restrict__ nxt, bool copy_next,
                                         __amdgpu_buffer_rsrc_t rsQ, __amdgpu_buffer_rsrc_t rsO, long ldq,
                                         long ldo, int nvalid_next, const bf16x8 (&kf)[DH / 16],
                                         const bf16x8 (&vf)[DH / 16], floatx16 (&dk)[DH / 32],
                                         floatx16 (&dv)[DH / 32], int qs0, int key, int S, int causal,
                                         float sc, bool active, int wave, int lane) {
  using SG = KVStage<DH>;
  using TT = typename SG::TT;
  using RT = typename SG::RT;
  if (copy_next) {
    RT::copy(rsQ, ldq, nvalid_next, nxt, wave);
    RT::copy(rsO, ldo, nvalid_next, nxt + SG::RQ, wave);
  }
  if (!active) return;
  const int g = lane >> 5, row = lane & 31;
  const bf16* Qs = SG::rows(cur, 0);
  const bf16* dOs = SG::rows(cur, 1);
  const float* ls = SG::lse(cur);
  floatx16 sv = zero16(), dp = zero16();
#pragma unroll
  for (int c = 0; c < DH / 16; ++c) {
    sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(Qs + RT::off(row, 2 * c + g)),
                                                 kf[c], sv, 0, 0, 0);
    dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(dOs + RT::off(row, 2 * c + g)),
                                                 vf[c], dp, 0, 0, 0);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int qi = acc_row(r, g);
    const int qq = qs0 + qi;
    const bool ok = qq < S && key < S && !(causal && key > qq);
    const float pr = ok ? exp2f(sv[r] * sc - ls[qi]) : 0.f;
    sv[r] = pr;
    dp[r] = pr * (dp[r] - ls[BQB + qi]);
  }
  const bf16* QT = SG::trans(cur, 0);
  const bf16* dOT = SG::trans(cur, 1);
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const bf16x8 pb = acc_to_bf16(sv, hh);
    const bf16x8 db = acc_to_bf16(dp, hh);
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot) {
      const int tr = ot * 32 + row;
      dv[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(TT::read_perm(dOT, tr, hh * 16, g), pb, dv[ot], 0, 0, 0);
      dk[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(TT::read_perm(QT, tr, hh * 16, g), db, dk[ot], 0, 0, 0);
    }
  }
}

template <int DH>
__global__ __launch_bounds__(NT) void attn_bwd_dkdv_fast(AttnBwdArgs a) {
  using SG = KVStage<DH>;
  using RT = typename SG::RT;
  using TR = KVTrans<DH, NT>;
  constexpr int KPW = WG_ROWS;  // keys per workgroup
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * SG::SIZE];
  const int S = a.f.S;
  const int bh = blockIdx.y, b = bh / a.f.H, h = bh % a.f.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int grp = wave;
  const int k0 = blockIdx.x * KPW;
  const int kmin = k0 + grp * WROWS;
  const int key = kmin + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;
  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;
  const float* lse_g = a.f.lse + hs;
  const float* dlt_g = a.delta + hs;

  constexpr int NACC = 2;  // acc[0] = dK^T, acc[1] = dV^T
  bf16x8 rf[NACC][DH / 16];
  floatx16 acc[NACC][DH / 32];
  load_row_operand<DH>(Kb, a.f.ldk, key, S, g, rf[0]);
  load_row_operand<DH>(Vb, a.f.ldv, key, S, g, rf[1]);
#pragma unroll
  for (int i = 0; i < NACC; ++i)
#pragma unroll
    for (int t = 0; t < DH / 32; ++t) acc[i][t] = zero16();
  const float sc = a.f.scale * LOG2E;
  const int q_start = a.f.causal ? k0 : 0;
  const int nqb = (S - q_start + BQB - 1) / BQB;
  const int nld = TR::loads(wave);
  TR tr;

  // prologue: block 0 resident in stage 0, transposes of block 1 in registers
  RT::copy(rows_rsrc(Qb, q_start, a.f.ldq), a.f.ldq, S - q_start, smem, wave);
  RT::copy(rows_rsrc(dOb, q_start, a.lddo), a.lddo, S - q_start, smem + SG::RQ, wave);
  tr.load(rows_rsrc(Qb, q_start, a.f.ldq), rows_rsrc(dOb, q_start, a.lddo), a.f.ldq, a.lddo, S - q_start,
          lse_g + q_start, dlt_g + q_start);
  wait_vm_lgkm0<0>();
  tr.store(smem);
  if (nqb > 1)
    tr.load(rows_rsrc(Qb, q_start + BQB, a.f.ldq), rows_rsrc(dOb, q_start + BQB, a.lddo), a.f.ldq, a.lddo,
            S - q_start - BQB, lse_g + q_start + BQB, dlt_g + q_start + BQB);
  wait_loads_upto(nqb > 1 ? nld : 0);
  cta_barrier();

  for (int j = 0; j < nqb; ++j) {
    const int qs0 = q_start + j * BQB;
    bf16* cur = smem + (j & 1) * SG::SIZE;
    bf16* nxt = smem + ((j + 1) & 1) * SG::SIZE;
    const bool next = j + 1 < nqb;
    const bool active = !(a.f.causal && qs0 + BQB - 1 < kmin);
    const auto rq = rows_rsrc(Qb, qs0 + BQB, a.f.ldq);
    const auto ro = rows_rsrc(dOb, qs0 + BQB, a.lddo);
    kv_block<DH>(cur, nxt, next, rq, ro, a.f.ldq, a.lddo, S - qs0 - BQB, rf[0], rf[1], acc[0], acc[1], qs0,
                 key, S, a.f.causal, sc, active, wave, lane);
    if (next) {
      tr.store(nxt);
      if (j + 2 < nqb)
        tr.load(rows_rsrc(Qb, qs0 + 2 * BQB, a.f.ldq), rows_rsrc(dOb, qs0 + 2 * BQB, a.lddo), a.f.ldq, a.lddo,
                S - qs0 - 2 * BQB, lse_g + qs0 + 2 * BQB, dlt_g + qs0 + 2 * BQB);
      wait_loads_upto(j + 2 < nqb ? nld : 0);
      cta_barrier();
    }
  }
  if (key < S) {
    bf16* ok_ = a.dk + ((long)b * S + key) * a.lddk + (long)h * DH;
    bf16* ov = a.dv + ((long)b * S + key) * a.lddv + (long)h * DH;
#pragma unroll
    for (int i = 0; i < NACC; ++i) {
      const bool is_k = i == 0;
      bf16* o = is_k ? ok_ : ov;
      const float f = is_k ? a.f.scale : 1.f;
#pragma unroll
      for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[ot * 32 + acc_row(r, g)] = f2bf(acc[i][ot][r] * f);
    }
  }
}

// dQ stage: K rows, V rows, K^T of 32 keys.
template <int DH>
struct QStage {
  using RT = RowTile<BKB, DH>;
  using TT = TransTile<BKB, DH>;
  static constexpr int RK = BKB * DH;
  static constexpr int SIZE = 2 * RK + TT::SIZE;
};

template <int DH, int NTH>
struct QTrans {
  using TT = TransTile<BKB, DH>;
  static constexpr int PER = (TT::NP + NTH - 1) / NTH;
  u32x4 r[4 * PER];
  __device__ __forceinline__ static int loads(int wave) {
    int n = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (wave * 64 + j * NTH < TT::NP) n += 4;
    return n;
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rsK, long ldk, int nvalid) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int p = threadIdx.x + j * NTH;
      if (p < TT::NP) TT::load(rsK, ldk, nvalid, p, r + 4 * j);
    }
  }
  __device__ __forceinline__ void store(bf16* __restrict__ st) const {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int p = threadIdx.x + j * NTH;
      if (p < TT::NP) TT::store(st + 2 * QStage<DH>::RK, p, r + 4 * j);
    }
  }
};

// One key block of the dQ kernel: S^T = K Q^T, dP^T = V dO^T,
// dS^T = P^T (dP^T - delta), dQ^T += K^T dS^T.
template <int DH>
__device__ __forceinline__ void q_block(const bf16* __restrict__ cur, bf16* __restrict__ nxt, bool copy_next,
                                        __amdgpu_buffer_rsrc_t rsK, __amdgpu_buffer_rsrc_t rsV, long ldk,
                                        long ldv, int nvalid_next, const bf16x8 (&qf)[DH / 16],
                                        const bf16x8 (&df)[DH / 16], floatx16 (&dq)[DH / 32], int kv0, int q,
                                        int S, int causal, float sc, float lse2, float dlt, bool active,
                                        int wave, int lane) {
  using SG = QStage<DH>;
  using TT = typename SG::TT;
  using RT = typename SG::RT;
  if (copy_next) {
    RT::copy(rsK, ldk, nvalid_next, nxt, wave);
    RT::copy(rsV, ldv, nvalid_next, nxt + SG::RK, wave);
  }
  if (!active) return;
  const int g = lane >> 5, row = lane & 31;
  const bf16* Ks = cur;
  const bf16* Vs = cur + SG::RK;
  floatx16 sv = zero16(), dp = zero16();
#pragma unroll
  for (int c = 0; c < DH / 16; ++c) {
    sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(Ks + RT::off(row, 2 * c + g)),
                                                 qf[c], sv, 0, 0, 0);
    dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(Vs + RT::off(row, 2 * c + g)),
                                                 df[c], dp, 0, 0, 0);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int kk = kv0 + acc_row(r, g);
    const bool ok = kk < S && q < S && !(causal && kk > q);
    const float pr = ok ? exp2f(sv[r] * sc - lse2) : 0.f;
    sv[r] = pr * (dp[r] - dlt);
  }
  const bf16* KT = cur + 2 * SG::RK;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const bf16x8 db = acc_to_bf16(sv, hh);
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot)
      dq[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(TT::read_perm(KT, ot * 32 + row, hh * 16, g), db, dq[ot], 0,
                                                       0, 0);
  }
}

template <int DH>
__global__ __launch_bounds__(NT) void attn_bwd_dq_fast(AttnBwdArgs a) {
  using SG = QStage<DH>;
  using RT = typename SG::RT;
  using TR = QTrans<DH, NT>;
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * SG::SIZE];
  const int S = a.f.S;
  const int nqb = (S + WG_ROWS - 1) / WG_ROWS;
  const int qb = block_index(nqb, a.f.causal);
  const int bh = blockIdx.y, b = bh / a.f.H, h = bh % a.f.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int q0 = qb * WG_ROWS;
  const int q = q0 + wave * WROWS + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;
  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;

  bf16x8 qf[DH / 16], df[DH / 16];
  load_row_operand<DH>(Qb, a.f.ldq, q, S, g, qf);
  load_row_operand<DH>(dOb, a.lddo, q, S, g, df);
  const float sc = a.f.scale * LOG2E;
  const float lse2 = (q < S) ? a.f.lse[hs + q] * LOG2E : 0.f;
  const float dlt = (q < S) ? a.delta[hs + q] : 0.f;
  floatx16 dq[DH / 32];
#pragma unroll
  for (int t = 0; t < DH / 32; ++t) dq[t] = zero16();
  const int wave_qmax = q0 + wave * WROWS + WROWS - 1;
  const int kv_end = a.f.causal ? min(S, q0 + WG_ROWS) : S;
  const int nkb = (kv_end + BKB - 1) / BKB;
  const int nld = TR::loads(wave);
  TR tr;

  RT::copy(rows_rsrc(Kb, 0, a.f.ldk), a.f.ldk, S, smem, wave);
  RT::copy(rows_rsrc(Vb, 0, a.f.ldv), a.f.ldv, S, smem + SG::RK, wave);
  tr.load(rows_rsrc(Kb, 0, a.f.ldk), a.f.ldk, S);
  wait_vm_lgkm0<0>();
  tr.store(smem);
  if (nkb > 1) tr.load(rows_rsrc(Kb, BKB, a.f.ldk), a.f.ldk, S - BKB);
  wait_loads_upto(nkb > 1 ? nld : 0);
  cta_barrier();

  for (int j = 0; j < nkb; ++j) {
    const int kv0 = j * BKB;
    bf16* cur = smem + (j & 1) * SG::SIZE;
    bf16* nxt = smem + ((j + 1) & 1) * SG::SIZE;
    const bool next = j + 1 < nkb;
    q_block<DH>(cur, nxt, next, rows_rsrc(Kb, kv0 + BKB, a.f.ldk), rows_rsrc(Vb, kv0 + BKB, a.f.ldv), a.f.ldk,
                a.f.ldv, S - kv0 - BKB, qf, df, dq, kv0, q, S, a.f.causal, sc, lse2, dlt,
                !(a.f.causal && kv0 > wave_qmax), wave, lane);
    if (next) {
      tr.store(nxt);
      if (j + 2 < nkb) tr.load(rows_rsrc(Kb, kv0 + 2 * BKB, a.f.ldk), a.f.ldk, S - kv0 - 2 * BKB);
      wait_loads_upto(j + 2 < nkb ? nld : 0);
      cta_barrier();
    }
  }
  if (q < S) {
    bf16* out = a.dq + ((long)b * S + q) * a.lddq + (long)h * DH;
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) out[ot * 32 + acc_row(r, g)] = f2bf(dq[ot][r] * a.f.scale);
  }
}

// Tile shape of the first-generation kernels (head dims 16 and 32: one output
// slice of the whole head).
template <int DH>
struct AttnCfg {
  static constexpr int BKV = 64;
  static constexpr int DHS = round32(DH);
  static constexpr int NSLICE = 1;
  static constexpr int BQ = 64;
};

// Head dims 16 and 32: the first-generation kernels; 128: the pipelined
// ones.  64, 80 and 256 run only in their own files' kernels (attn_small.hip,
// attn256.hip), which the callers below pick first.
template <int DH>
hipError_t fwd_launch(const AttnArgs& a, hipStream_t s) {
  static_assert(DH == 16 || DH == 32 || DH == 128, "head dim served by attn_small / attn256");
  dim3 grid((a.S + WG_ROWS - 1) / WG_ROWS, a.B * a.H);
  if (DH == 128)
    hipLaunchKernelGGL((attn_fwd_fast<128>), grid, dim3(NT), 0, s, a);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<DH, AttnCfg<DH>::BKV>), grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

template <int DH>
hipError_t bwd_launch(const AttnBwdArgs& a, hipStream_t s) {
  static_assert(DH == 16 || DH == 32 || DH == 128, "head dim served by attn_small / attn256");
  using C = AttnCfg<DH>;
  long rows = (long)a.f.B * a.f.S * a.f.H;
  hipLaunchKernelGGL(attn_delta_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (DH == 128) {
    dim3 gkv((a.f.S + WG_ROWS - 1) / WG_ROWS, a.f.B * a.f.H);
    hipLaunchKernelGGL((attn_bwd_dkdv_fast<128>), gkv, dim3(NT), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 gq((a.f.S + WG_ROWS - 1) / WG_ROWS, a.f.B * a.f.H);
    hipLaunchKernelGGL((attn_bwd_dq_fast<128>), gq, dim3(NT), 0, s, a);
    return hipGetLastError();
  }
  dim3 grid((a.f.S + WG_ROWS - 1) / WG_ROWS, a.f.B * a.f.H, C::NSLICE);
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<DH, C::DHS, C::BQ>), grid, dim3(NT), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<DH, C::DHS, C::BKV>), grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

bool ok16(const void* p, long ld) {
  return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 8 == 0;
}

}  // namespace

hipError_t launch_attention_fwd(const AttnArgs& a, hipStream_t s) {
  if (a.B * a.H * a.S == 0) return hipSuccess;
  if (!ok16(a.q, a.ldq) || !ok16(a.k, a.ldk) || !ok16(a.v, a.ldv)) return hipErrorInvalidValue;
  switch (a.dh) {
    case 16: return fwd_launch<16>(a, s);
    case 32: return fwd_launch<32>(a, s);
    case 128: return fwd_launch<128>(a, s);
    case 64:
    case 80: return attn_small_fwd_eligible(a) ? launch_attn_small_fwd(a, s) : hipErrorInvalidValue;
    case 256: return attn256_fwd_eligible(a) ? launch_attn256_fwd(a, s) : hipErrorInvalidValue;
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention_bwd(const AttnBwdArgs& a, hipStream_t s) {
  if (a.f.B * a.f.H * a.f.S == 0) return hipSuccess;
  if (!ok16(a.f.q, a.f.ldq) || !ok16(a.f.k, a.f.ldk) || !ok16(a.f.v, a.f.ldv) ||
      !ok16(a.dout, a.lddo))
    return hipErrorInvalidValue;
  switch (a.f.dh) {
    case 16: return bwd_launch<16>(a, s);
    case 32: return bwd_launch<32>(a, s);
    case 128: return bwd_launch<128>(a, s);
    case 64:
    case 80: return attn_small_bwd_eligible(a) ? launch_attn_small_bwd(a, s) : hipErrorInvalidValue;
    case 256:
      if (!attn256_bwd_eligible(a)) return hipErrorInvalidValue;
      {  // dQ (which also writes delta), then dK / dV
        hipError_t e = launch_attn256_bwd_dq(a, s);
        return e != hipSuccess ? e : launch_attn256_bwd_dkdv(a, s);
      }
  }
  return hipErrorInvalidValue;
}

// Supported head dims (host query for argument checks).
bool attention_supports_dh(int dh) {
  return dh == 16 || dh == 32 || dh == 64 || dh == 80 || dh == 128 || dh == 256;
}
