// bf16 MFMA GEMM for gfx950 with fused epilogues.
//
// Every dense contraction of the fine-tuning step (QKV, out-projection, MLP,
// LM / class head, ViT patch embedding; forward, input-gradient and
// weight-gradient products) runs through this kernel:
//   C[m, n] = sum_k A(m, k) B(n, k), bf16 operands, fp32 accumulation.
//
// Design (CDNA4):
//  * 256 x 256 x 64 block tile (256 x 128 when the grid would not fill the
//    chip), 4 wavefronts in a 2 x 2 grid; each wave owns a 128 x 128 (or
//    128 x 64) sub-tile of v_mfma_f32_32x32x16_bf16 accumulators held in AGPRs.
//  * LDS holds both operand tiles K-contiguous, 64 bf16 (128 bytes) per row,
//    two stages.  The eight 16-byte chunks of a row are XOR-swizzled with the
//    row index (chunk c of row r sits at position c ^ ((r >> 1) & 7)), so the
//    16 lanes of a fragment read that the LDS serves together hit distinct
//    banks without padding.
//  * K-contiguous operands go HBM -> LDS directly with buffer_load ... lds
//    (no VGPR staging, no LDS store instructions); out-of-range rows and the K
//    tail are given an out-of-range buffer offset and read as zeros.
//    M/N-contiguous operands (input-gradient and weight-gradient products) are
//    loaded as 8 x 8 blocks into VGPRs, transposed with v_perm and stored.
//  * Per K-tile: one barrier, then all MFMA fragments of the tile are read
//    into registers, then the next tile's loads are issued into the other
//    stage, then the 64 MFMAs run while those loads are in flight.
//  * Workgroups are renumbered so that consecutive tiles land on the same XCD
//    (the dispatcher deals workgroups round-robin over the 8 XCDs), then
//    ordered in groups of 8 tile-rows for L2 reuse of the B tiles.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace {

constexpr int BK = 64;
constexpr int NT = 256;      // 4 wavefronts in a 2 x 2 grid
constexpr int KV = BK / 8;   // 16-byte chunks per K-row of a tile
constexpr uint32_t OOB = 0x80000000u;  // buffer offset that reads as zero

#define LDS_PTR(p) ((void __attribute__((address_space(3)))*)(p))


// Element offset of (row, chunk) in a swizzled tile.  A 128-bit LDS read is
// served 16 lanes at a time; the 16 lanes of a fragment read cover 16
// consecutive rows (8 even, 8 odd) at one logical chunk, so XOR-ing the chunk
// with bits 1..3 of the row spreads each parity class over all 8 positions.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int sw(int row, int chunk) { return row * BK + ((chunk ^ swz(row)) << 3); }

__device__ __forceinline__ u32x4 load_vec_guarded(const bf16* g, bool ok) {
  u32x4 z = {0u, 0u, 0u, 0u};
  return ok ? *reinterpret_cast<const u32x4*>(g) : z;
}

// Scalar gather of up to 8 consecutive bf16, zero beyond `n_ok`.
__device__ __forceinline__ u32x4 load_scalar8(const bf16* g, int n_ok) {
  uint16_t h[8];
  const uint16_t* gs = reinterpret_cast<const uint16_t*>(g);
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (e < n_ok) ? gs[e] : (uint16_t)0;
  u32x4 r;
  r[0] = h[0] | ((uint32_t)h[1] << 16);
  r[1] = h[2] | ((uint32_t)h[3] << 16);
  r[2] = h[4] | ((uint32_t)h[5] << 16);
  r[3] = h[6] | ((uint32_t)h[7] << 16);
  return r;
}

// ---- K-contiguous operand (row r, k) at G[r * ld + k], straight to LDS.
// Instruction i of wave w fills rows (i*4 + w)*8 .. +7 (1 KB); lane L writes
// LDS chunk position L % 8 of row L / 8, which holds logical chunk
// (L % 8) ^ swz(row).
template <int ROWS>
struct KDma {
  static constexpr int N = 0;  // no staging registers
  static constexpr int NI = ROWS * KV / NT;
  // Byte offsets of this lane's chunks relative to (tile row 0, k = 0);
  // rows past the matrix get the out-of-range offset once, up front.
  uint32_t off[NI];
  __device__ __forceinline__ void init(long ld, int nrows, int wave) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = (i * 4 + wave) * 8 + (lane >> 3);
      const int c = (lane & 7) ^ swz(row);
      off[i] = (row < nrows) ? (uint32_t)(((long)row * ld + c * 8) * 2) : OOB;
    }
  }
  // k0: first column of the K-tile; `tail` = the tile crosses K (then the
  // chunks at or past K are redirected out of range).
  __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t rs, int k0, int K, bool tail, bf16* S,
                                       int wave) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      uint32_t o = off[i];
      if (tail) {
        const int row = (i * 4 + wave) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ swz(row);
        if (k0 + c * 8 >= K) o = OOB;
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, LDS_PTR(S + (i * 4 + wave) * 8 * BK), 16, o,
                                               k0 * 2, 0, 0);
    }
  }
};

// ---- K-contiguous operand through registers (scalar fallback path).
template <int ROWS>
struct KReg {
  static constexpr int N = ROWS * KV / NT;
  __device__ __forceinline__ static void load(const bf16* G, long ld, int r0, int nrows, int k0,
                                              int K, u32x4* regs) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      int v = threadIdx.x + i * NT;
      int r = v / KV, kv = (v % KV) * 8;
      int gr = r0 + r, gk = k0 + kv;
      regs[i] = load_scalar8(G + (long)gr * ld + gk, (gr < nrows) ? min(8, K - gk) : 0);
    }
  }
  __device__ __forceinline__ static void store(bf16* S, const u32x4* regs) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      int v = threadIdx.x + i * NT;
      *reinterpret_cast<u32x4*>(S + sw(v / KV, v % KV)) = regs[i];
    }
  }
};

// ---- M/N-contiguous operand: (row r, k) at G[k * ld + r].  Each thread owns
// 8 x 8 blocks (8 rows x 8 k), loaded as 8 row vectors and transposed in
// registers.  Block b = (rb = b / KV, kb = b % KV): eight consecutive lanes
// cover the eight k-blocks of one row block, so their global loads form
// 128-byte segments.
template <int ROWS>
struct MNReg {
  static constexpr int NB = (ROWS / 8) * KV;          // 8 x 8 blocks per tile
  static constexpr int NPT = (NB + NT - 1) / NT;      // blocks per thread
  static constexpr int N = 8 * NPT;
  template <bool VEC>
  __device__ __forceinline__ static void load(const bf16* G, long ld, int r0, int nrows, int k0,
                                              int K, u32x4* regs) {
    // buffer resource rebased at (k0, r0): out-of-range blocks read as zeros
    __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(G + (long)k0 * ld + r0), (short)0, 0x7FFFFFFF, 0x00020000);
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      int b = threadIdx.x + j * NT;
      if (b >= NB) break;
      int rb = b / KV, kb = b % KV;
      int gr = r0 + rb * 8;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        int gk = k0 + kb * 8 + kk;
        if (VEC) {
          const uint32_t off = (gk < K && gr < nrows) ? (uint32_t)((((long)(kb * 8 + kk)) * ld + rb * 8) * 2) : OOB;
          regs[8 * j + kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
        } else {
          const bf16* src = G + (long)gk * ld + gr;
          regs[8 * j + kk] = load_scalar8(src, (gk < K) ? max(0, min(8, nrows - gr)) : 0);
        }
      }
    }
  }
  __device__ __forceinline__ static void store(bf16* S, const u32x4* regs) {
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      int b = threadIdx.x + j * NT;
      if (b >= NB) break;
      int rb = b / KV, kb = b % KV;
      const u32x4* x = regs + 8 * j;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        u32x4 lo, hi;
#pragma unroll
        for (int w2 = 0; w2 < 4; ++w2) {
          uint32_t a = x[2 * w2][w], c = x[2 * w2 + 1][w];
          lo[w2] = __builtin_amdgcn_perm(c, a, 0x05040100u);  // (a.lo, c.lo)
          hi[w2] = __builtin_amdgcn_perm(c, a, 0x07060302u);  // (a.hi, c.hi)
        }
        *reinterpret_cast<u32x4*>(S + sw(rb * 8 + 2 * w, kb)) = lo;
        *reinterpret_cast<u32x4*>(S + sw(rb * 8 + 2 * w + 1, kb)) = hi;
      }
    }
  }
};

// Operand staging modes.
enum { OP_DMA = 0, OP_KREG = 1, OP_MN = 2 };

template <int MODE, int ROWS, bool VEC>
struct Operand {
  static constexpr int N = MODE == OP_DMA ? 1 : (MODE == OP_KREG ? KReg<ROWS>::N : MNReg<ROWS>::N);
  u32x4 regs[N];
  KDma<ROWS> dma;
  __device__ __forceinline__ void init(long ld, int nrows_from_r0, int wave) {
    if (MODE == OP_DMA) dma.init(ld, nrows_from_r0, wave);
  }
  __device__ __forceinline__ void fetch(const bf16* G, __amdgpu_buffer_rsrc_t rs, long ld, int r0,
                                        int nrows, int k0, int K, bf16* S, int wave) {
    if (MODE == OP_DMA) dma.issue(rs, k0, K, k0 + BK > K, S, wave);
    else if (MODE == OP_KREG) KReg<ROWS>::load(G, ld, r0, nrows, k0, K, regs);
    else MNReg<ROWS>::template load<VEC>(G, ld, r0, nrows, k0, K, regs);
  }
  __device__ __forceinline__ void commit(bf16* S) {
    if (MODE == OP_KREG) KReg<ROWS>::store(S, regs);
    else if (MODE == OP_MN) MNReg<ROWS>::store(S, regs);
  }
};

// One K-tile on stage `cur`: barrier (the tile has landed and no wave still
// reads `nxt`), fragment reads for k-steps 0 and 1, MFMAs of step 0 while the
// reads of steps 2 and 3 are issued, then the next tile's loads into `nxt`
// (issued only after every read of `cur`, so no LDS read waits on them), then
// the MFMAs of steps 1 to 3 while those loads are in flight.
template <int TM, int TN, class OA, class OB>
__device__ __forceinline__ void ktile(floatx16 (&acc)[TM][TN], OA& opA, OB& opB, const GemmArgs& p,
                                      __amdgpu_buffer_rsrc_t rsA, __amdgpu_buffer_rsrc_t rsB,
                                      int a_r0, int a_n, int b_r0, int b_n, const bf16* cur,
                                      bf16* nxt, int kt, int nk, int BMr, int aoff, int boff,
                                      int fhalf, int fsw, int wave) {
  __syncthreads();
  const bool more = kt + 1 < nk;
  const bf16* As = cur + aoff;
  const bf16* Bs = cur + BMr * BK + boff;
  bf16x8 af[BK / 16][TM], bfv[BK / 16][TN];
#define SAT_RD(ks)                                                                    \
  {                                                                                   \
    const int pos = ((2 * (ks) + fhalf) ^ fsw) << 3;                                 \
    _Pragma("unroll") for (int i = 0; i < TM; ++i) af[ks][i] =                        \
        *reinterpret_cast<const bf16x8*>(As + i * 32 * BK + pos);                     \
    _Pragma("unroll") for (int j = 0; j < TN; ++j) bfv[ks][j] =                       \
        *reinterpret_cast<const bf16x8*>(Bs + j * 32 * BK + pos);                     \
  }
#define SAT_MM(ks)                                                                    \
  {                                                                                   \
    _Pragma("unroll") for (int i = 0; i < TM; ++i)                                    \
    _Pragma("unroll") for (int j = 0; j < TN; ++j) acc[i][j] =                        \
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks][i], bfv[ks][j], acc[i][j], 0, 0, 0); \
  }
  SAT_RD(0);
  SAT_RD(1);
  __builtin_amdgcn_sched_barrier(0);
  SAT_MM(0);
  SAT_RD(2);
  SAT_RD(3);
  __builtin_amdgcn_sched_barrier(0);
  if (more) {
    opA.fetch(p.A, rsA, p.lda, a_r0, a_n, (kt + 1) * BK, p.K, nxt, wave);
    opB.fetch(p.B, rsB, p.ldb, b_r0, b_n, (kt + 1) * BK, p.K, nxt + BMr * BK, wave);
  }
  __builtin_amdgcn_sched_barrier(0);
  SAT_MM(1);
  SAT_MM(2);
  SAT_MM(3);
#undef SAT_RD
#undef SAT_MM
  if (more) {
    opA.commit(nxt);
    opB.commit(nxt + BMr * BK);
  }
}

// Epilogue shared by both main loops, staged through LDS one 32-row slab per
// wave at a time: the accumulators (lane = column lane & 31, rows
// 8*(r/4) + 4*(lane/32) + r%4) are written with compile-time indices, then
// each row is read back so that one store instruction covers 64 consecutive
// columns.  `smem` must hold at least 4 * 32 * (BN/2 + 4) floats.
template <int BM, int BN, int EPI, int GE>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& p, floatx16 (&acc)[BM / 64][BN / 64],
                                              bf16* smem, int m0, int n0, int wave, int lane) {
  constexpr int WTM = BM / 2, WTN = BN / 2, TM = WTM / 32, TN = WTN / 32;
  const int M = p.M, N = p.N;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int SP = WTN + 4;           // fp32 pitch of a slab row
  constexpr int CPL = WTN / 64;         // columns per lane in the read phase
  static_assert(4 * 32 * SP * 4 <= 2 * (BM + BN) * BK * 2, "epilogue slabs exceed the LDS tile space");
  float* stage = reinterpret_cast<float*>(smem) + wave * 32 * SP;
  const int colbase = n0 + wn * WTN;
  float bias[CPL];
  bool gel[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int col = colbase + lane + 64 * c;
    bias[c] = (p.bias != nullptr && col < N && col >= p.bias_col0) ? p.bias[col - p.bias_col0] : 0.f;
    gel[c] = (EPI == EPI_BF16) && p.out2 != nullptr && col >= p.gelu_col0;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * SP + j * 32 + (lane & 31)] = acc[i][j][r];
    __syncthreads();
    const int rowbase = m0 + wm * WTM + i * 32;
    // unrolled by 8 so that the residual / pre-activation loads of 8 rows are
    // in flight together instead of one round trip per row
#pragma unroll 8
    for (int rr = 0; rr < 32; ++rr) {
      const long row = rowbase + rr;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int col = colbase + lane + 64 * c;
        if (col >= N || row >= M) continue;
        const float x = stage[rr * SP + lane + 64 * c] + bias[c];
        const long o = row * p.ldo + col;
        if (EPI == EPI_F32) {
          reinterpret_cast<float*>(p.out)[o] = x;
        } else if (EPI == EPI_RESID_F32) {
          reinterpret_cast<float*>(p.out)[o] = p.resid[row * p.ldr + col] + x;
        } else if (EPI == EPI_BF16) {
          reinterpret_cast<bf16*>(p.out)[o] = f2bf(x);
          if (gel[c]) p.out2[row * p.ldo2 + (col - p.gelu_col0)] = f2bf(gelu_t<GE>(x));
        } else {  // EPI_DGELU_BF16
          const float u = bf2f(p.aux[row * p.ldaux + col]);
          reinterpret_cast<bf16*>(p.out)[o] = f2bf(x * gelu_grad_t<GE>(u));
        }
      }
    }
  }
}

// Block tile BM x BN x 64; 4 waves in a 2 x 2 grid, wave tile (BM/2) x (BN/2)
// made of 32 x 32 MFMA tiles.
template <int BM, int BN, int ALAY, int BLAY, int EPI, int GE, bool VEC>
__global__ __launch_bounds__(NT) void gemm_kernel_simple(GemmArgs p) {
  constexpr int WTM = BM / 2, WTN = BN / 2, TM = WTM / 32, TN = WTN / 32;
  constexpr int AMODE = ALAY == LAY_MN ? OP_MN : (VEC ? OP_DMA : OP_KREG);
  constexpr int BMODE = BLAY == LAY_MN ? OP_MN : (VEC ? OP_DMA : OP_KREG);
  constexpr int STAGE = (BM + BN) * BK;  // bf16 elements per stage
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * STAGE];

  const int M = p.M, N = p.N, K = p.K;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int nwg = tiles_m * tiles_n;
  int bid = blockIdx.x;
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  constexpr int G = 8;
  const int per_group = G * tiles_n;
  const int group = bid / per_group;
  const int first_m = group * G;
  const int gsize = min(tiles_m - first_m, G);
  const int in_g = bid - group * per_group;
  const int tile_m = first_m + in_g % gsize;
  const int tile_n = in_g / gsize;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // buffer resources rebased at the tile's first row (K-contiguous operands)
  __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.A + (ALAY == LAY_K ? (long)m0 * p.lda : 0)), (short)0, 0x7FFFFFFF, 0x00020000);
  __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.B + (BLAY == LAY_K ? (long)n0 * p.ldb : 0)), (short)0, 0x7FFFFFFF, 0x00020000);
  const int a_r0 = (AMODE == OP_DMA) ? 0 : m0, a_n = (AMODE == OP_DMA) ? M - m0 : M;
  const int b_r0 = (BMODE == OP_DMA) ? 0 : n0, b_n = (BMODE == OP_DMA) ? N - n0 : N;

  Operand<AMODE, BM, VEC> opA;
  Operand<BMODE, BN, VEC> opB;

  floatx16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (K + BK - 1) / BK;
  opA.init(p.lda, M - m0, wave);
  opB.init(p.ldb, N - n0, wave);
  opA.fetch(p.A, rsA, p.lda, a_r0, a_n, 0, K, smem, wave);
  opB.fetch(p.B, rsB, p.ldb, b_r0, b_n, 0, K, smem + BM * BK, wave);
  opA.commit(smem);
  opB.commit(smem + BM * BK);

  // fragment addressing: row (lane & 31) of each 32-row tile, logical chunk
  // 2 * ks + (lane >> 5), swizzled with swz(row) == swz(lane & 31)
  const int frow = lane & 31, fhalf = lane >> 5, fsw = swz(lane & 31);
  const int aoff = (wm * WTM + frow) * BK, boff = (wn * WTN + frow) * BK;
  for (int kt = 0; kt < nk; ++kt) {
    bf16* cur = smem + (kt & 1) * STAGE;
    bf16* nxt = smem + ((kt + 1) & 1) * STAGE;
    ktile<TM, TN>(acc, opA, opB, p, rsA, rsB, a_r0, a_n, b_r0, b_n, cur, nxt, kt, nk, BM, aoff,
                  boff, fhalf, fsw, wave);
  }

  gemm_epilogue<BM, BN, EPI, GE>(p, acc, smem, m0, n0, wave, lane);
}

// ------------------------------------------------------------------------
// Pipelined main loop (16-byte aligned operands).
//
// Per K-tile k (stage k & 1): MFMAs of k-step 0, fragment reads of k-steps 2
// and 3, MFMAs of steps 1 and 2, then [wait for this wave's copies of tile
// k + 1, barrier], fragment reads of steps 0 and 1 of tile k + 1, the copies of
// tile k + 2 into stage k & 1 (now free), and only then the MFMAs of step 3 of
// tile k, so the matrix cores keep working across the barrier.  Waits are
// explicit s_waitcnt and the barrier carries no memory fence: a fence would
// also wait for the copies that are meant to stay in flight.  The tile
// stages are passed to the inlined helpers as __restrict__ pointers, which
// tells the compiler that reads of one stage never wait on copies into the
// other.

// Operand of the pipelined loop: MODE OP_DMA (K-contiguous, straight to LDS)
// or OP_MN (M/N-contiguous, through registers).
template <int MODE, int ROWS>
struct PipeOperand {
  static constexpr int NREG = MODE == OP_MN ? MNReg<ROWS>::N : 1;
  u32x4 regs[NREG];
  KDma<ROWS> dma;
  // loads issued per wave by one `load` (OP_MN) -- waves past the block
  // count issue none
  __device__ __forceinline__ static int mn_loads(int wave) {
    if (MODE != OP_MN) return 0;
    int n = 0;
#pragma unroll
    for (int j = 0; j < MNReg<ROWS>::NPT; ++j)
      if (wave * 64 + j * NT < MNReg<ROWS>::NB) n += 8;
    return n;
  }
};

template <int MODE, int ROWS>
__device__ __forceinline__ void op_copy(PipeOperand<MODE, ROWS>& o, __amdgpu_buffer_rsrc_t rs,
                                        int k0, int K, bf16* __restrict__ S, int wave) {
  if (MODE == OP_DMA) o.dma.issue(rs, k0, K, k0 + BK > K, S, wave);
}
template <int MODE, int ROWS>
__device__ __forceinline__ void op_load(PipeOperand<MODE, ROWS>& o, const bf16* G, long ld, int r0,
                                        int nrows, int k0, int K) {
  if (MODE == OP_MN) MNReg<ROWS>::template load<true>(G, ld, r0, nrows, k0, K, o.regs);
}
template <int MODE, int ROWS>
__device__ __forceinline__ void op_store(PipeOperand<MODE, ROWS>& o, bf16* __restrict__ S) {
  if (MODE == OP_MN) MNReg<ROWS>::store(S, o.regs);
}

template <int TM, int TN>
__device__ __forceinline__ void frag_read(bf16x8 (&af)[2][TM], bf16x8 (&bfv)[2][TN],
                                          const bf16* __restrict__ stage, int BMr, int aoff,
                                          int boff, int ks0, int fhalf, int fsw) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int pos = ((2 * (ks0 + h) + fhalf) ^ fsw) << 3;
#pragma unroll
    for (int i = 0; i < TM; ++i)
      af[h][i] = *reinterpret_cast<const bf16x8*>(stage + aoff + i * 32 * BK + pos);
#pragma unroll
    for (int j = 0; j < TN; ++j)
      bfv[h][j] = *reinterpret_cast<const bf16x8*>(stage + BMr * BK + boff + j * 32 * BK + pos);
  }
}

template <int TM, int TN>
__device__ __forceinline__ void mfma_step(floatx16 (&acc)[TM][TN], const bf16x8 (&af)[TM],
                                          const bf16x8 (&bfv)[TN]) {
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfv[j], acc[i][j], 0, 0, 0);
}

// After barrier B_j: start tile j + 1 (copies into `nxt`, or register store),
// then the register loads of tile j + 2.
template <int AM, int BMODE, int BM, int BN>
__device__ __forceinline__ void post_barrier(PipeOperand<AM, BM>& A, PipeOperand<BMODE, BN>& B,
                                             const GemmArgs& p, __amdgpu_buffer_rsrc_t rsA,
                                             __amdgpu_buffer_rsrc_t rsB, int m0, int n0, int j,
                                             int nk, bf16* __restrict__ nxt, int wave) {
  if (j + 1 < nk) {
    op_copy(A, rsA, (j + 1) * BK, p.K, nxt, wave);
    op_copy(B, rsB, (j + 1) * BK, p.K, nxt + BM * BK, wave);
    op_store(A, nxt);
    op_store(B, nxt + BM * BK);
  }
  if (j + 2 < nk) {
    op_load(A, p.A, p.lda, m0, p.M, (j + 2) * BK, p.K);
    op_load(B, p.B, p.ldb, n0, p.N, (j + 2) * BK, p.K);
  }
}

template <int BM, int BN, int ALAY, int BLAY, int EPI, int GE>
__global__ __launch_bounds__(NT) void gemm_kernel_pipe(GemmArgs p) {
  constexpr int WTM = BM / 2, WTN = BN / 2, TM = WTM / 32, TN = WTN / 32;
  constexpr int AM = ALAY == LAY_MN ? OP_MN : OP_DMA;
  constexpr int BMD = BLAY == LAY_MN ? OP_MN : OP_DMA;
  constexpr int STAGE = (BM + BN) * BK;
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * STAGE];

  const int M = p.M, N = p.N, K = p.K;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int nwg = tiles_m * tiles_n;
  int bid = blockIdx.x;
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  constexpr int G = 8;
  const int per_group = G * tiles_n;
  const int group = bid / per_group;
  const int first_m = group * G;
  const int gsize = min(tiles_m - first_m, G);
  const int in_g = bid - group * per_group;
  const int m0 = (first_m + in_g % gsize) * BM, n0 = (in_g / gsize) * BN;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.A + (ALAY == LAY_K ? (long)m0 * p.lda : 0)), (short)0, 0x7FFFFFFF, 0x00020000);
  __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.B + (BLAY == LAY_K ? (long)n0 * p.ldb : 0)), (short)0, 0x7FFFFFFF, 0x00020000);
  PipeOperand<AM, BM> A;
  PipeOperand<BMD, BN> B;
  if (AM == OP_DMA) A.dma.init(p.lda, M - m0, wave);
  if (BMD == OP_DMA) B.dma.init(p.ldb, N - n0, wave);
  // register loads outstanding after a post_barrier (per wave)
  const int vm_mn = PipeOperand<AM, BM>::mn_loads(wave) + PipeOperand<BMD, BN>::mn_loads(wave);

  floatx16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (K + BK - 1) / BK;
  // prologue: tile 0 resident in stage 0, registers of tile 1 requested
  op_copy(A, rsA, 0, K, smem, wave);
  op_copy(B, rsB, 0, K, smem + BM * BK, wave);
  op_load(A, p.A, p.lda, m0, M, 0, K);
  op_load(B, p.B, p.ldb, n0, N, 0, K);
  op_store(A, smem);
  op_store(B, smem + BM * BK);
  if (1 < nk) {
    op_load(A, p.A, p.lda, m0, M, BK, K);
    op_load(B, p.B, p.ldb, n0, N, BK, K);
  }
  if (1 < nk && vm_mn == 16) wait_vm_lgkm0<16>();
  else if (1 < nk && vm_mn == 8) wait_vm_lgkm0<8>();
  else wait_vm_lgkm0<0>();
  cta_barrier();

  const int frow = lane & 31, fhalf = lane >> 5, fsw = swz(lane & 31);
  const int aoff = (wm * WTM + frow) * BK, boff = (wn * WTN + frow) * BK;
  bf16x8 f01a[2][TM], f01b[2][TN], f23a[2][TM], f23b[2][TN];
  frag_read<TM, TN>(f01a, f01b, smem, BM, aoff, boff, 0, fhalf, fsw);
  post_barrier<AM, BMD, BM, BN>(A, B, p, rsA, rsB, m0, n0, 0, nk, smem + STAGE, wave);

  for (int kt = 0; kt < nk; ++kt) {
    const bf16* cur = smem + (kt & 1) * STAGE;
    bf16* other = smem + ((kt + 1) & 1) * STAGE;
    __builtin_amdgcn_sched_barrier(0);
    mfma_step<TM, TN>(acc, f01a[0], f01b[0]);
    frag_read<TM, TN>(f23a, f23b, cur, BM, aoff, boff, 2, fhalf, fsw);
    __builtin_amdgcn_sched_barrier(0);
    mfma_step<TM, TN>(acc, f01a[1], f01b[1]);
    mfma_step<TM, TN>(acc, f23a[0], f23b[0]);
    if (kt + 1 < nk) {
      // tile kt + 1 resident: this wave's copies done (only the register
      // loads of tile kt + 2, issued after them, may remain) and its reads done
      const bool loads = kt + 2 < nk;
      if (loads && vm_mn == 16) wait_vm_lgkm0<16>();
      else if (loads && vm_mn == 8) wait_vm_lgkm0<8>();
      else wait_vm_lgkm0<0>();
      cta_barrier();
      frag_read<TM, TN>(f01a, f01b, other, BM, aoff, boff, 0, fhalf, fsw);
      post_barrier<AM, BMD, BM, BN>(A, B, p, rsA, rsB, m0, n0, kt + 1, nk,
                                    smem + (kt & 1) * STAGE, wave);
    }
    __builtin_amdgcn_sched_barrier(0);
    mfma_step<TM, TN>(acc, f23a[1], f23b[1]);
  }
  __syncthreads();
  gemm_epilogue<BM, BN, EPI, GE>(p, acc, smem, m0, n0, wave, lane);
}

template <int BM, int BN, int ALAY, int BLAY, int EPI, int GE>
hipError_t launch5(const GemmArgs& a, bool vec, hipStream_t s) {
  dim3 grid((unsigned)(sat_cdiv(a.M, BM) * sat_cdiv(a.N, BN)));
  if (vec) hipLaunchKernelGGL((gemm_kernel_pipe<BM, BN, ALAY, BLAY, EPI, GE>), grid, dim3(NT), 0, s, a);
  else hipLaunchKernelGGL((gemm_kernel_simple<BM, BN, ALAY, BLAY, EPI, GE, false>), grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int ALAY, int BLAY, int EPI>
hipError_t launch4(const GemmArgs& a, bool vec, hipStream_t s) {
  if (EPI == EPI_BF16 || EPI == EPI_DGELU_BF16) {
    if (a.gelu_erf) return launch5<BM, BN, ALAY, BLAY, EPI, 1>(a, vec, s);
  }
  return launch5<BM, BN, ALAY, BLAY, EPI, 0>(a, vec, s);
}

template <int ALAY, int BLAY, int EPI>
hipError_t launch3(const GemmArgs& a, bool vec, hipStream_t s) {
  // 256 x 256 tiles when they still give every CU at least one tile,
  // 256 x 128 otherwise (and for the scalar-load fallback).
  const long big_tiles = (long)sat_cdiv(a.M, 256) * sat_cdiv(a.N, 256);
  if (vec && big_tiles >= 256) return launch4<256, 256, ALAY, BLAY, EPI>(a, vec, s);
  return launch4<256, 128, ALAY, BLAY, EPI>(a, vec, s);
}

template <int ALAY, int BLAY>
hipError_t launch2(const GemmArgs& a, int epi, bool vec, hipStream_t s) {
  switch (epi) {
    case EPI_F32: return launch3<ALAY, BLAY, EPI_F32>(a, vec, s);
    case EPI_RESID_F32: return launch3<ALAY, BLAY, EPI_RESID_F32>(a, vec, s);
    case EPI_BF16: return launch3<ALAY, BLAY, EPI_BF16>(a, vec, s);
    case EPI_DGELU_BF16: return launch3<ALAY, BLAY, EPI_DGELU_BF16>(a, vec, s);
  }
  return hipErrorInvalidValue;
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

bool gemm_tail_split(int M, int N, int K, int smax, int* M1, int* S, int* kc) {
  const long mt = sat_cdiv(M, 256), nt = sat_cdiv(N, 256), tiles = mt * nt;
  if (tiles <= 256 || tiles % 256 == 0 || nt > 256) return false;
  // head: the rows whose tiles fill whole rounds of 256 workgroups
  const long mh = 256 * (tiles / 256) / nt;
  if (mh <= 0 || mh >= mt) return false;
  const int m2 = M - (int)mh * 256;
  int c = 0;
  const int s = gemm_splitk(m2, N, K, &c, smax);
  if (s <= 1) return false;
  // the same estimate as gemm_splitk, in K-tile steps of one tile: the head's
  // rounds, the tail's slices and their reduction, against every round unsplit
  const double kt = (double)sat_cdiv(K, 64);
  const double head = (double)((mh * nt + 255) / 256) * kt;
  const double tail = (double)((sat_cdiv(m2, 256) * nt * s + 255) / 256) * (c / 64) +
                      (double)(s + 1) * m2 * N * 4.0 / 9e6;
  if (head + tail >= (double)((tiles + 255) / 256) * kt) return false;
  *M1 = (int)mh * 256;
  *S = s;
  *kc = c;
  return true;
}

long gemm_tail_ws_elems(int M, int N, int K, int smax) {
  int m1 = 0, s = 0, c = 0;
  return gemm_tail_split(M, N, K, smax, &m1, &s, &c) ? (long)s * (M - m1) * N : 0;
}

hipError_t launch_gemm(const GemmArgs& a, int alay, int blay, int epi, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.K <= 0) return hipErrorInvalidValue;
  // fp32 outputs with too few tiles to fill the chip: split-K into the
  // caller's workspace, then one reduction that applies bias and residual
  if ((epi == EPI_F32 || epi == EPI_RESID_F32) && alay == LAY_K && blay == LAY_K &&
      a.splitk <= 1 && a.splitk_ws != nullptr) {
    int kc = 0;
    const int S = gemm_splitk(a.M, a.N, a.K, &kc, a.splitk_max);
    if (S > 1 && (long)S * a.M * a.N <= a.splitk_ws_elems) {
      GemmArgs b = a;
      b.out = a.splitk_ws;
      b.ldo = a.N;
      b.bias = nullptr;
      b.resid = nullptr;
      b.splitk = S;
      b.splitk_kc = kc;
      b.split_stride = (long)a.M * a.N;
      if (gemm256_eligible(b, LAY_K, LAY_K, EPI_F32)) {
        hipError_t e = launch_gemm256(b, LAY_K, LAY_K, EPI_F32, s);
        if (e != hipSuccess) return e;
        return launch_splitk_reduce(a.splitk_ws, S, b.split_stride, a.M, a.N,
                                    reinterpret_cast<float*>(a.out), a.ldo, a.bias, a.bias_col0,
                                    epi == EPI_RESID_F32 ? a.resid : nullptr, a.ldr, s);
      }
    }
  }
  // more than 256 tiles with a mostly empty last round: whole rounds of rows
  // unsplit, the remaining rows split-K into the workspace
  if ((epi == EPI_F32 || epi == EPI_RESID_F32) && alay == LAY_K && blay == LAY_K &&
      a.splitk <= 1 && a.splitk_ws != nullptr && !a.no_tail_split) {
    int M1 = 0, S = 0, kc = 0;
    if (gemm_tail_split(a.M, a.N, a.K, a.splitk_max, &M1, &S, &kc) &&
        (long)S * (a.M - M1) * a.N <= a.splitk_ws_elems) {
      GemmArgs h = a;
      h.M = M1;
      GemmArgs t = a;
      t.A = a.A + (long)M1 * a.lda;
      t.M = a.M - M1;
      t.out = a.splitk_ws;
      t.ldo = a.N;
      t.bias = nullptr;
      t.resid = nullptr;
      t.splitk = S;
      t.splitk_kc = kc;
      t.split_stride = (long)t.M * a.N;
      if (gemm256_eligible(h, LAY_K, LAY_K, epi) && gemm256_eligible(t, LAY_K, LAY_K, EPI_F32)) {
        hipError_t e = launch_gemm256(h, LAY_K, LAY_K, epi, s);
        if (e != hipSuccess) return e;
        e = launch_gemm256(t, LAY_K, LAY_K, EPI_F32, s);
        if (e != hipSuccess) return e;
        return launch_splitk_reduce(a.splitk_ws, S, t.split_stride, t.M, a.N,
                                    reinterpret_cast<float*>(a.out) + (long)M1 * a.ldo, a.ldo,
                                    a.bias, a.bias_col0,
                                    epi == EPI_RESID_F32 ? a.resid + (long)M1 * a.ldr : nullptr,
                                    a.ldr, s);
      }
    }
  }
  if (gemm256_eligible(a, alay, blay, epi)) return launch_gemm256(a, alay, blay, epi, s);
  // the optimizer epilogue and the fused column sums exist in the 256 x 256 kernel only
  if (epi == EPI_ADAMW || a.colsum_part != nullptr) return hipErrorInvalidValue;
  // 16-byte loads need aligned rows.  Along K a partial vector would mix in
  // values past K, so K must be a multiple of 8; along M / N a partial vector
  // only feeds output rows / columns that are never stored, so it suffices that
  // the rows are long enough (ld >= M or N rounded up to 8) to stay in bounds.
  auto r8 = [](long x) { return (x + 7) / 8 * 8; };
  bool vec = aligned16(a.A) && aligned16(a.B) && (a.lda % 8 == 0) && (a.ldb % 8 == 0);
  vec = vec && (alay == LAY_K ? (a.K % 8 == 0) : (a.lda >= r8(a.M)));
  vec = vec && (blay == LAY_K ? (a.K % 8 == 0) : (a.ldb >= r8(a.N)));
  if (alay == LAY_K && blay == LAY_K) return launch2<LAY_K, LAY_K>(a, epi, vec, s);
  if (alay == LAY_K && blay == LAY_MN) return launch2<LAY_K, LAY_MN>(a, epi, vec, s);
  if (alay == LAY_MN && blay == LAY_K) return launch2<LAY_MN, LAY_K>(a, epi, vec, s);
  return launch2<LAY_MN, LAY_MN>(a, epi, vec, s);
}
