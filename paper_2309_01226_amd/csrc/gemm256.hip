// bf16 MFMA GEMM for large, aligned problems: 256 x 256 output tiles,
// K-tiles of 64.
//
//   C[m, n] = sum_k A(m, k) B(n, k), bf16 operands, fp32 accumulation, with
//   the same fused epilogues as the general kernel in gemm.hip.
//
// What bounds it on MI355X (measured with single-purpose variants of this
// kernel): the L2 -> LDS copy stream and, for an M/N-contiguous operand, the
// pass through registers that transposes it, not the matrix cores.  One
// 256 x 256 tile needs 32 bytes per clock per CU at full MFMA rate.  A CU's
// copy throughput is set by the number of 128-byte cache lines it requests,
// not by bytes: rows copied in 64-byte pieces (K-tiles of 32) deliver about
// half of what full-line pieces do.  So K-tiles are 64 deep (a K-contiguous
// row of the tile is exactly one line), 64 KB per K-tile, and the 160 KB of
// LDS holds two and a half of them.  On long K the loop runs at 1.70 PFLOP/s
// with the copies taken out and at about 1.40 with them; staging the copies
// through VGPRs, a second wave per SIMD (8 waves of 128 x 64), staggering the
// first K-tile per workgroup and L2-resident operands each moved that by 4%
// or less.
//
// Both operands K-contiguous (gemm256_kernel): a ring of five single-operand
// slots, three for A and two for B, so that A is copied two K-tiles ahead and
// B one.  The copies are spread evenly: four per wave in every k-step, one
// after every fourth MFMA (details above the kernel).  Issuing the sixteen
// copies of a wave in bursts fills the address unit's queue and stalls the
// MFMAs behind them in the in-order instruction stream (counter
// SQ_VMEM_TA_ADDR_FIFO_FULL).
//
// Layout of an operand tile in LDS: [256 rows][64 k], 128 B per row; the
// eight 16-byte chunks of row r are XOR-swizzled with (r >> 1) & 7, which
// keeps the fragment reads (16 lanes = 16 consecutive rows at one chunk) free
// of bank conflicts.  K-contiguous operands go HBM -> LDS with buffer_load
// ... lds (16 bytes per lane, 1 KB per instruction, no VGPR staging).  Rows
// past M / N and k past K get an out-of-range buffer offset and read as
// zeros.  An M/N-contiguous operand (gemm256_rs_kernel) is loaded into
// registers, transposed there and written in the same layout: the CDNA4
// transposing LDS read (ds_read_b64_tr_b16) would spare the register pass,
// but it costs more LDS time than the MFMAs leave (measured 10-30% slower).
//
// Main loop per K-tile (four k-steps of 16), per wave (128 x 128 sub-tile,
// 4 x 4 MFMA 32x32x16 accumulators in AGPRs): the MFMAs of each k-step are
// interleaved with the fragment reads of the next and with that k-step's
// copies; one wait and one barrier per K-tile, before its last k-step, which
// reads the first fragments of the next tile.
//
// Epilogue: each wave stages one 32-row slab of its sub-tile in its own LDS
// region and stores 4 consecutive columns per lane (16-byte fp32 or 8-byte
// bf16 vectors), so no workgroup barrier is needed between slabs.
#include <algorithm>

#include "adamw_math.h"
#include "common.h"
#include "kernels.h"

namespace {

constexpr int BT = 256;               // tile rows and columns
constexpr int NT = 256;               // 4 wavefronts, 2 x 2
constexpr uint32_t OOB = 0x80000000u; // buffer offset past num_records: reads zero
constexpr int EP = 136;               // fp32 pitch of an epilogue staging row

// Epilogue stores of the interior tiles are nontemporal: a whole tile-wave
// writes its outputs at once, and the streaming hint drains that burst
// measurably faster (about 4% of a 4096 x 28672 x 4096 product).
template <typename T>
__device__ __forceinline__ void store_nt(T* p, const T& v) {
  __builtin_nontemporal_store(v, p);
}

typedef __attribute__((address_space(3))) void lds_void;

// Chunk swizzle of the K-contiguous tile layout (eight 16-byte chunks per row)
__device__ __forceinline__ int swz_k(int row) { return (row >> 1) & 7; }

__device__ __forceinline__ lds_void* lds(const bf16* p) { return (lds_void*)(const_cast<bf16*>(p)); }

constexpr int BK = 64;                // K-tile depth
constexpr int OPE = BT * BK;          // bf16 elements of one operand tile

// Copies of one K-contiguous operand tile: 32 instructions of 1 KB, eight per
// wave.  Instruction j = 4 i + wave fills LDS bytes [1024 j, 1024 j + 1024) of
// the tile (rows 8 j .. 8 j + 7); lane L writes the 16 bytes at 1024 j + 16 L.
// A copy whose k lies at or past K (the K tail, and the tiles past the last
// one that the steady-state loop issues to keep its wait counts constant)
// reads zeros and touches no memory.

struct Loader {
  static constexpr int NI = (BT * BK * 2 / 1024) / 4;  // copy instructions per wave
  uint32_t off[NI];  // byte offsets relative to (tile row 0, k0)
  int kof[NI];       // k of this lane's chunk relative to k0
  __device__ __forceinline__ void init(long ld, int nrows, int wave) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = 8 * (4 * i + wave) + lane / 8;
      const int c = (lane % 8) ^ swz_k(row);
      off[i] = row < nrows ? (uint32_t)(((long)row * ld + 8 * c) * 2) : OOB;
      kof[i] = 8 * c;
    }
  }
  template <int I0 = 0, int I1 = NI>
  __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t rs, int k0, int K, bf16* dst,
                                        int wave) const {
#pragma unroll
    for (int i = I0; i < I1; ++i) {
      const uint32_t o = (k0 + kof[i] < K) ? off[i] : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds(dst + (4 * i + wave) * 512), 16, o,
                                               (uint32_t)(k0 * 2), 0, 0);
    }
  }
};

// Fragment addressing of one operand inside a stage, for the wave's 128-row
// (or column) half `w0` (0 or 128).  frag(sub, ks) is the 32 x 16 MFMA operand
// of rows w0 + 32 sub .. + 31, k = 16 ks .. + 15.
struct Frags {
  static constexpr int KS = BK / 16;
  int o[KS];  // element offsets of k-step ks
  __device__ __forceinline__ void init(int w0) {
    const int lane = threadIdx.x & 63;
    const int r = lane & 31;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) o[ks] = (w0 + r) * BK + 8 * ((2 * ks + (lane >> 5)) ^ swz_k(r));
  }
  __device__ __forceinline__ bf16x8 read(const bf16* tile, int sub, int ks) const {
    return *reinterpret_cast<const bf16x8*>(tile + o[ks] + sub * 32 * BK);
  }
};

__device__ __forceinline__ void read_step(bf16x8 (&fa)[4], bf16x8 (&fb)[4], const Frags& FA,
                                          const Frags& FB, const bf16* sa, const bf16* sb, int ks) {
#pragma unroll
  for (int i = 0; i < 4; ++i) fa[i] = FA.read(sa, i, ks);
#pragma unroll
  for (int j = 0; j < 4; ++j) fb[j] = FB.read(sb, j, ks);
}

__device__ __forceinline__ void mfma_step(floatx16 (&acc)[4][4], const bf16x8 (&fa)[4],
                                          const bf16x8 (&fb)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
}

// Scheduling templates for one k-step of 16 MFMAs: one DS read after each of
// the first ND MFMAs, and one copy after each of the first NV.
template <int ND, int NV>
__device__ __forceinline__ void interleave() {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    if (i < ND) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
}

template <int EPI, int GE>
__device__ __forceinline__ void store4(const GemmArgs& p, long row, int col, floatx4 x) {
  const int N = p.N;
  const long o = row * p.ldo + col;
  if (col + 3 < N) {
    if (EPI == EPI_F32) {
      store_nt(reinterpret_cast<floatx4*>(reinterpret_cast<float*>(p.out) + o), x);
    } else if (EPI == EPI_RESID_F32) {
      const floatx4 r = *reinterpret_cast<const floatx4*>(p.resid + row * p.ldr + col);
      *reinterpret_cast<floatx4*>(reinterpret_cast<float*>(p.out) + o) = x + r;
    } else if (EPI == EPI_BF16) {
      bf16x4 y = {f2bf(x[0]), f2bf(x[1]), f2bf(x[2]), f2bf(x[3])};
      *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(p.out) + o) = y;
      if (p.out2 != nullptr && col >= p.gelu_col0) {
        bf16x4 g = {f2bf(gelu_t<GE>(x[0])), f2bf(gelu_t<GE>(x[1])), f2bf(gelu_t<GE>(x[2])),
                    f2bf(gelu_t<GE>(x[3]))};
        *reinterpret_cast<bf16x4*>(p.out2 + row * p.ldo2 + (col - p.gelu_col0)) = g;
      }
    } else {
      const bf16x4 u = *reinterpret_cast<const bf16x4*>(p.aux + row * p.ldaux + col);
      bf16x4 y;
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = f2bf(x[e] * gelu_grad_t<GE>(bf2f(u[e])));
      *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(p.out) + o) = y;
    }
    return;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int c = col + e;
    if (c >= N) break;
    if (EPI == EPI_F32) {
      reinterpret_cast<float*>(p.out)[o + e] = x[e];
    } else if (EPI == EPI_RESID_F32) {
      reinterpret_cast<float*>(p.out)[o + e] = p.resid[row * p.ldr + c] + x[e];
    } else if (EPI == EPI_BF16) {
      reinterpret_cast<bf16*>(p.out)[o + e] = f2bf(x[e]);
      if (p.out2 != nullptr && c >= p.gelu_col0)
        p.out2[row * p.ldo2 + (c - p.gelu_col0)] = f2bf(gelu_t<GE>(x[e]));
    } else {
      const float u = bf2f(p.aux[row * p.ldaux + c]);
      reinterpret_cast<bf16*>(p.out)[o + e] = f2bf(x[e] * gelu_grad_t<GE>(u));
    }
  }
}

// bf16 epilogues of interior tiles with 16-byte aligned rows: each lane
// stores 8 consecutive columns (one 16-byte store per output, half the store
// instructions of the 4-column layout).  Same per-wave LDS slab staging.
template <int EPI, int GE>
__device__ __forceinline__ void epilogue_bf16_wide(const GemmArgs& p, floatx16 (&acc)[4][4],
                                                   float* st, int m0, int n0, int wave, int lane) {
  const int wm = wave >> 1, wn = wave & 1;
  const int cl = 8 * (lane & 15);
  const int col = n0 + wn * 128 + cl;
  floatx4 b0 = {0.f, 0.f, 0.f, 0.f}, b1 = {0.f, 0.f, 0.f, 0.f};
  if (p.bias != nullptr) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (col + e >= p.bias_col0) b0[e] = p.bias[col + e - p.bias_col0];
      if (col + 4 + e >= p.bias_col0) b1[e] = p.bias[col + 4 + e - p.bias_col0];
    }
  }
  const bool gel = EPI == EPI_BF16 && p.out2 != nullptr && col >= p.gelu_col0;
  // DGELU with column sums: this lane's 8 columns over its rows of the wave's 128
  const bool csum_on = EPI == EPI_DGELU_BF16 && p.colsum_part != nullptr;
  float csum[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) csum[e] = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const long rowbase = m0 + wm * 128 + 32 * i;
    bf16x8 uv[8];
    if (EPI == EPI_DGELU_BF16) {
#pragma unroll
      for (int s = 0; s < 8; ++s)
        uv[s] = *reinterpret_cast<const bf16x8*>(p.aux + (rowbase + 4 * s + (lane >> 4)) * p.ldaux + col);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        st[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * EP + 32 * j + (lane & 31)] = acc[i][j][r];
#pragma unroll(EPI == EPI_BF16 ? 2 : 8)
    for (int s = 0; s < 8; ++s) {
      const int rl = 4 * s + (lane >> 4);
      const long row = rowbase + rl;
      const floatx4 x0 = *reinterpret_cast<const floatx4*>(st + rl * EP + cl) + b0;
      const floatx4 x1 = *reinterpret_cast<const floatx4*>(st + rl * EP + cl + 4) + b1;
      bf16x8 y;
      if (EPI == EPI_BF16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          y[e] = f2bf(x0[e]);
          y[4 + e] = f2bf(x1[e]);
        }
        store_nt(reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(p.out) + row * p.ldo + col), y);
        if (gel) {
          bf16x8 gv;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            gv[e] = f2bf(gelu_t<GE>(x0[e]));
            gv[4 + e] = f2bf(gelu_t<GE>(x1[e]));
          }
          store_nt(reinterpret_cast<bf16x8*>(p.out2 + row * p.ldo2 + (col - p.gelu_col0)), gv);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          y[e] = f2bf(x0[e] * gelu_grad_t<GE>(bf2f(uv[s][e])));
          y[4 + e] = f2bf(x1[e] * gelu_grad_t<GE>(bf2f(uv[s][4 + e])));
        }
        store_nt(reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(p.out) + row * p.ldo + col), y);
        if (csum_on) {
#pragma unroll
          for (int e = 0; e < 8; ++e) csum[e] += bf2f(y[e]);
        }
      }
    }
  }
  if (csum_on) {
    // the four lane groups of a column (rows 4 s + group), added in group order
#pragma unroll
    for (int e = 0; e < 8; ++e) st[(lane >> 4) * 128 + 8 * (lane & 15) + e] = csum[e];
    float* part = p.colsum_part + (long)((m0 + wm * 128) / 128) * p.N + n0 + wn * 128;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = lane + 64 * h;
      const float v = ((st[c] + st[128 + c]) + st[256 + c]) + st[384 + c];
      if (n0 + wn * 128 + c < p.N) part[c] = v;
    }
  }
}

template <int EPI, int GE>
__device__ __forceinline__ void epilogue(const GemmArgs& p, floatx16 (&acc)[4][4], float* stage,
                                         int m0, int n0, int wave, int lane) {
  const int wm = wave >> 1, wn = wave & 1;
  float* st = stage + wave * 32 * EP;
  const int cl = 4 * (lane & 31);
  const int col = n0 + wn * 128 + cl;
  floatx4 bias = {0.f, 0.f, 0.f, 0.f};
  if (p.bias != nullptr) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (col + e < p.N && col + e >= p.bias_col0) bias[e] = p.bias[col + e - p.bias_col0];
  }
  // Tiles wholly inside C (all but the ragged edge) take a branch-free path
  // whose residual / pre-activation loads for a slab are all issued before the
  // slab is staged, so their latency overlaps the LDS traffic.
  const bool interior = m0 + BT <= p.M && n0 + BT <= p.N;
  float csum4[4] = {0.f, 0.f, 0.f, 0.f};  // DGELU column sums of the ragged path
  if (EPI == EPI_BF16 || EPI == EPI_DGELU_BF16) {
    auto a16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    const bool wide = interior && a16(p.out) && p.ldo % 8 == 0 &&
                      (EPI == EPI_BF16 ? (p.out2 == nullptr || (a16(p.out2) && p.ldo2 % 8 == 0 &&
                                                                p.gelu_col0 % 8 == 0))
                                       : (a16(p.aux) && p.ldaux % 8 == 0));
    if (wide) {
      epilogue_bf16_wide<EPI, GE>(p, acc, st, m0, n0, wave, lane);
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const long rowbase = m0 + wm * 128 + 32 * i;
    if (interior) {
      floatx4 rv[16];
      bf16x4 uv[16];
      if (EPI == EPI_RESID_F32) {
#pragma unroll
        for (int s = 0; s < 16; ++s)
          rv[s] = *reinterpret_cast<const floatx4*>(p.resid + (rowbase + 2 * s + (lane >> 5)) * p.ldr + col);
      }
      if (EPI == EPI_DGELU_BF16) {
#pragma unroll
        for (int s = 0; s < 16; ++s)
          uv[s] = *reinterpret_cast<const bf16x4*>(p.aux + (rowbase + 2 * s + (lane >> 5)) * p.ldaux + col);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          st[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * EP + 32 * j + (lane & 31)] = acc[i][j][r];
      const bool gel = EPI == EPI_BF16 && p.out2 != nullptr && col >= p.gelu_col0;
#pragma unroll(EPI == EPI_BF16 ? 4 : 16)
      for (int s = 0; s < 16; ++s) {
        const int rl = 2 * s + (lane >> 5);
        const long row = rowbase + rl;
        const floatx4 x = *reinterpret_cast<const floatx4*>(st + rl * EP + cl) + bias;
        const long o = row * p.ldo + col;
        if (EPI == EPI_F32) {
          store_nt(reinterpret_cast<floatx4*>(reinterpret_cast<float*>(p.out) + o), x);
        } else if (EPI == EPI_RESID_F32) {
          store_nt(reinterpret_cast<floatx4*>(reinterpret_cast<float*>(p.out) + o), floatx4(x + rv[s]));
        } else if (EPI == EPI_BF16) {
          bf16x4 y = {f2bf(x[0]), f2bf(x[1]), f2bf(x[2]), f2bf(x[3])};
          store_nt(reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(p.out) + o), y);
          if (gel) {
            bf16x4 gv = {f2bf(gelu_t<GE>(x[0])), f2bf(gelu_t<GE>(x[1])), f2bf(gelu_t<GE>(x[2])),
                         f2bf(gelu_t<GE>(x[3]))};
            store_nt(reinterpret_cast<bf16x4*>(p.out2 + row * p.ldo2 + (col - p.gelu_col0)), gv);
          }
        } else {
          bf16x4 y;
#pragma unroll
          for (int e = 0; e < 4; ++e) y[e] = f2bf(x[e] * gelu_grad_t<GE>(bf2f(uv[s][e])));
          store_nt(reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(p.out) + o), y);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          st[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * EP + 32 * j + (lane & 31)] = acc[i][j][r];
#pragma unroll 2
      for (int s = 0; s < 16; ++s) {
        const int rl = 2 * s + (lane >> 5);
        const long row = rowbase + rl;
        floatx4 x = *reinterpret_cast<const floatx4*>(st + rl * EP + cl) + bias;
        if (row < p.M) store4<EPI, GE>(p, row, col, x);
        if (EPI == EPI_DGELU_BF16 && p.colsum_part != nullptr) {
          // the values store4 writes, zero past M or N
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int c = col + e;
            const float y = (row < p.M && c < p.N)
                                ? bf2f(f2bf(x[e] * gelu_grad_t<GE>(bf2f(p.aux[row * p.ldaux + c]))))
                                : 0.f;
            csum4[e] += y;
          }
        }
      }
    }
  }
  if (EPI == EPI_DGELU_BF16 && p.colsum_part != nullptr && m0 + wm * 128 < p.M) {
    // the two lane groups of a column (rows 2 s + group), added in group order
#pragma unroll
    for (int e = 0; e < 4; ++e) st[(lane >> 5) * 128 + cl + e] = csum4[e];
    float* part = p.colsum_part + (long)((m0 + wm * 128) / 128) * p.N + n0 + wn * 128;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = lane + 64 * h;
      const float v = st[c] + st[128 + c];
      if (n0 + wn * 128 + c < p.N) part[c] = v;
    }
  }
}

// EPI_ADAMW: the tile is the gradient of a weight W [M, N]; apply one AdamW
// step to the matching elements of W instead of storing the gradient.  Each
// wave stages a 32-row slab of its fp32 sub-tile in its own LDS region (as the
// other epilogues do), updates it four rows at a time with the master /
// moment loads of the next four rows in flight, and stages the updated bf16
// values transposed ([128 columns][32 rows], pitch TP) in a second region, from
// which the transposed copy is written as 16-byte pieces of 8 rows.  Element
// loads and stores stream past the caches: every byte is touched once.
constexpr int TP = 40;  // bf16 pitch of one column of the transposed staging
#ifndef ADAMW_PD
#define ADAMW_PD 2  // groups of four rows whose loads run ahead of the update
#endif

__device__ __forceinline__ void epilogue_adamw(const GemmArgs& p, floatx16 (&acc)[4][4],
                                               float* stage, int m0, int n0, int wave, int lane) {
  const int wm = wave >> 1, wn = wave & 1;
  float* st = stage + wave * 32 * EP;
  bf16* tt = reinterpret_cast<bf16*>(stage + 4 * 32 * EP) + wave * 128 * TP;
  const int cl = 4 * (lane & 31);
  const int col = n0 + wn * 128 + cl;
  const long N = p.N;
  const bool colok = col < p.N;  // N % 8 == 0: a 4-column vector is wholly inside or outside
  const AdamWConsts c = p.opt_c;
  // Buffer resources from the tile's first row: element offsets stay below
  // 2^31 bytes, and an offset past the range (rows at or past M) reads zeros
  // and drops stores, so the loop has no branches (which would turn every
  // wait for loads into a wait for everything).
  constexpr int NT_AUX = 2;  // nontemporal
  const long tile0 = (long)m0 * N;
  auto rsrc = [](const void* q) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(q), (short)0, 0x7FFFFFFF, 0x00020000);
  };
  const __amdgpu_buffer_rsrc_t rP = rsrc(p.opt_p + tile0), rM = rsrc(p.opt_m + tile0),
                               rV = rsrc(p.opt_v + tile0), rS = rsrc(p.opt_sh + tile0);
  // the wave's first column of the transposed copy
  const __amdgpu_buffer_rsrc_t rT = rsrc(p.opt_sht + (long)(n0 + wn * 128) * p.opt_trows);
  const bool keep = p.out != nullptr;
  const __amdgpu_buffer_rsrc_t rG =
      rsrc(keep ? reinterpret_cast<float*>(p.out) + (long)m0 * p.ldo : p.opt_p);
  // The wave's 128 rows are 16 groups of four rows per lane (slab k / 4, group
  // k % 4 of it), software-pipelined across the slabs: the loads of group
  // k + ADAMW_PD are issued before group k is updated and stored, so
  // ADAMW_PD groups (12 KB per wave each) are in flight while the wave
  // computes.  A wave's one vmcnt counts loads and stores in issue order, so
  // the loads must precede the stores they are to overlap.
  auto offs = [&](int k, int u, uint32_t& oe, uint32_t& og) {
    const int r0 = wm * 128 + 32 * (k >> 2);
    const int rl = 2 * (4 * (k & 3) + u) + (lane >> 5);
    const bool ok = colok && m0 + r0 + rl < p.M;
    oe = ok ? (uint32_t)(((long)(r0 + rl) * N + col) * 4) : OOB;
    og = ok ? (uint32_t)(((long)(r0 + rl) * p.ldo + col) * 4) : OOB;
  };
  constexpr int NB = ADAMW_PD + 1;
  floatx4 pv[NB][4], mv[NB][4], vv[NB][4];
  auto load = [&](int k) {
    const int buf = k % NB;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint32_t oe, og;
      offs(k, u, oe, og);
      pv[buf][u] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rP, oe, 0, NT_AUX));
      mv[buf][u] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rM, oe, 0, NT_AUX));
      vv[buf][u] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rV, oe, 0, NT_AUX));
    }
  };
#pragma unroll
  for (int k = 0; k < ADAMW_PD; ++k) load(k);
  // fully unrolled: a slab index that is not a compile-time constant would put
  // the accumulators in scratch memory
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r0 = wm * 128 + 32 * i;  // slab's first row within the tile
    const long rowbase = m0 + r0;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        st[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * EP + 32 * j + (lane & 31)] = acc[i][j][r];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int k = 4 * i + g, buf = k % NB;
      if (k + ADAMW_PD < 16) load(k + ADAMW_PD);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int rl = 2 * (4 * g + u) + (lane >> 5);
        uint32_t oe, og;
        offs(k, u, oe, og);
        const floatx4 gv = *reinterpret_cast<const floatx4*>(st + rl * EP + cl);
        floatx4 pp = pv[buf][u], mm = mv[buf][u], vq = vv[buf][u];
        adamw_four(pp, gv, mm, vq, c);
        // rows past M: zeros in the transposed copy (nothing else is stored)
        const bool ok = oe != OOB;
        bf16x4 b;
#pragma unroll
        for (int e = 0; e < 4; ++e) b[e] = f2bf(ok ? pp[e] : 0.f);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, pp), rP, oe, 0, NT_AUX);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, mm), rM, oe, 0, NT_AUX);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, vq), rV, oe, 0, NT_AUX);
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, b), rS, oe == OOB ? OOB : oe / 2, 0,
                                              NT_AUX);
        if (keep) __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, gv), rG, og, 0, NT_AUX);
#pragma unroll
        for (int e = 0; e < 4; ++e) tt[(cl + e) * TP + rl] = b[e];
      }
    }
    // column jj of the wave's 128, rows 8 q .. 8 q + 7 of the slab (zeros past M)
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int idx = lane + 64 * k;
      const int jj = idx >> 2, q = idx & 3;
      const long r8 = rowbase + 8 * q;
      const bool ok = n0 + wn * 128 + jj < p.N && r8 < p.opt_trows;
      const uint32_t o = ok ? (uint32_t)(((long)jj * p.opt_trows + r8) * 2) : OOB;
      const bf16x8 w = *reinterpret_cast<const bf16x8*>(tt + jj * TP + 8 * q);
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, w), rT, o, 0, NT_AUX);
    }
  }
}

// Output tile of this workgroup.  Workgroups are dealt round-robin over the 8
// XCDs; renumber so that each XCD walks a contiguous range of the tile order,
// then order tiles in groups of 8 tile-rows so that the B tiles of a group
// stay in L2.
// With split-K the grid is (slice, tile) pairs: the renumbered id gives the
// slice (id / tiles) and the tile (id % tiles), so each XCD walks tiles of one
// slice.
__device__ __forceinline__ int xcd_order_id() {
  const int nwg = gridDim.x;
  int bid = blockIdx.x;
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  return bid;
}

__device__ __forceinline__ void tile_origin(int M, int N, int bid, int& m0, int& n0) {
  const int tiles_m = (M + BT - 1) / BT, tiles_n = (N + BT - 1) / BT;
  constexpr int G = 8;
  const int per_group = G * tiles_n;
  const int group = bid / per_group;
  const int first_m = group * G;
  const int gsize = min(tiles_m - first_m, G);
  const int in_g = bid - group * per_group;
  m0 = (first_m + in_g % gsize) * BT;
  n0 = (in_g / gsize) * BT;
}

// Both operands K-contiguous: the five-slot ring.
//
// Slots 0 - 2 hold A tiles (A_t in slot t % 3), slots 3 - 4 B tiles (B_t in
// slot 3 + t % 2).  Iteration t runs k-steps 0 - 2 of tile t, then waits for
// its copies and passes barrier_t, then runs k-step 3 of tile t while reading
// the first fragments of tile t + 1.  After barrier_t no wave reads tile t
// again, so the slots of A_t and B_t are free; the copies of one iteration go
// to slots freed by the previous barrier or by this one:
//   k-step 0: B_{t+1}, second half      k-step 2: A_{t+2}, second half
//   k-step 1: A_{t+2}, first half       k-step 3: B_{t+2}, first half
// Each k-step thus carries exactly four copies per wave, one after every
// fourth MFMA, and eight fragment reads, one after every second MFMA, in the
// order the next k-step consumes them.  At barrier_t only A_{t+2}'s eight
// copies may still be in flight.  Bunching the copies (four or eight at a
// time) stalls the in-order instruction stream behind a full address queue;
// this even spacing measured 3 - 5% faster on the GPT-J shapes.

// Fragment q (0 - 7) of a k-step in the order the MFMAs use it: a0, b0 - b3, a1 - a3.
__device__ __forceinline__ void read_q(bf16x8 (&fa)[4], bf16x8 (&fb)[4], const Frags& FA,
                                       const Frags& FB, const bf16* sa, const bf16* sb, int ks,
                                       int q) {
  if (q == 0) fa[0] = FA.read(sa, 0, ks);
  else if (q <= 4) fb[q - 1] = FB.read(sb, q - 1, ks);
  else fa[q - 4] = FA.read(sa, q - 4, ks);
}

// One k-step: 16 MFMAs on (ca, cb); after MFMA i, fragment read i / 2 of the
// next k-step (odd i) and copy i / 4 (i % 4 == 2).  The scheduling barrier
// after every MFMA pins this order.
template <typename CopyF>
__device__ __forceinline__ void kstep_ring(floatx16 (&acc)[4][4], const bf16x8 (&ca)[4],
                                           const bf16x8 (&cb)[4], bf16x8 (&na)[4], bf16x8 (&nb)[4],
                                           const Frags& FA, const Frags& FB, const bf16* sa,
                                           const bf16* sb, int ks, CopyF copy) {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    acc[i >> 2][i & 3] =
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(ca[i >> 2], cb[i & 3], acc[i >> 2][i & 3], 0, 0, 0);
    if (i & 1) read_q(na, nb, FA, FB, sa, sb, ks, i >> 1);
    if ((i & 3) == 2) copy(i >> 2);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int EPI, int GE>
__global__ __launch_bounds__(NT, 1) void gemm256_kernel(GemmArgs p) {
  static_assert(5 * OPE * 2 <= 163840 && BK == 64 && Loader::NI == 8, "LDS budget / copies");
  __shared__ __attribute__((aligned(1024))) bf16 smem[5 * OPE];

  const int M = p.M, N = p.N;
  int m0, n0, bid = xcd_order_id();
  // split-K: slice `split` covers k in [kb, kb + K) and writes its partial
  // product to the slice's own output block
  const bool sk = EPI == EPI_F32 && p.splitk > 1;
  int split = 0;
  if (sk) {
    const int tiles = ((M + BT - 1) / BT) * ((N + BT - 1) / BT);
    split = bid / tiles;
    bid -= split * tiles;
  }
  tile_origin(M, N, bid, m0, n0);
  const int kb = split * p.splitk_kc;
  const int K = sk ? min(p.splitk_kc, p.K - kb) : p.K;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.A + (long)m0 * p.lda + kb), (short)0, 0x7FFFFFFF, 0x00020000);
  __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.B + (long)n0 * p.ldb + kb), (short)0, 0x7FFFFFFF, 0x00020000);
  Loader la, lb;
  la.init(p.lda, M - m0, wave);
  lb.init(p.ldb, N - n0, wave);
  Frags FA, FB;
  FA.init(wm * 128);
  FB.init(wn * 128);

  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto sA = [&](int t) { return smem + (t % 3) * OPE; };
  auto sB = [&](int t) { return smem + (3 + (t & 1)) * OPE; };
  const int nk = (K + BK - 1) / BK;
  // k offset of tile t; tiles past the last one copy zeros (every chunk at or past K)
  auto kof = [&](int t) { return t < nk ? t * BK : K; };
  // tile 0 resident; A_1 and the first half of B_1 in flight
  la.issue(rsA, 0, K, sA(0), wave);
  lb.issue(rsB, 0, K, sB(0), wave);
  wait_vm_lgkm0<0>();
  cta_barrier();
  la.issue(rsA, kof(1), K, sA(1), wave);
  lb.issue<0, 4>(rsB, kof(1), K, sB(1), wave);
  bf16x8 f0a[4], f0b[4], f1a[4], f1b[4];
#pragma unroll
  for (int q = 0; q < 8; ++q) read_q(f0a, f0b, FA, FB, sA(0), sB(0), 0, q);
  for (int t = 0; t < nk; ++t) {
    const bf16* a = sA(t);
    const bf16* b = sB(t);
    bf16* b1 = sB(t + 1);
    bf16* a2 = sA(t + 2);
    bf16* b2 = sB(t + 2);
    const int k1 = kof(t + 1), k2 = kof(t + 2);
    __builtin_amdgcn_sched_barrier(0);
    kstep_ring(acc, f0a, f0b, f1a, f1b, FA, FB, a, b, 1, [&](int c) {
      switch (c) {
        case 0: lb.issue<4, 5>(rsB, k1, K, b1, wave); break;
        case 1: lb.issue<5, 6>(rsB, k1, K, b1, wave); break;
        case 2: lb.issue<6, 7>(rsB, k1, K, b1, wave); break;
        default: lb.issue<7, 8>(rsB, k1, K, b1, wave); break;
      }
    });
    kstep_ring(acc, f1a, f1b, f0a, f0b, FA, FB, a, b, 2, [&](int c) {
      switch (c) {
        case 0: la.issue<0, 1>(rsA, k2, K, a2, wave); break;
        case 1: la.issue<1, 2>(rsA, k2, K, a2, wave); break;
        case 2: la.issue<2, 3>(rsA, k2, K, a2, wave); break;
        default: la.issue<3, 4>(rsA, k2, K, a2, wave); break;
      }
    });
    kstep_ring(acc, f0a, f0b, f1a, f1b, FA, FB, a, b, 3, [&](int c) {
      switch (c) {
        case 0: la.issue<4, 5>(rsA, k2, K, a2, wave); break;
        case 1: la.issue<5, 6>(rsA, k2, K, a2, wave); break;
        case 2: la.issue<6, 7>(rsA, k2, K, a2, wave); break;
        default: la.issue<7, 8>(rsA, k2, K, a2, wave); break;
      }
    });
    wait_vm_lgkm0<Loader::NI>();  // A_{t+1}, B_{t+1} resident; reads of tile t done
    cta_barrier();                // ... in every wave: A_t's and B_t's slots are free
    kstep_ring(acc, f1a, f1b, f0a, f0b, FA, FB, sA(t + 1), b1, 0, [&](int c) {
      switch (c) {
        case 0: lb.issue<0, 1>(rsB, k2, K, b2, wave); break;
        case 1: lb.issue<1, 2>(rsB, k2, K, b2, wave); break;
        case 2: lb.issue<2, 3>(rsB, k2, K, b2, wave); break;
        default: lb.issue<3, 4>(rsB, k2, K, b2, wave); break;
      }
    });
  }
  wait_vm_lgkm0<0>();  // the zero-filling copies past the last tile
  __syncthreads();
  if constexpr (EPI == EPI_ADAMW) {
    epilogue_adamw(p, acc, reinterpret_cast<float*>(smem), m0, n0, wave, lane);
  } else if constexpr (EPI == EPI_F32) {
    if (split > 0) {
      GemmArgs q = p;
      q.out = reinterpret_cast<float*>(p.out) + split * p.split_stride;
      epilogue<EPI, GE>(q, acc, reinterpret_cast<float*>(smem), m0, n0, wave, lane);
    } else {
      epilogue<EPI, GE>(p, acc, reinterpret_cast<float*>(smem), m0, n0, wave, lane);
    }
  } else {
    epilogue<EPI, GE>(p, acc, reinterpret_cast<float*>(smem), m0, n0, wave, lane);
  }
}

// An M/N-contiguous operand tile (64 k-rows of 256 contiguous m or n) staged
// through registers and written to LDS in the K-contiguous layout, so that
// its fragments are read with plain 16-byte LDS reads like a K-contiguous
// operand's (the transposing LDS read costs more LDS time than the MFMAs
// leave).  Lane (c, g) loads the 8 x 8 block of k-rows 8g .. 8g + 7 and
// columns 8c .. 8c + 7 (one 16-byte load per k-row), transposes it with byte
// permutes and writes it as eight 16-byte pieces: row 8c + e, logical chunk g
// (swizzled like the copied K-contiguous tiles).  Lane assignment:
// c = 8 wave + 2 (lane >> 4) + ((lane >> 3) & 1), g = lane & 7, so that one
// load instruction reads eight whole 128-byte lines (8 lanes per k-row), and
// the 16 lanes of a quarter-wave write 16 different (chunk, row parity) bank
// groups: of the two c in a quarter-wave, the odd one writes the two rows of
// each pair in the opposite order.
struct RegStage {
  static constexpr int NL = 8;  // loads per lane per K-tile
  uint32_t off;                 // byte offset of (k-row 8g, column 8c), or OOB past M / N
  int kr;                       // 8g
  uint32_t sel0, sel1;          // v_perm selectors of even / odd writes
  uint32_t wa[4];               // LDS element offset of write 2s (write 2s + 1: ^ 64)
  u32x4 r[8];                   // r[i]: k-row 8g + i, columns 8c .. 8c + 7
  __device__ __forceinline__ void init(long ld, int nrows) {
    const int t = threadIdx.x, lane = t & 63;
    const int c = 8 * (t >> 6) + 2 * (lane >> 4) + ((lane >> 3) & 1), g = lane & 7;
    const int cp = c & 1;
    kr = 8 * g;
    off = 8 * c < nrows ? (uint32_t)(((long)kr * ld + 8 * c) * 2) : OOB;
    // element h of a pair of bf16 from k-rows 2t (low half) and 2t + 1 (high)
    sel0 = cp ? 0x07060302u : 0x05040100u;  // writes 2s: element cp of dword s
    sel1 = cp ? 0x05040100u : 0x07060302u;  // writes 2s + 1: element 1 - cp
#pragma unroll
    for (int q = 0; q < 4; ++q)
      wa[q] = (uint32_t)(512 * c + 128 * q + 64 * cp + 8 * (g ^ ((4 * cp + q) & 7)));
  }
  template <int I0 = 0, int I1 = NL>
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, int k0, int K, long ld) {
#pragma unroll
    for (int i = I0; i < I1; ++i) {
      const uint32_t o = (k0 + kr + i < K) ? off : OOB;
      r[i] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, o, (uint32_t)((long)(k0 + i) * ld * 2), 0));
    }
  }
  __device__ __forceinline__ void store(bf16* tile) const {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int q = j >> 1;
      const uint32_t sel = (j & 1) ? sel1 : sel0;
      u32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = __builtin_amdgcn_perm(r[2 * e + 1][q], r[2 * e][q], sel);
      *reinterpret_cast<u32x4*>(tile + ((j & 1) ? (wa[q] ^ 64u) : wa[q])) = v;
    }
  }
};

// Scheduling template for one k-step of 16 MFMAs: after MFMA i, one DS read
// if i < ND, one DS write if i < NW, one VMEM instruction if i < NV.
template <int ND, int NW, int NV>
__device__ __forceinline__ void interleave3() {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    if (i < NW) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    if (i < ND) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
}

// GEMM with at least one M/N-contiguous operand: those operands are staged
// through registers (RegStage), a K-contiguous one is copied straight into
// LDS; two LDS stages, both operands in the K-contiguous layout.  Per K-tile
// kt, the staged operands of tile kt + 1 are written into the stage that tile
// kt - 1 released, and the registers are then reloaded with tile kt + 2:
//  * one staged operand: write in k-step 0, loads in k-step 1, and the copies
//    of the other operand's tile kt + 2 after the barrier;
//  * two: A written in k-step 0, B in k-step 1; A's loads over k-steps 0 - 1,
//    B's over k-steps 2 - 3, so that the address unit sees four loads per
//    k-step instead of sixteen at once.
template <int AL, int BL, int EPI, int GE>
__global__ __launch_bounds__(NT, 1) void gemm256_rs_kernel(GemmArgs p) {
  constexpr bool RA = AL == LAY_MN, RB = BL == LAY_MN;
  constexpr int NR = (RA ? 1 : 0) + (RB ? 1 : 0);
  constexpr int NI = Loader::NI;  // copies per wave, or loads per lane, per operand tile
  static_assert(NR >= 1 && NI == RegStage::NL, "staged operand count");
  __shared__ __attribute__((aligned(1024))) bf16 smem[4 * OPE];

  const int M = p.M, N = p.N, K = p.K;
  int m0, n0;
  tile_origin(M, N, xcd_order_id(), m0, n0);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.A + (RA ? (long)m0 : (long)m0 * p.lda)), (short)0, 0x7FFFFFFF, 0x00020000);
  __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.B + (RB ? (long)n0 : (long)n0 * p.ldb)), (short)0, 0x7FFFFFFF, 0x00020000);
  Loader la, lb;
  RegStage ra, rb;
  if constexpr (RA) ra.init(p.lda, M - m0); else la.init(p.lda, M - m0, wave);
  if constexpr (RB) rb.init(p.ldb, N - n0); else lb.init(p.ldb, N - n0, wave);
  Frags FA, FB;
  FA.init(wm * 128);
  FB.init(wn * 128);

  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto copy = [&](int k0, bf16* st) {
    if constexpr (!RA) la.issue(rsA, k0, K, st, wave);
    if constexpr (!RB) lb.issue(rsB, k0, K, st + OPE, wave);
  };
  const int nk = (K + BK - 1) / BK;
  // tile 0 and the registers of tile 1; the operations of tile 1 (NI per
  // operand) are the last issued, so waiting down to 2 NI leaves tile 0 resident
  if constexpr (RA) ra.load(rsA, 0, K, p.lda);
  if constexpr (RB) rb.load(rsB, 0, K, p.ldb);
  copy(0, smem);
  if constexpr (RA) ra.store(smem);
  if constexpr (RB) rb.store(smem + OPE);
  if constexpr (RA) ra.load(rsA, BK, K, p.lda);
  if constexpr (RB) rb.load(rsB, BK, K, p.ldb);
  copy(BK, smem + 2 * OPE);
  wait_vm_lgkm0<2 * NI>();
  cta_barrier();

  bf16x8 f0a[4], f0b[4], f1a[4], f1b[4];
  read_step(f0a, f0b, FA, FB, smem, smem + OPE, 0);
  for (int kt = 0; kt + 1 < nk; ++kt) {
    bf16* cur = smem + (kt & 1) * 2 * OPE;
    bf16* nxt = smem + ((kt + 1) & 1) * 2 * OPE;
    const int k2 = (kt + 2) * BK;
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(acc, f0a, f0b);
    read_step(f1a, f1b, FA, FB, cur, cur + OPE, 1);
    if constexpr (NR == 2) {
      ra.store(nxt);
      ra.template load<0, NI / 2>(rsA, k2, K, p.lda);
      interleave3<8, 8, NI / 2>();
    } else {
      if constexpr (RA) ra.store(nxt);
      else rb.store(nxt + OPE);
      interleave3<8, 8, 0>();
    }
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(acc, f1a, f1b);
    read_step(f0a, f0b, FA, FB, cur, cur + OPE, 2);
    if constexpr (NR == 2) {
      rb.store(nxt + OPE);
      ra.template load<NI / 2, NI>(rsA, k2, K, p.lda);
      interleave3<8, 8, NI / 2>();
    } else {
      if constexpr (RA) ra.load(rsA, k2, K, p.lda);
      else rb.load(rsB, k2, K, p.ldb);
      interleave3<8, 0, NI>();
    }
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(acc, f0a, f0b);
    read_step(f1a, f1b, FA, FB, cur, cur + OPE, 3);
    if constexpr (NR == 2) {
      rb.template load<0, NI / 2>(rsB, k2, K, p.ldb);
      interleave3<8, 0, NI / 2>();
    } else {
      interleave3<8, 0, 0>();
    }
    __builtin_amdgcn_sched_barrier(0);
    // this wave's copies of tile kt + 1 (issued before the register loads of
    // tile kt + 2), its LDS writes and reads; then every other wave's
    wait_vm_lgkm0<NR * NI>();
    cta_barrier();
    copy(k2, cur);
    if constexpr (NR == 2) rb.template load<NI / 2, NI>(rsB, k2, K, p.ldb);
    read_step(f0a, f0b, FA, FB, nxt, nxt + OPE, 0);
    mfma_step(acc, f1a, f1b);
    interleave3<8, 0, NR == 2 ? NI / 2 : NI>();
    __builtin_amdgcn_sched_barrier(0);
  }
  {
    const bf16* cur = smem + ((nk - 1) & 1) * 2 * OPE;
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(acc, f0a, f0b);
    read_step(f1a, f1b, FA, FB, cur, cur + OPE, 1);
    interleave<8, 0>();
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(acc, f1a, f1b);
    read_step(f0a, f0b, FA, FB, cur, cur + OPE, 2);
    interleave<8, 0>();
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(acc, f0a, f0b);
    read_step(f1a, f1b, FA, FB, cur, cur + OPE, 3);
    interleave<8, 0>();
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(acc, f1a, f1b);
  }
  wait_vm_lgkm0<0>();  // the register loads and copies past the last tile
  __syncthreads();
  epilogue<EPI, GE>(p, acc, reinterpret_cast<float*>(smem), m0, n0, wave, lane);
}

template <int AL, int BL, int EPI>
hipError_t launch_e(const GemmArgs& a, hipStream_t s) {
  const int slices = (EPI == EPI_F32 && a.splitk > 1) ? a.splitk : 1;
  dim3 grid((unsigned)(sat_cdiv(a.M, BT) * sat_cdiv(a.N, BT) * slices));
  const bool ge = (EPI == EPI_BF16 || EPI == EPI_DGELU_BF16) && a.gelu_erf;
  if constexpr (EPI == EPI_ADAMW) {
    static_assert(AL == LAY_K && BL == LAY_K, "optimizer epilogue: K-contiguous operands");
    hipLaunchKernelGGL((gemm256_kernel<EPI, 0>), grid, dim3(NT), 0, s, a);
  } else if constexpr (AL == LAY_K && BL == LAY_K) {
    if (ge) hipLaunchKernelGGL((gemm256_kernel<EPI, 1>), grid, dim3(NT), 0, s, a);
    else hipLaunchKernelGGL((gemm256_kernel<EPI, 0>), grid, dim3(NT), 0, s, a);
  } else {
    if (ge) hipLaunchKernelGGL((gemm256_rs_kernel<AL, BL, EPI, 1>), grid, dim3(NT), 0, s, a);
    else hipLaunchKernelGGL((gemm256_rs_kernel<AL, BL, EPI, 0>), grid, dim3(NT), 0, s, a);
  }
  return hipGetLastError();
}

template <int AL, int BL>
hipError_t launch_l(const GemmArgs& a, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_F32: return launch_e<AL, BL, EPI_F32>(a, s);
    case EPI_RESID_F32: return launch_e<AL, BL, EPI_RESID_F32>(a, s);
    case EPI_BF16: return launch_e<AL, BL, EPI_BF16>(a, s);
    case EPI_DGELU_BF16: return launch_e<AL, BL, EPI_DGELU_BF16>(a, s);
    case EPI_ADAMW:
      if constexpr (AL == LAY_K && BL == LAY_K) return launch_e<AL, BL, EPI_ADAMW>(a, s);
      break;
  }
  return hipErrorInvalidValue;
}

inline bool al(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) % bytes) == 0; }

}  // namespace

bool gemm256_eligible(const GemmArgs& a, int alay, int blay, int epi) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return false;
  if (a.splitk > 1) {
    // split-K: fp32 partials without bias, K-contiguous operands, whole 64-deep slices
    if (epi != EPI_F32 || alay != LAY_K || blay != LAY_K || a.bias != nullptr ||
        a.splitk_kc <= 0 || a.splitk_kc % BK || (long)(a.splitk - 1) * a.splitk_kc >= a.K ||
        a.split_stride < (long)(a.M - 1) * a.ldo + a.N)
      return false;
  }
  // at least 64 tiles of 256 x 256: down to a quarter of the CUs, this kernel
  // still beats the general one on twice as many 256 x 128 tiles (measured on
  // the ResNet convolutions, the grid's GPT-2-medium members and GPT-2-small:
  // 1.9 %, 3.1 % and 2.1 % per step), even when half of every tile is padding
  // (128 output columns); split-K products are small by construction and run
  // whatever their tile count
  if (a.splitk <= 1 && (long)sat_cdiv(a.M, BT) * sat_cdiv(a.N, BT) < 64 && a.colsum_part == nullptr)
    return false;
  if (a.colsum_part != nullptr) {
    // DGELU column sums: K-contiguous operands and the 16-byte epilogue for
    // every interior tile
    auto a16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    if (epi != EPI_DGELU_BF16 || alay != LAY_K || blay != LAY_K || !a16(a.out) || a.ldo % 8 ||
        !a16(a.aux) || a.ldaux % 8)
      return false;
  }
  auto r8 = [](long x) { return (x + 7) / 8 * 8; };
  const long lim = 1L << 31;
  // operands: 16-byte copies, 32-bit buffer offsets
  if (!al(a.A, 16) || !al(a.B, 16) || a.lda % 8 || a.ldb % 8) return false;
  if (alay == LAY_K ? (a.K % 8 || (long)BT * a.lda * 2 + 2L * a.K >= lim)
                    : (a.lda < r8(a.M) || ((long)a.K + 256) * a.lda * 2 >= lim))
    return false;
  if (blay == LAY_K ? (a.K % 8 || (long)BT * a.ldb * 2 + 2L * a.K >= lim)
                    : (a.ldb < r8(a.N) || ((long)a.K + 256) * a.ldb * 2 >= lim))
    return false;
  if (epi == EPI_ADAMW) {
    // K-contiguous operands; 4-column vectors of W and 8-row pieces of its
    // transposed copy; the gradient itself only if requested
    auto a16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    return alay == LAY_K && blay == LAY_K && a.N % 8 == 0 && a16(a.opt_p) && a16(a.opt_m) &&
           a16(a.opt_v) && al(a.opt_sh, 8) && a16(a.opt_sht) && a.opt_trows % 8 == 0 &&
           a.opt_trows >= a.M && (a.out == nullptr || (a16(a.out) && a.ldo % 4 == 0));
  }
  // epilogue: 4-column vectors
  if (a.ldo % 4) return false;
  if (epi == EPI_F32 || epi == EPI_RESID_F32) {
    if (!al(a.out, 16)) return false;
    if (epi == EPI_RESID_F32 && (!al(a.resid, 16) || a.ldr % 4)) return false;
  } else {
    if (!al(a.out, 8)) return false;
    if (epi == EPI_BF16 && a.out2 != nullptr && (!al(a.out2, 8) || a.ldo2 % 4 || a.gelu_col0 % 4))
      return false;
    if (epi == EPI_DGELU_BF16 && (!al(a.aux, 8) || a.ldaux % 4)) return false;
  }
  return true;
}

hipError_t launch_gemm256(const GemmArgs& a, int alay, int blay, int epi, hipStream_t s) {
  if (alay == LAY_K && blay == LAY_K) return launch_l<LAY_K, LAY_K>(a, epi, s);
  if (alay == LAY_K && blay == LAY_MN) return launch_l<LAY_K, LAY_MN>(a, epi, s);
  if (alay == LAY_MN && blay == LAY_K) return launch_l<LAY_MN, LAY_K>(a, epi, s);
  return launch_l<LAY_MN, LAY_MN>(a, epi, s);
}

int gemm_splitk(int M, int N, int K, int* kc, int smax) {
  const long tiles = (long)sat_cdiv(M, BT) * sat_cdiv(N, BT);
  if (M <= 0 || N <= 0 || tiles >= 256 || K < 1024) return 1;
  // Estimated time of S slices, in K-tile steps of one tile: the slices run
  // in rounds of 256 workgroups (one per CU), each round as long as one
  // slice; the reduction streams S partial products plus the output (about
  // 9 MB per K-tile step at the measured GEMM and copy rates).  A slice
  // count that spills a few workgroups into a second round loses to a
  // smaller one that fits in the first.
  const int Smax = std::min(smax > 0 ? smax : 16, K / 512);
  int best = 1;
  double best_cost = (double)sat_cdiv(K, BK);
  for (int S = 2; S <= Smax; ++S) {
    const int c = (sat_cdiv(K, S) + BK - 1) / BK * BK;
    const int Se = sat_cdiv(K, c);
    const double rounds = (double)((tiles * Se + 255) / 256);
    const double cost = rounds * (c / BK) + (double)(Se + 1) * M * N * 4.0 / 9e6;
    if (cost < best_cost) {
      best_cost = cost;
      best = S;
    }
  }
  if (best < 2) return 1;
  const int c = (sat_cdiv(K, best) + BK - 1) / BK * BK;
  if (kc) *kc = c;
  return sat_cdiv(K, c);
}

long gemm_splitk_ws_elems(int M, int N, int K, int smax) {
  int kc = 0;
  const int S = gemm_splitk(M, N, K, &kc, smax);
  return S > 1 ? (long)S * M * N : 0;
}

namespace {

// One thread per 4 consecutive outputs of a row; slices summed in order.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ ws, int S,
                                                            long stride, int M, int N,
                                                            float* __restrict__ out, long ldo,
                                                            const float* __restrict__ bias,
                                                            int bias_col0,
                                                            const float* __restrict__ resid,
                                                            long ldr, bool vec) {
  const int n4 = (N + 3) / 4;
  const long total = (long)M * n4;
  for (long t = (long)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (long)gridDim.x * blockDim.x) {
    const long m = t / n4;
    const int n = (int)(t - m * n4) * 4;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (vec) {
      // eight slices' loads in flight per thread, added in slice order
      const float* base = ws + m * N + n;
      for (int s = 0; s < S; s += 8) {
        floatx4 x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (s + u < S) x[u] = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(base + (s + u) * stride));
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (s + u < S) {
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] += x[u][e];
          }
      }
    } else {
      for (int s = 0; s < S; ++s)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e < N) acc[e] += ws[s * stride + m * N + n + e];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int c = n + e;
      if (c >= N) break;
      float v = acc[e];
      if (bias != nullptr && c >= bias_col0) v += bias[c - bias_col0];
      if (resid != nullptr) v = resid[m * ldr + c] + v;
      out[m * ldo + c] = v;
    }
  }
}

}  // namespace

hipError_t launch_splitk_reduce(const float* ws, int S, long stride, int M, int N, float* out,
                                long ldo, const float* bias, int bias_col0, const float* resid,
                                long ldr, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const long total = (long)M * ((N + 3) / 4);
  const bool vec = N % 4 == 0 && stride % 4 == 0 && (reinterpret_cast<uintptr_t>(ws) & 15) == 0;
  const unsigned blocks = (unsigned)std::min<long>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, s, ws, S, stride, M, N, out,
                     ldo, bias, bias_col0, resid, ldr, vec);
  return hipGetLastError();
}
