// Attention forward and backward for 64- and 80-wide heads (GPT-2-style
// decoders, ViT-H/14), causal or bidirectional, on gfx950 MFMA
// (v_mfma_f32_32x32x16_bf16, bf16 operands, fp32 accumulation).
//
// Forward: O = softmax(scale * Q K^T + mask) V per head and the per-query
// natural-log log-sum-exp.  Backward: dV = P^T dO, dP = dO V^T,
// dS = P * (dP - delta), dK = scale dS^T Q, dQ = scale dS K, with P
// recomputed from the saved log-sum-exp and delta = rowsum(dO * O).
//
// Small heads make the softmax, not the matrix cores, the scarce resource:
// per score there are only 4 dh (forward) or 8 dh (backward) MFMA flops
// against one exp and a handful of vector instructions.  So these kernels
// keep the vector work per score minimal (scores are scaled inside the FMA
// that feeds exp2, the running max is raised lazily, masks are evaluated
// only on blocks that cross the diagonal or the sequence end) and keep
// several waves per SIMD so that one wave's exp overlaps another's MFMAs.
//
// Workgroup = 4 waves x 32 rows (queries for the forward and dQ kernels,
// keys for the dK/dV kernel) of one (batch, head); the other operand streams
// through LDS in blocks of 64 rows, two stages, copied HBM -> LDS with
// buffer_load ... lds (no VGPR staging).
//
// Tile layout in LDS (R rows of a [rows][dh] bf16 block):
//  * dims 0..63: R rows of 128 B, eight 16-byte chunks, chunk c of row r
//    stored at c ^ swz(r).  Row-fragment reads (16 lanes = 16 consecutive
//    rows at one chunk) and transposing reads ds_read_b64_tr_b16 (32 lanes
//    = 4 consecutive rows x 4 chunks) then both touch 16 distinct 16-byte
//    bank groups per 256 bytes.
//  * dims 64..79 (80-wide heads): two chunks per row stored chunk-major,
//    [2][R] with row r of chunk t at slot r ^ 4t, after the 64-dim part.
// Products whose output rows are head dims (O^T, dV^T, dK^T, dQ^T) use
// 32-row MFMA tiles; for 80-wide heads the third tile's rows 80..95 read
// dims 64..79 again and are discarded at the store.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int NT = 256;        // 4 waves
constexpr int WR = 32;         // rows owned by a wave
constexpr int WGR = 4 * WR;    // rows owned by a workgroup
constexpr int KB = 64;         // rows per staged block
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr float RESCALE_SLACK = 8.f;
constexpr uint32_t OOB = 0x80000000u;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// The CDNA4 transposing LDS read through a restrict-qualified pointer: once
// inlined, the read carries alias-scope information, so the compiler does not
// make it wait for every LDS copy still in flight (the next block's, which
// land in another stage); the current stage's copies are waited for, and
// published by a barrier, before any wave reads it.
__device__ __forceinline__ bf16x4 ds_read_tr(const lds_bf16x4* __restrict__ p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(const_cast<lds_bf16x4*>(p));
}
__device__ __forceinline__ lds_void* lds(const bf16* p) { return (lds_void*)(const_cast<bf16*>(p)); }

template <int DH>
struct Cfg {
  static_assert(DH == 64 || DH == 80, "64- or 80-wide heads");
  static constexpr bool TAIL = DH == 80;
  static constexpr int KS = DH / 16;         // k-steps over the head dims
  static constexpr int OT = (DH + 31) / 32;  // 32-dim output tiles
};

// chunk swizzle of the 64-dim part
__device__ __forceinline__ int swz(int r) { return (((r >> 1) & 1) << 2) | ((r >> 2) & 3); }

__device__ __forceinline__ floatx16 zero16() {
  floatx16 z;
#pragma unroll
  for (int r = 0; r < 16; ++r) z[r] = 0.f;
  return z;
}
// Row (within a 32 x 32 tile) held by accumulator register r of lane group g.
__device__ __forceinline__ int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }
__device__ __forceinline__ float halves_max(float x) { return fmaxf(x, __shfl_xor(x, 32, 64)); }
__device__ __forceinline__ float halves_sum(float x) { return x + __shfl_xor(x, 32, 64); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* base, long byte_off) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)((const char*)base + byte_off), (short)0, 0x7FFFFFFF,
                                           0x00020000);
}

// Copies of R rows (a block of K, V, Q or dO) into an LDS tile; rows >=
// nvalid read zero.  rs addresses row 0 of the block, rows ld elements apart.
template <int DH, int R>
__device__ __forceinline__ void copy_tile(__amdgpu_buffer_rsrc_t rs, long ld, int nvalid, bf16* dst,
                                          int wave) {
  const int lane = threadIdx.x & 63;
  constexpr int NM = R / 8;  // 1 KB instructions of the 64-dim part
#pragma unroll
  for (int i = 0; i < (NM + 3) / 4; ++i) {
    const int j = 4 * i + wave;
    if (NM % 4 == 0 || j < NM) {
      const int row = 8 * j + (lane >> 3);
      const int c = (lane & 7) ^ swz(row);
      const uint32_t o = row < nvalid ? (uint32_t)(((long)row * ld + 8 * c) * 2) : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds(dst + j * 512), 16, o, 0, 0, 0);
    }
  }
  if constexpr (Cfg<DH>::TAIL) {
    if (wave < R / 32) {  // 2 R slots of 16 bytes
      const int slot = 64 * wave + lane;
      const int t = slot / R;
      const int row = (slot % R) ^ (4 * t);
      const uint32_t o = row < nvalid ? (uint32_t)(((long)row * ld + 64 + 8 * t) * 2) : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds(dst + R * 64 + 512 * wave), 16, o, 0, 0, 0);
    }
  }
}

// Lane-dependent LDS offsets of the two kinds of tile read.
template <int DH, int R>
struct TileOfs {
  int rf[4];   // row fragment, k-step c < 4: row lane % 32, dims 16 c + 8 g .. + 7
  int rft;     // row fragment of k-step 4 (80-wide heads)
  int tr[2];   // transposed read, output tile ot < 2, 16-row step 0, low half
  int trt;     // transposed read of output tile 2 (80-wide heads)
  __device__ __forceinline__ void init(int lane) {
    const int g = lane >> 5, l31 = lane & 31;
#pragma unroll
    for (int c = 0; c < 4; ++c) rf[c] = l31 * 64 + 8 * ((2 * c + g) ^ swz(l31));
    rft = R * 64 + 8 * (g * R + (l31 ^ (4 * g)));
    // lane group G = lane / 16 reads rows 4 (G >> 1) + {0..3} (lo; +8 hi) of
    // dims 32 ot + 16 (G & 1) + 0..15; lane 4 e + q: row e, dims 4 q .. 4 q + 3
    const int G = lane >> 4, ll = lane & 15;
    const int r = 4 * (G >> 1) + (ll >> 2);
#pragma unroll
    for (int ot = 0; ot < 2; ++ot) {
      const int c = 4 * ot + 2 * (G & 1) + ((ll >> 1) & 1);
      tr[ot] = r * 64 + 8 * (c ^ swz(r)) + 4 * (ll & 1);
    }
    const int t = (ll >> 1) & 1;
    trt = R * 64 + 8 * (t * R + (r ^ (4 * t))) + 4 * (ll & 1);
  }
  // Row fragment of k-step c for rows 32 u + lane % 32.
  __device__ __forceinline__ bf16x8 row(const bf16* tile, int u, int c) const {
    const int o = c < 4 ? rf[c & 3] + 32 * u * 64 : rft + 32 * u * 8;
    return *reinterpret_cast<const bf16x8*>(tile + o);
  }
  // Transposed operand (rows = head dims 32 ot + lane % 32, k = 16 tile rows
  // 16 kk .. + 15 in the accumulator permutation) of output tile ot.
  __device__ __forceinline__ bf16x8 trans(const bf16* tile, int kk, int ot) const {
    bf16x4 lo, hi;
    if (ot < 2) {
      const int o = tr[ot & 1] + 16 * kk * 64;
      lo = ds_read_tr((const lds_bf16x4*)lds(tile + o));
      // rows + 8 flip bit 1 of swz, i.e. chunk bit 1
      hi = ds_read_tr((const lds_bf16x4*)lds(tile + ((o ^ 16) + 8 * 64)));
    } else {
      const int o = trt + 16 * kk * 8;
      lo = ds_read_tr((const lds_bf16x4*)lds(tile + o));
      hi = ds_read_tr((const lds_bf16x4*)lds(tile + o + 8 * 8));
    }
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  }
};

// Row fragments (dims 16 c + 8 g .. + 7) of one row per lane, from global;
// rows >= nvalid read zero.
template <int DH>
__device__ __forceinline__ void load_rows(const bf16* base, long ld, int r0, int nvalid, int lane,
                                          bf16x8 (&f)[Cfg<DH>::KS]) {
  const __amdgpu_buffer_rsrc_t rs = rows_rsrc(base, (long)r0 * ld * 2);
  const int r = lane & 31, g = lane >> 5;
  const uint32_t o = r < nvalid ? (uint32_t)(((long)r * ld + 8 * g) * 2) : OOB;
#pragma unroll
  for (int c = 0; c < Cfg<DH>::KS; ++c)
    f[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, o, 32 * c, 0));
}

// Store a transposed accumulator set (rows = head dims, column = this lane's
// row) times f as bf16 into out[0 .. DH).
template <int DH>
__device__ __forceinline__ void store_rowT(bf16* out, const floatx16 (&acc)[Cfg<DH>::OT], float f, int g) {
#pragma unroll
  for (int ot = 0; ot < Cfg<DH>::OT; ++ot)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      if (32 * ot + acc_row(4 * r4, g) >= DH) continue;
      bf16x4 y;
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = f2bf(acc[ot][4 * r4 + e] * f);
      *reinterpret_cast<bf16x4*>(out + 32 * ot + acc_row(4 * r4, g)) = y;
    }
}

// ================================================================ forward
// The score tile is computed transposed, S^T = K Q^T: each lane owns one
// query (two lanes per query, 16 keys each per 32-key tile), so the running
// max and sum are per-lane scalars and the probabilities are directly the B
// operand of O^T += V^T P^T.

template <int DH>
struct FwdState {
  bf16x8 qf[Cfg<DH>::KS];
  floatx16 o[Cfg<DH>::OT];
  float m, l;  // running max (base 2, scaled, lazily raised) and sum
};

// One block of up to 64 keys.  two: keys 32..63 of the block hold a valid
// key for some query of the wave; MASK: some score of the block is masked
// (key >= lim, lim = first excluded key of this lane's query), always the
// case when `two` is false.
template <int DH, bool MASK>
__device__ __forceinline__ void fwd_block(FwdState<DH>& st, const TileOfs<DH, KB>& to, const bf16* Ks,
                                          const bf16* Vs, float sc, bool two, int lim_rel) {
  using C = Cfg<DH>;
  floatx16 s0 = zero16(), s1 = zero16();
#pragma unroll
  for (int c = 0; c < C::KS; ++c) s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.row(Ks, 0, c), st.qf[c], s0, 0, 0, 0);
  if (two) {
#pragma unroll
    for (int c = 0; c < C::KS; ++c) s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.row(Ks, 1, c), st.qf[c], s1, 0, 0, 0);
  }
  float x[32];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    x[r] = s0[r];
    x[16 + r] = s1[r];
  }
  if (MASK) {
    // lim_rel: first excluded key, relative to the block start and 4 g
#pragma unroll
    for (int r = 0; r < 32; ++r) {
      const int kr = 32 * (r >> 4) + 8 * ((r & 15) >> 2) + (r & 3);
      x[r] = kr < lim_rel ? x[r] : -INFINITY;
    }
  }
  float mx = fmaxf(x[0], x[1]);
#pragma unroll
  for (int r = 2; r < 32; r += 2) mx = fmaxf(mx, fmaxf(x[r], x[r + 1]));
  const float mloc = halves_max(mx) * sc;
  const bool raise = mloc > st.m + RESCALE_SLACK;
  if (__builtin_amdgcn_ballot_w64(raise) != 0) {
    const float alpha = (raise && st.m != -INFINITY) ? __builtin_amdgcn_exp2f(st.m - mloc)
                                                     : (raise ? 0.f : 1.f);
    st.l *= alpha;
#pragma unroll
    for (int ot = 0; ot < C::OT; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.o[ot][r] *= alpha;
    st.m = raise ? mloc : st.m;
  }
  const float nm = (st.m == -INFINITY) ? 0.f : -st.m;
  float lsum = 0.f;
  bf16x8 pb[4];
#pragma unroll
  for (int r = 0; r < 32; ++r) {
    const float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(x[r], sc, nm));
    lsum += pr;
    pb[r >> 3][r & 7] = f2bf(pr);
  }
  st.l += halves_sum(lsum);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    if (kk >= 2 && !two) break;
#pragma unroll
    for (int ot = 0; ot < C::OT; ++ot)
      st.o[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.trans(Vs, kk, ot), pb[kk], st.o[ot], 0, 0, 0);
  }
}

template <int DH>
__global__ __launch_bounds__(NT, 2) void attn_small_fwd_kernel(AttnArgs a) {
  using C = Cfg<DH>;
  constexpr int TILE = KB * DH;
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * 2 * TILE];  // 2 stages x (K, V)
  const int S = a.S;
  const int nqb = (S + WGR - 1) / WGR;
  // query blocks outermost; causal: heaviest block of every head first
  const int BH = a.B * a.H;
  const int xb = (int)blockIdx.x / BH, bh = (int)blockIdx.x % BH;
  const int qb = a.causal ? (nqb - 1 - xb) : xb;
  const int b = bh / a.H, h = bh % a.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int q0 = qb * WGR, wq0 = q0 + wave * WR, q = wq0 + (lane & 31);
  const bf16* Qb = a.q + (long)b * S * a.ldq + (long)h * DH;
  const bf16* Kb = a.k + (long)b * S * a.ldk + (long)h * DH;
  const bf16* Vb = a.v + (long)b * S * a.ldv + (long)h * DH;

  FwdState<DH> st;
  load_rows<DH>(Qb, a.ldq, wq0, S - wq0, lane, st.qf);
#pragma unroll
  for (int t = 0; t < C::OT; ++t) st.o[t] = zero16();
  st.m = -INFINITY;
  st.l = 0.f;
  TileOfs<DH, KB> to;
  to.init(lane);
  const float sc = a.scale * LOG2E;
  const int kv_end = a.causal ? min(S, q0 + WGR) : S;
  const int nblk = (kv_end + KB - 1) / KB;
  // keys this wave's queries may see: [0, wk_end); this lane's: [0, lim)
  const int wk_end = a.causal ? min(S, wq0 + WR) : S;
  const int lim = a.causal ? min(S, q + 1) : S;
  const bool wave_live = wq0 < S;

  copy_tile<DH, KB>(rows_rsrc(Kb, 0), a.ldk, S, smem, wave);
  copy_tile<DH, KB>(rows_rsrc(Vb, 0), a.ldv, S, smem + TILE, wave);
  wait_vm_lgkm0<0>();
  cta_barrier();

  for (int j = 0; j < nblk; ++j) {
    const int kv0 = j * KB;
    const bf16* Ks = smem + (j & 1) * 2 * TILE;
    bf16* nxt = smem + ((j + 1) & 1) * 2 * TILE;
    if (j + 1 < nblk) {
      copy_tile<DH, KB>(rows_rsrc(Kb, (long)(kv0 + KB) * a.ldk * 2), a.ldk, S - kv0 - KB, nxt, wave);
      copy_tile<DH, KB>(rows_rsrc(Vb, (long)(kv0 + KB) * a.ldv * 2), a.ldv, S - kv0 - KB, nxt + TILE, wave);
    }
    if (wave_live && kv0 < wk_end) {
      const int nk = min(KB, wk_end - kv0);
      const bool two = nk > 32;
      const bool mask = kv0 + KB > wk_end || (a.causal && kv0 + KB - 1 > wq0);
      if (mask) fwd_block<DH, true>(st, to, Ks, Ks + TILE, sc, two, lim - kv0 - 4 * g);
      else fwd_block<DH, false>(st, to, Ks, Ks + TILE, sc, two, lim - kv0 - 4 * g);
    }
    if (j + 1 < nblk) {
      wait_vm_lgkm0<0>();
      cta_barrier();
    }
  }
  if (q < S) {
    const float inv = (st.l > 0.f) ? 1.f / st.l : 0.f;
    store_rowT<DH>(a.o + ((long)b * S + q) * a.ldo + (long)h * DH, st.o, inv, g);
    if (g == 0) a.lse[((long)b * a.H + h) * S + q] = (st.m + log2f(st.l)) * LN2;
  }
}

// ================================================================ backward, dK and dV
// Each wave owns 32 keys and holds their K and V rows in registers; 64-query
// blocks of Q and dO (with lse * log2 e and delta) stream through LDS.  Per
// 32-query sub-tile: S = Q K^T and dP = dO V^T with queries as rows (lane =
// key), P = exp2(S scale log2e - lse2), dS = P (dP - delta), then
// dV^T += dO^T P and dK^T += Q^T dS with dO^T / Q^T from transposing reads.
template <int DH>
__global__ __launch_bounds__(NT, 2) void attn_small_dkdv_kernel(AttnBwdArgs a) {
  using C = Cfg<DH>;
  constexpr int BQ = KB;
  constexpr int QT = BQ * DH;
  constexpr int STG = 2 * QT + 2 * 2 * BQ;  // Q, dO, lse2[64], delta[64]
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * STG];
  const int S = a.f.S;
  // key blocks outermost: with a causal mask the first keys see the most queries
  const int BH = a.f.B * a.f.H;
  const int bh = (int)blockIdx.x % BH, b = bh / a.f.H, h = bh % a.f.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int k0 = ((int)blockIdx.x / BH) * WGR;
  const int kmin = k0 + wave * WR;
  const int key = kmin + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;
  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;
  const float sc = a.f.scale * LOG2E;

  bf16x8 kf[C::KS], vf[C::KS];
  load_rows<DH>(Kb, a.f.ldk, kmin, S - kmin, lane, kf);
  load_rows<DH>(Vb, a.f.ldv, kmin, S - kmin, lane, vf);
  floatx16 dk[C::OT], dv[C::OT];
#pragma unroll
  for (int t = 0; t < C::OT; ++t) {
    dk[t] = zero16();
    dv[t] = zero16();
  }
  TileOfs<DH, BQ> to;
  to.init(lane);

  const int q_start = a.f.causal ? k0 : 0;
  const int nqb = (S - q_start + BQ - 1) / BQ;
  const bool wave_live = kmin < S;
  float lsd = 0.f;  // wave 0: lse of the next block's query `lane`; wave 1: its delta

  auto stage = [&](int j) { return smem + (j & 1) * STG; };
  auto fetch = [&](int j) {
    const int qs = q_start + j * BQ;
    bf16* st = stage(j);
    copy_tile<DH, BQ>(rows_rsrc(Qb, (long)qs * a.f.ldq * 2), a.f.ldq, S - qs, st, wave);
    copy_tile<DH, BQ>(rows_rsrc(dOb, (long)qs * a.lddo * 2), a.lddo, S - qs, st + QT, wave);
    if (wave < 2) {
      const int qi = qs + lane;
      lsd = qi < S ? (wave ? a.delta[hs + qi] : a.f.lse[hs + qi]) : 0.f;
    }
  };
  auto publish = [&](int j) {
    if (wave < 2) reinterpret_cast<float*>(stage(j) + 2 * QT)[wave * BQ + lane] = wave ? lsd : lsd * LOG2E;
  };

  fetch(0);
  wait_vm_lgkm0<0>();
  publish(0);
  wait_vm_lgkm0<0>();
  cta_barrier();

  for (int j = 0; j < nqb; ++j) {
    const int qs0 = q_start + j * BQ;
    const bf16* Qs = stage(j);
    const bf16* dOs = Qs + QT;
    const float* l2s = reinterpret_cast<const float*>(Qs + 2 * QT);
    const float* dls = l2s + BQ;
    if (j + 1 < nqb) fetch(j + 1);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int qs = qs0 + 32 * u;
      if (!wave_live || qs >= S || (a.f.causal && qs + 31 < kmin)) continue;
      floatx16 x = zero16(), y = zero16();
#pragma unroll
      for (int c = 0; c < C::KS; ++c) x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.row(Qs, u, c), kf[c], x, 0, 0, 0);
#pragma unroll
      for (int c = 0; c < C::KS; ++c) y = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.row(dOs, u, c), vf[c], y, 0, 0, 0);
      const bool mask = qs + 32 > S || (a.f.causal && qs < kmin + 31);
      // query rows acc_row(r, g): valid when row < lim_q and (causal) row >= lim_k
      const int lim_q = S - qs - 4 * g;
      const int lim_k = a.f.causal ? key - qs - 4 * g : -(1 << 30);
      bf16x8 pb[2], db[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const floatx4 l4 = *reinterpret_cast<const floatx4*>(l2s + 32 * u + 8 * i + 4 * g);
        const floatx4 d4 = *reinterpret_cast<const floatx4*>(dls + 32 * u + 8 * i + 4 * g);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * i + e;
          float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(x[r], sc, -l4[e]));
          if (mask) {
            const int rr = 8 * i + e;  // acc_row - 4 g
            pr = (rr < lim_q && rr >= lim_k) ? pr : 0.f;
          }
          pb[r >> 3][r & 7] = f2bf(pr);
          db[r >> 3][r & 7] = f2bf(pr * (y[r] - d4[e]));
        }
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int ot = 0; ot < C::OT; ++ot) {
          dv[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.trans(dOs, 2 * u + hh, ot), pb[hh], dv[ot], 0, 0, 0);
          dk[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.trans(Qs, 2 * u + hh, ot), db[hh], dk[ot], 0, 0, 0);
        }
    }
    if (j + 1 < nqb) {
      wait_vm_lgkm0<0>();
      publish(j + 1);
      wait_vm_lgkm0<0>();
      cta_barrier();
    }
  }
  if (key < S) {
    store_rowT<DH>(a.dk + ((long)b * S + key) * a.lddk + (long)h * DH, dk, a.f.scale, g);
    store_rowT<DH>(a.dv + ((long)b * S + key) * a.lddv + (long)h * DH, dv, 1.f, g);
  }
}

// ================================================================ backward, dQ
// Each wave owns 32 queries and holds their Q and dO rows, lse2 and delta in
// registers; 64-key blocks of K and V stream through LDS.  Per 32-key
// sub-tile: S^T = K Q^T and dP^T = V dO^T (lane = query),
// dS^T = P^T (dP^T - delta), dQ^T += K^T dS^T with K^T from transposing reads.
// This kernel runs first and also computes delta = rowsum(dO * O) for the
// dK / dV kernel.
template <int DH>
__global__ __launch_bounds__(NT, 2) void attn_small_dq_kernel(AttnBwdArgs a) {
  using C = Cfg<DH>;
  constexpr int TILE = KB * DH;
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * 2 * TILE];  // 2 stages x (K, V)
  const int S = a.f.S;
  const int nqb = (S + WGR - 1) / WGR;
  const int BH = a.f.B * a.f.H;
  const int xb = (int)blockIdx.x / BH, bh = (int)blockIdx.x % BH;
  const int qb = a.f.causal ? (nqb - 1 - xb) : xb;
  const int b = bh / a.f.H, h = bh % a.f.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int q0 = qb * WGR, wq0 = q0 + wave * WR, q = wq0 + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;
  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;
  const float sc = a.f.scale * LOG2E;

  bf16x8 qf[C::KS], of[C::KS];
  load_rows<DH>(Qb, a.f.ldq, wq0, S - wq0, lane, qf);
  load_rows<DH>(dOb, a.lddo, wq0, S - wq0, lane, of);
  const float nl2 = q < S ? -a.f.lse[hs + q] * LOG2E : 0.f;
  // delta = rowsum(dO * O) of this lane's query, from the two halves of its row
  float dlt;
  {
    bf16x8 ov[C::KS];
    load_rows<DH>(a.f.o + (long)b * S * a.f.ldo + (long)h * DH, a.f.ldo, wq0, S - wq0, lane, ov);
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < C::KS; ++c)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = __builtin_fmaf(bf2f(of[c][e]), bf2f(ov[c][e]), acc);
    dlt = halves_sum(acc);
    if (g == 0 && q < S) a.delta[hs + q] = dlt;
  }
  floatx16 dq[C::OT];
#pragma unroll
  for (int t = 0; t < C::OT; ++t) dq[t] = zero16();
  TileOfs<DH, KB> to;
  to.init(lane);

  const int kv_end = a.f.causal ? min(S, q0 + WGR) : S;
  const int nkb = (kv_end + KB - 1) / KB;
  const int wk_end = a.f.causal ? min(S, wq0 + WR) : S;
  const int lim = a.f.causal ? min(S, q + 1) : S;
  const bool wave_live = wq0 < S;

  copy_tile<DH, KB>(rows_rsrc(Kb, 0), a.f.ldk, S, smem, wave);
  copy_tile<DH, KB>(rows_rsrc(Vb, 0), a.f.ldv, S, smem + TILE, wave);
  wait_vm_lgkm0<0>();
  cta_barrier();

  for (int j = 0; j < nkb; ++j) {
    const int kv0 = j * KB;
    const bf16* Ks = smem + (j & 1) * 2 * TILE;
    const bf16* Vs = Ks + TILE;
    bf16* nxt = smem + ((j + 1) & 1) * 2 * TILE;
    if (j + 1 < nkb) {
      copy_tile<DH, KB>(rows_rsrc(Kb, (long)(kv0 + KB) * a.f.ldk * 2), a.f.ldk, S - kv0 - KB, nxt, wave);
      copy_tile<DH, KB>(rows_rsrc(Vb, (long)(kv0 + KB) * a.f.ldv * 2), a.f.ldv, S - kv0 - KB, nxt + TILE, wave);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int kv = kv0 + 32 * u;
      if (!wave_live || kv >= wk_end) continue;
      floatx16 x = zero16(), y = zero16();
#pragma unroll
      for (int c = 0; c < C::KS; ++c) x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.row(Ks, u, c), qf[c], x, 0, 0, 0);
#pragma unroll
      for (int c = 0; c < C::KS; ++c) y = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.row(Vs, u, c), of[c], y, 0, 0, 0);
      const bool mask = kv + 32 > wk_end || (a.f.causal && kv + 31 > wq0);
      const int lim_rel = lim - kv - 4 * g;  // keys with acc_row - 4 g < lim_rel are valid
      bf16x8 db[2];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(x[r], sc, nl2));
        if (mask) {
          const int kr = 8 * (r >> 2) + (r & 3);
          pr = kr < lim_rel ? pr : 0.f;
        }
        db[r >> 3][r & 7] = f2bf(pr * (y[r] - dlt));
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int ot = 0; ot < C::OT; ++ot)
          dq[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to.trans(Ks, 2 * u + hh, ot), db[hh], dq[ot], 0, 0, 0);
    }
    if (j + 1 < nkb) {
      wait_vm_lgkm0<0>();
      cta_barrier();
    }
  }
  if (q < S) store_rowT<DH>(a.dq + ((long)b * S + q) * a.lddq + (long)h * DH, dq, a.f.scale, g);
}

bool ok16(const void* p, long ld) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 8 == 0; }
bool ok8(const void* p, long ld) { return (reinterpret_cast<uintptr_t>(p) & 7) == 0 && ld % 4 == 0; }
// byte offsets of a 128-row block stay below 2^31
bool rows_fit(long ld) { return (long)WGR * ld * 2 < (1L << 30); }

}  // namespace

bool attn_small_fwd_eligible(const AttnArgs& a) {
  return (a.dh == 64 || a.dh == 80) && a.scale > 0.f && ok16(a.q, a.ldq) && ok16(a.k, a.ldk) && ok16(a.v, a.ldv) &&
         ok8(a.o, a.ldo) && rows_fit(a.ldq) && rows_fit(a.ldk) && rows_fit(a.ldv);
}

bool attn_small_bwd_eligible(const AttnBwdArgs& a) {
  return attn_small_fwd_eligible(a.f) && ok16(a.dout, a.lddo) && rows_fit(a.lddo) && ok16(a.f.o, a.f.ldo) &&
         rows_fit(a.f.ldo) && a.delta != nullptr && ok8(a.dq, a.lddq) &&
         ok8(a.dk, a.lddk) && ok8(a.dv, a.lddv);
}

hipError_t launch_attn_small_fwd(const AttnArgs& a, hipStream_t s) {
  dim3 grid((unsigned)(((a.S + WGR - 1) / WGR) * a.B * a.H));
  if (a.dh == 64) hipLaunchKernelGGL(attn_small_fwd_kernel<64>, grid, dim3(NT), 0, s, a);
  else hipLaunchKernelGGL(attn_small_fwd_kernel<80>, grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

// dQ (which also writes delta), then dK / dV.
hipError_t launch_attn_small_bwd(const AttnBwdArgs& a, hipStream_t s) {
  dim3 grid((unsigned)(((a.f.S + WGR - 1) / WGR) * a.f.B * a.f.H));
  if (a.f.dh == 64) hipLaunchKernelGGL(attn_small_dq_kernel<64>, grid, dim3(NT), 0, s, a);
  else hipLaunchKernelGGL(attn_small_dq_kernel<80>, grid, dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.f.dh == 64) hipLaunchKernelGGL(attn_small_dkdv_kernel<64>, grid, dim3(NT), 0, s, a);
  else hipLaunchKernelGGL(attn_small_dkdv_kernel<80>, grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}
