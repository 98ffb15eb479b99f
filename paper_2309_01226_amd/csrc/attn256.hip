// Attention forward for 256-wide heads (GPT-J), causal or bidirectional:
// O = softmax(scale * Q K^T + mask) V per head, plus the per-query natural-log
// log-sum-exp that the backward pass recomputes P from.
//
// Layout (one workgroup = 4 waves x 32 queries of one (batch, head)):
//  * The score tile is computed transposed, S^T = K Q^T, so every lane owns
//    one query: its running max and sum are per-lane scalars, and its 16
//    probabilities per 32-key tile already form the B operand of
//    O^T += V^T P^T.  Q stays in registers for the whole key loop.
//  * Per 64-key block, K and V arrive by direct HBM -> LDS copies (two
//    stages; the copies of block j + 1 are issued as soon as block j - 1 is
//    released).  K rows are read as 16-byte row fragments (chunk c of key row
//    r stored at c ^ (r & 15)).  V stays key-major and is read with the CDNA4
//    transposing LDS read ds_read_b64_tr_b16, which hands each lane four
//    consecutive keys of one head dimension, in exactly the key order of the
//    probabilities' accumulator layout (chunk c of key row r stored at
//    c ^ {0, 4, 10, 14}[r & 3] so that the four key rows and the two 16-dim
//    groups a pass serves fall on distinct banks).  No register transposes.
//  * Online softmax in base 2 with a lazily refreshed maximum: the running
//    max m is raised (and O, l rescaled) only when a new score exceeds it by
//    more than 8, so the probabilities exp2(x - m) stay below 2^8 and the
//    128 accumulator rescales are skipped on almost every block.  The result
//    is exact: O and l always share the same m.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int DH = 256;
constexpr int NT = 256;        // 4 waves
constexpr int WQ = 32;         // queries per wave
constexpr int QPB = 4 * WQ;    // queries per workgroup
constexpr int KB = 64;         // keys per block
constexpr int TILE = KB * DH;  // bf16 elements of one K or V block
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

__device__ __forceinline__ int swz_row(int r) { return r & 15; }
__device__ __forceinline__ int swz_tr(int r) { return (0xEA40 >> ((r & 3) << 2)) & 15; }

__device__ __forceinline__ floatx16 zero16() {
  floatx16 z;
#pragma unroll
  for (int r = 0; r < 16; ++r) z[r] = 0.f;
  return z;
}
// Row (within a 32 x 32 tile) held by accumulator register r of lane group g.
__device__ __forceinline__ int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// Copies of one 64-row block (K or V) of this (batch, head): 32 instructions
// of 1 KB (two 512-byte rows each), eight per wave; rows >= nvalid read zero.
// SWZ selects the row-fragment (0) or transposed-read (1) chunk swizzle.
template <int SWZ>
__device__ __forceinline__ void copy_block(__amdgpu_buffer_rsrc_t rs, long ld, int nvalid,
                                           bf16* dst, int wave) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int j = 4 * i + wave;
    const int row = 2 * j + (lane >> 5);
    const int c = (lane & 31) ^ (SWZ ? swz_tr(row) : swz_row(row));
    const uint32_t o = row < nvalid ? (uint32_t)(((long)row * ld + 8 * c) * 2) : OOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds(dst + j * 512), 16, o, 0, 0, 0);
  }
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const bf16* base, int r0, long ld) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)(base + (long)r0 * ld), (short)0, 0x7FFFFFFF,
                                           0x00020000);
}

// Max / sum over the two 32-lane halves (lanes l and l + 32 hold the same
// query).  v_permlane32_swap on a register and itself leaves every lane with
// its own value and its partner's, in one VALU instruction (a cross-lane
// shuffle would go through the LDS unit and wait for it); both lanes of a
// pair then form the same result (IEEE max and add are commutative).
__device__ __forceinline__ float halves_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Per-lane state of one wave: 32 queries, lane = query (two lanes per query).
struct FwdState {
  bf16x8 qf[DH / 16];   // Q operand: dims 16 c + 8 g .. + 7
  floatx16 o[DH / 32];  // O^T accumulators: dims 32 ot + acc_row(r, g)
  float m, l;           // running max (base 2, lazily raised) and sum
  int kofs[8];          // K row-fragment offsets of k-steps 0..7 (+128 for 8..15)
  int vofs[4];          // V^T transposed-read offsets of ot = 0..3 (+128 for 4..7)
};

// One 64-key block: S^T = K Q^T, online softmax (masked only where the block
// crosses the causal diagonal or the sequence end), O^T += V^T P^T.
//
// Both products keep their LDS operand reads a fixed number of MFMAs ahead:
// the reads of step i + PF are issued before the MFMAs of step i, and a
// scheduling barrier after every step pins that order.  Left to itself the
// compiler issued each fragment read right before the MFMA that consumes it
// and waited for it there, so every MFMA of the block paid a full LDS
// latency.
constexpr int PF_K = 3;  // k-steps (two MFMAs each) of K fragments in flight
constexpr int PF_V = 3;  // MFMAs of V^T fragments in flight

__device__ __forceinline__ void fwd_block(FwdState& st, const bf16* Ks, const bf16* Vs, float sc,
                                          int kv0, int q, int S, int causal, int g, bool mask) {
  floatx16 s0 = zero16(), s1 = zero16();
  // K fragment of k-step c, tile t (keys kv0 + 32 t ..): k-steps 8..15 sit 16 chunks further
  auto kread = [&](int c, int t) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(Ks + t * 32 * DH + st.kofs[c & 7] + (c >> 3) * 128);
  };
  bf16x8 kf[PF_K + 1][2];
#pragma unroll
  for (int c = 0; c < PF_K; ++c) {
    kf[c][0] = kread(c, 0);
    kf[c][1] = kread(c, 1);
  }
#pragma unroll
  for (int c = 0; c < DH / 16; ++c) {
    if (c + PF_K < DH / 16) {
      kf[(c + PF_K) % (PF_K + 1)][0] = kread(c + PF_K, 0);
      kf[(c + PF_K) % (PF_K + 1)][1] = kread(c + PF_K, 1);
    }
    s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[c % (PF_K + 1)][0], st.qf[c], s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[c % (PF_K + 1)][1], st.qf[c], s1, 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (mask) {
    // keys past the end, or (causal) past the query, score -inf; lim = first key excluded
    const int lim = min(S, causal ? q + 1 : S) - kv0 - 4 * g;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int kr = 8 * (r >> 2) + (r & 3);  // key - kv0 - 4 g in the first tile
      s0[r] = kr < lim ? s0[r] : -INFINITY;
      s1[r] = kr + 32 < lim ? s1[r] : -INFINITY;
    }
  }
  // the scale is positive, so the largest scaled score is the scaled largest score
  float mraw = fmaxf(s0[0], s1[0]);
#pragma unroll
  for (int r = 1; r < 16; ++r) mraw = fmaxf(mraw, fmaxf(s0[r], s1[r]));
  const float mloc = halves_max(mraw) * sc;
  // lazy max: raise m only when a score exceeds it by more than the slack
  const bool raise = mloc > st.m + RESCALE_SLACK;
  if (__builtin_amdgcn_ballot_w64(raise) != 0) {
    const float alpha = (raise && st.m != -INFINITY) ? __builtin_amdgcn_exp2f(st.m - mloc)
                                                     : (raise ? 0.f : 1.f);
    st.l *= alpha;
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.o[ot][r] *= alpha;
    st.m = raise ? mloc : st.m;
  }
  const float nm = (st.m == -INFINITY) ? 0.f : -st.m;  // all-masked rows: -inf scores give p = 0
  float lsum = 0.f;
  bf16x8 pb[4];
#pragma unroll
  for (int r = 0; r < 32; ++r) {
    const float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(r < 16 ? s0[r] : s1[r - 16], sc, nm));
    lsum += pr;
    pb[r >> 3][r & 7] = f2bf(pr);
  }
  st.l += halves_sum(lsum);
  __builtin_amdgcn_sched_barrier(0);
  // MFMA i = 8 kk + ot: 16-key step kk (keys 16 kk + {4g .. 4g+3, 8+4g .. 8+4g+3}),
  // head dims 32 ot ..; each accumulator still takes its key steps in order
  auto vread = [&](int i) -> bf16x8 {
    const int kk = i >> 3, ot = i & 7;
    const bf16* vb = Vs + 16 * kk * DH + st.vofs[ot & 3] + (ot >> 2) * 128;
    const bf16x4 lo = ds_read_tr((const lds_bf16x4*)lds(vb));
    const bf16x4 hi = ds_read_tr((const lds_bf16x4*)lds(vb + 8 * DH));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  bf16x8 vf[PF_V + 1];
#pragma unroll
  for (int i = 0; i < PF_V; ++i) vf[i] = vread(i);
#pragma unroll
  for (int i = 0; i < 4 * (DH / 32); ++i) {
    if (i + PF_V < 4 * (DH / 32)) vf[(i + PF_V) % (PF_V + 1)] = vread(i + PF_V);
    st.o[i & 7] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[i % (PF_V + 1)], pb[i >> 3], st.o[i & 7], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

__global__ __launch_bounds__(NT, 1) void attn256_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * 2 * TILE];  // 2 stages x (K, V)
  const int S = a.S;
  const int nqb = (S + QPB - 1) / QPB;
  // one-dimensional grid, query blocks outermost: with a causal mask every
  // (batch, head)'s heaviest block is dispatched before any lighter one
  const int BH = a.B * a.H;
  const int xb = (int)blockIdx.x / BH, bh = (int)blockIdx.x % BH;
  const int qb = a.causal ? (nqb - 1 - xb) : xb;
  const int b = bh / a.H, h = bh % a.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int q0 = qb * QPB;
  const int wq0 = q0 + wave * WQ;
  const int q = wq0 + (lane & 31);
  const bf16* Qb = a.q + (long)b * S * a.ldq + (long)h * DH;
  const bf16* Kb = a.k + (long)b * S * a.ldk + (long)h * DH;
  const bf16* Vb = a.v + (long)b * S * a.ldv + (long)h * DH;

  FwdState st;
  {
    const __amdgpu_buffer_rsrc_t rq = rows_rsrc(Qb, wq0, a.ldq);
    const int qr = lane & 31;
    const uint32_t qo = wq0 + qr < S ? (uint32_t)(((long)qr * a.ldq + 8 * g) * 2) : OOB;
#pragma unroll
    for (int c = 0; c < DH / 16; ++c)
      st.qf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rq, qo, 32 * c, 0));
  }
#pragma unroll
  for (int t = 0; t < DH / 32; ++t) st.o[t] = zero16();
  st.m = -INFINITY;
  st.l = 0.f;
  // K fragment of k-step c for key row fr (+32 for the second tile): chunk
  // 2c + g stored at (2c + g) ^ (fr & 15); k-steps 8..15 sit 16 chunks further.
  const int fr = lane & 31;
#pragma unroll
  for (int c = 0; c < 8; ++c) st.kofs[c] = fr * DH + 8 * ((2 * c + g) ^ swz_row(fr));
  // V^T operand: lane group G = lane / 16 reads keys 4 (G >> 1) + {0..3} (low
  // half) and + 8 (high half) of head dims 32 ot + 16 (G & 1) + 0..15; lane
  // 4e + q addresses key e, dims 4q .. 4q + 3.  ot = 4..7 sit 16 chunks further.
  const int G = lane >> 4, ll = lane & 15;
#pragma unroll
  for (int ot = 0; ot < 4; ++ot) {
    const int key = 4 * (G >> 1) + (ll >> 2);
    const int c = 4 * ot + 2 * (G & 1) + ((ll >> 1) & 1);
    st.vofs[ot] = key * DH + 8 * (c ^ swz_tr(key)) + 4 * (ll & 1);
  }
  const float sc = a.scale * LOG2E;
  const int kv_end = a.causal ? min(S, q0 + QPB) : S;
  const int nblk = (kv_end + KB - 1) / KB;

  // prologue: block 0 in stage 0
  copy_block<0>(rows_rsrc(Kb, 0, a.ldk), a.ldk, S, smem, wave);
  copy_block<1>(rows_rsrc(Vb, 0, a.ldv), a.ldv, S, smem + TILE, wave);
  wait_vm_lgkm0<0>();
  cta_barrier();

  for (int j = 0; j < nblk; ++j) {
    const int kv0 = j * KB;
    const bf16* Ks = smem + (j & 1) * 2 * TILE;
    bf16* nxt = smem + ((j + 1) & 1) * 2 * TILE;
    if (j + 1 < nblk) {
      copy_block<0>(rows_rsrc(Kb, kv0 + KB, a.ldk), a.ldk, S - kv0 - KB, nxt, wave);
      copy_block<1>(rows_rsrc(Vb, kv0 + KB, a.ldv), a.ldv, S - kv0 - KB, nxt + TILE, wave);
    }
    if (!(a.causal && kv0 > wq0 + WQ - 1)) {
      const bool mask = kv0 + KB > S || (a.causal && kv0 + KB - 1 > wq0);
      fwd_block(st, Ks, Ks + TILE, sc, kv0, q, S, a.causal, g, mask);
    }
    if (j + 1 < nblk) {
      wait_vm_lgkm0<0>();
      cta_barrier();
    }
  }
  if (q < S) {
    const float inv = (st.l > 0.f) ? 1.f / st.l : 0.f;
    bf16* Ob = a.o + ((long)b * S + q) * a.ldo + (long)h * DH;
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        bf16x4 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = f2bf(st.o[ot][4 * r4 + e] * inv);
        *reinterpret_cast<bf16x4*>(Ob + 32 * ot + acc_row(4 * r4, g)) = y;
      }
    if (g == 0) a.lse[((long)b * a.H + h) * S + q] = (st.m + log2f(st.l)) * LN2;
  }
}


// ================================================================ backward, dK and dV
// Workgroup = 8 waves = 4 pairs; pair p owns keys k0 + 32 p .. + 31 of one
// (batch, head) and loops over 32-query blocks.  Wave p (role A) holds K
// (half in registers, half in LDS), forms P = exp2(S log2e - lse) from S = Q K^T and accumulates
// dV^T += dO^T P; wave p + 4 (role B) holds V, forms dP = dO V^T, takes P from
// its partner through LDS and accumulates dK^T += Q^T dS, dS = P (dP - delta).
// Every SIMD hosts one wave of each role.  The Q and dO rows of a block are
// copied HBM -> LDS once and read both as row fragments (S, dP) and, through
// the transposing LDS read, as Q^T / dO^T (dK, dV); their chunk swizzle
// c ^ (4 (r & 3) + ((r >> 2) & 3)) keeps both kinds of read free of bank
// conflicts.  lse (times log2 e) and delta of the block travel with it.
constexpr int BQ = 32;          // queries per block
constexpr int KPW = 128;        // keys per workgroup
constexpr int NT8 = 512;        // 8 waves
constexpr int QT = BQ * DH;     // bf16 elements of one 32-row tile
constexpr int STG_B = 2 * QT + 2 * 2 * BQ;  // Q rows, dO rows, lse2[32], delta[32] (fp32 as bf16 pairs)
// Fragment reads are issued ahead of the MFMAs that take them (the compiler
// otherwise waits for each read right before its MFMA).  The first NRF of a
// lane's 16 resident K / V fragments stay in registers and the rest in LDS,
// which keeps the read-ahead registers within the budget of two waves per SIMD.
constexpr int PF_R = 2;   // dK / dV: row-fragment reads in flight (S, dP products)
constexpr int PF_T = 2;   // dK / dV: transposed reads in flight (dV, dK products)
constexpr int NRF = 8;    // dK / dV: resident fragments kept in registers
constexpr int PF_RQ = 1;  // dQ: row-fragment reads in flight (S^T, dP^T products)

__device__ __forceinline__ int swz_dual(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

// 32 rows of 512 bytes: 16 copy instructions, two per wave of eight.
__device__ __forceinline__ void copy_rows32(__amdgpu_buffer_rsrc_t rs, long ld, int nvalid, bf16* dst,
                                            int wave) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int j = 8 * i + wave;
    const int row = 2 * j + (lane >> 5);
    const int c = (lane & 31) ^ swz_dual(row);
    const uint32_t o = row < nvalid ? (uint32_t)(((long)row * ld + 8 * c) * 2) : OOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds(dst + j * 512), 16, o, 0, 0, 0);
  }
}

// Row fragment (A operand, rows = tile rows, k = dims 16 c + 8 g .. + 7) of
// row r of a dual-swizzled tile.
__device__ __forceinline__ bf16x8 row_frag(const bf16* tile, int r, int c, int g) {
  return *reinterpret_cast<const bf16x8*>(tile + r * DH + 8 * ((2 * c + g) ^ swz_dual(r)));
}

__global__ __launch_bounds__(NT8, 1) void attn256_bwd_dkdv_kernel(AttnBwdArgs a) {
  constexpr int SMEM = 2 * STG_B + 4 * 64 * 16 * 2 + 8 * (DH / 16 - NRF) * 64 * 8;
  static_assert(SMEM * 2 <= 163840, "LDS budget");
  __shared__ __attribute__((aligned(1024))) bf16 smem[SMEM];
  float* xbuf = reinterpret_cast<float*>(smem + 2 * STG_B);  // P exchange: [pair][16][64 lanes]
  // resident fragments NRF.. of every wave: [wave][fragment][lane], 16 bytes each
  bf16* rfs = smem + 2 * STG_B + 4 * 64 * 16 * 2;
  const int S = a.f.S;
  // one-dimensional grid, key blocks outermost: with a causal mask the
  // first key blocks see the most queries and are dispatched first
  const int BH = a.f.B * a.f.H;
  const int bh = (int)blockIdx.x % BH, b = bh / a.f.H, h = bh % a.f.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int pair = wave & 3, role = wave >> 2;
  const int k0 = ((int)blockIdx.x / BH) * KPW;
  const int kmin = k0 + pair * 32;
  const int key = kmin + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;
  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;
  const float sc = a.f.scale * LOG2E;

  // resident operand: K (role A) or V (role B) of this lane's key, dims 16 c + 8 g .. + 7
  bf16x8 rf[NRF];
  bf16* rfw = rfs + (wave * (DH / 16 - NRF) * 64 + lane) * 8;  // this lane's fragment NRF; next: + 512
  {
    const bf16* base = role ? Vb : Kb;
    const long ld = role ? a.f.ldv : a.f.ldk;
    const __amdgpu_buffer_rsrc_t rk = rows_rsrc(base, kmin, ld);
    const uint32_t ko = key < S ? (uint32_t)(((long)(lane & 31) * ld + 8 * g) * 2) : OOB;
#pragma unroll
    for (int c = 0; c < NRF; ++c)
      rf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, ko, 32 * c, 0));
#pragma unroll
    for (int c = NRF; c < DH / 16; ++c)
      *reinterpret_cast<bf16x8*>(rfw + (c - NRF) * 512) =
          __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, ko, 32 * c, 0));
  }
  floatx16 acc[DH / 32];  // dV^T (role A) or dK^T (role B): dims 32 ot + acc_row(r, g), key = lane
#pragma unroll
  for (int t = 0; t < DH / 32; ++t) acc[t] = zero16();
  // transposed reads of a 32-row tile (Q^T or dO^T): lane group G reads rows
  // 4 (G >> 1) + 8 hsel + {0..3} (+ 16 hh), dims 32 ot + 16 (G & 1) + 0..15
  const int G = lane >> 4, ll = lane & 15;
  int tofs[4];
#pragma unroll
  for (int ot = 0; ot < 4; ++ot) {
    const int r = 4 * (G >> 1) + (ll >> 2);
    const int c = 4 * ot + 2 * (G & 1) + ((ll >> 1) & 1);
    tofs[ot] = r * DH + 8 * (c ^ swz_dual(r)) + 4 * (ll & 1);
  }

  const int q_start = a.f.causal ? k0 : 0;
  const int nqb = (S - q_start + BQ - 1) / BQ;
  float* xw = xbuf + pair * 16 * 64;
  float lsd = 0.f;  // wave 0: lse2 (lanes 0..31) or delta (lanes 32..63) of the next block

  auto stage_ptr = [&](int j) { return smem + (j & 1) * STG_B; };
  auto fetch = [&](int j) {  // copies of block j; wave 0 also loads its lse / delta
    const int qs = q_start + j * BQ;
    bf16* st = stage_ptr(j);
    copy_rows32(rows_rsrc(Qb, qs, a.f.ldq), a.f.ldq, S - qs, st, wave);
    copy_rows32(rows_rsrc(dOb, qs, a.lddo), a.lddo, S - qs, st + QT, wave);
    if (wave == 0) {
      // the raw value: scaling it here would make the wave wait for the
      // copies just issued (one vmcnt counts loads in issue order)
      const int qi = qs + (lane & 31);
      lsd = qi < S ? (g ? a.delta[hs + qi] : a.f.lse[hs + qi]) : 0.f;
    }
  };
  auto publish = [&](int j) {  // wave 0 stores lse2 / delta of block j (after its loads landed)
    if (wave == 0) reinterpret_cast<float*>(stage_ptr(j) + 2 * QT)[lane] = g ? lsd : lsd * LOG2E;
  };

  fetch(0);
  wait_vm_lgkm0<0>();
  publish(0);
  wait_vm_lgkm0<0>();
  cta_barrier();

  for (int j = 0; j < nqb; ++j) {
    const int qs0 = q_start + j * BQ;
    const bf16* st = stage_ptr(j);
    const bf16* Qs = st;
    const bf16* dOs = st + QT;
    const float* lsd_s = reinterpret_cast<const float*>(st + 2 * QT);
    const bool active = !(a.f.causal && qs0 + BQ - 1 < kmin);
    // S = Q K^T (role A) or dP = dO V^T (role B): rows = queries, column = key
    floatx16 x = zero16();
    if (active) {
      // fragment reads PF_R k-steps ahead of their MFMA
      const bf16* rows = role ? dOs : Qs;
      bf16x8 fr[PF_R + 1], fb[PF_R + 1];
      auto rread = [&](int c) {
        fr[c % (PF_R + 1)] = row_frag(rows, lane & 31, c, g);
        if (c >= NRF) fb[c % (PF_R + 1)] = *reinterpret_cast<const bf16x8*>(rfw + (c - NRF) * 512);
      };
#pragma unroll
      for (int c = 0; c < PF_R; ++c) rread(c);
#pragma unroll
      for (int c = 0; c < DH / 16; ++c) {
        if (c + PF_R < DH / 16) rread(c + PF_R);
        x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[c % (PF_R + 1)], c < NRF ? rf[c] : fb[c % (PF_R + 1)], x,
                                                    0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // The next block's copies go out after this block's resident-operand
    // products (issued before them, the kernel alone ran 1.5 % faster but
    // the step, where it shares the chip, no faster).
    if (j + 1 < nqb) fetch(j + 1);
    if (active) {
      if (role == 0) {
        // P = exp2(S log2e - lse2); zero for queries past S and (causal) keys past the query
        const int lim_q = S - qs0 - 4 * g;            // rows r with acc_row < lim_q are valid
        const int lim_k = key - qs0 - 4 * g;          // causal: need acc_row >= key - qs0
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const floatx4 l4 = *reinterpret_cast<const floatx4*>(lsd_s + 8 * i + 4 * g);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int rr = 8 * i + e;  // acc_row - 4 g
            float pr = __builtin_amdgcn_exp2f(x[4 * i + e] * sc - l4[e]);
            const bool ok = (rr < lim_q) & ((a.f.causal == 0) | (rr >= lim_k));
            pr = ok ? pr : 0.f;
            x[4 * i + e] = pr;
            xw[(4 * i + e) * 64 + lane] = pr;
          }
        }
      }
    }
    wait_lgkm0();
    cta_barrier();  // P of every pair visible
    if (active) {
      if (role == 1) {
        // dS = P (dP - delta)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const floatx4 d4 = *reinterpret_cast<const floatx4*>(lsd_s + BQ + 8 * i + 4 * g);
#pragma unroll
          for (int e = 0; e < 4; ++e) x[4 * i + e] = xw[(4 * i + e) * 64 + lane] * (x[4 * i + e] - d4[e]);
        }
      }
      // dV^T += dO^T P (role A) or dK^T += Q^T dS (role B); the transposed
      // reads run PF_T MFMAs ahead
      const bf16* tt = role ? Qs : dOs;
      bf16x8 xb[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int e = 0; e < 8; ++e) xb[hh][e] = f2bf(x[8 * hh + e]);
      auto tread = [&](int i) {  // i = 8 hh + ot
        const int hh = i >> 3, ot = i & 7;
        const bf16* tb = tt + 16 * hh * DH;
        // rows + 8 flip bit 1 of the row's swizzle group, i.e. chunk bit 1
        const int to = tofs[ot & 3] + (ot >> 2) * 128;
        const bf16x4 lo = ds_read_tr((const lds_bf16x4*)lds(tb + to));
        const bf16x4 hi = ds_read_tr((const lds_bf16x4*)lds(tb + ((to ^ 16) + 8 * DH)));
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      };
      bf16x8 tf[PF_T + 1];
#pragma unroll
      for (int i = 0; i < PF_T; ++i) tf[i] = tread(i);
#pragma unroll
      for (int i = 0; i < 2 * (DH / 32); ++i) {
        if (i + PF_T < 2 * (DH / 32)) tf[(i + PF_T) % (PF_T + 1)] = tread(i + PF_T);
        acc[i & 7] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tf[i % (PF_T + 1)], xb[i >> 3], acc[i & 7], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
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
    bf16* out = role ? a.dk + ((long)b * S + key) * a.lddk + (long)h * DH
                     : a.dv + ((long)b * S + key) * a.lddv + (long)h * DH;
    const float f = role ? a.f.scale : 1.f;
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        bf16x4 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = f2bf(acc[ot][4 * r4 + e] * f);
        *reinterpret_cast<bf16x4*>(out + 32 * ot + acc_row(4 * r4, g)) = y;
      }
  }
}


// ================================================================ backward, dQ
// Workgroup = 8 waves = 4 pairs; pair p owns queries q0 + 32 p .. + 31 of one
// (batch, head) and loops over 32-key blocks.  Wave p (role A) holds Q and
// forms P^T = exp2(S^T log2e - lse) from S^T = K Q^T; wave p + 4 (role B) holds
// dO, forms dP^T = V dO^T, takes P^T from its partner through LDS and
// accumulates dQ^T += K^T dS^T, dS^T = P^T (dP^T - delta).  Lanes own queries,
// so lse and delta are per-lane scalars.  K rows are read as row fragments and
// transposed (K^T) from the same dual-swizzled tile.  This kernel runs before
// the dK / dV kernel and also computes delta = rowsum(dO * O) for it.
//
// Four K / V stages (block j in stage j % 4, copied two blocks ahead) and two
// P^T exchange buffers (block j in buffer j % 2) leave one barrier per block:
// at barrier j, P^T of block j and the copies of block j + 1 are visible, and
// every wave has finished block j - 1, so the copies of block j + 2 issued
// after it overwrite block j - 2's stage and role A writes block j + 1's P^T
// over block j - 1's.  Role A can thus compute the next block's scores while
// role B accumulates the current block's dQ on the same SIMD.
constexpr int QPW = 128;   // queries per workgroup
constexpr int STG_Q = 2 * QT;  // K rows, V rows of a 32-key block
constexpr int NSTG_Q = 4;      // K / V stages
constexpr int XB = 4 * 16 * 64;  // floats of one P^T exchange buffer (4 pairs)

__global__ __launch_bounds__(NT8, 1) void attn256_bwd_dq_kernel(AttnBwdArgs a) {
  static_assert((NSTG_Q * STG_Q + 2 * XB * 2) * 2 <= 163840, "LDS budget");
  __shared__ __attribute__((aligned(1024))) bf16 smem[NSTG_Q * STG_Q + 2 * XB * 2];
  float* xbuf = reinterpret_cast<float*>(smem + NSTG_Q * STG_Q);
  const int S = a.f.S;
  const int nqb = (S + QPW - 1) / QPW;
  // one-dimensional grid, query blocks outermost, heaviest first
  const int BH = a.f.B * a.f.H;
  const int xb = (int)blockIdx.x / BH, bh = (int)blockIdx.x % BH;
  const int qb = a.f.causal ? (nqb - 1 - xb) : xb;
  const int b = bh / a.f.H, h = bh % a.f.H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int pair = wave & 3, role = wave >> 2;
  const int q0 = qb * QPW;
  const int pq0 = q0 + pair * 32;
  const int q = pq0 + (lane & 31);
  const long hs = ((long)b * a.f.H + h) * S;
  const bf16* Qb = a.f.q + (long)b * S * a.f.ldq + (long)h * DH;
  const bf16* Kb = a.f.k + (long)b * S * a.f.ldk + (long)h * DH;
  const bf16* Vb = a.f.v + (long)b * S * a.f.ldv + (long)h * DH;
  const bf16* dOb = a.dout + (long)b * S * a.lddo + (long)h * DH;
  const float sc = a.f.scale * LOG2E;

  bf16x8 rf[DH / 16];  // Q (role A) or dO (role B) of this lane's query
  {
    const bf16* base = role ? dOb : Qb;
    const long ld = role ? a.lddo : a.f.ldq;
    const __amdgpu_buffer_rsrc_t rq = rows_rsrc(base, pq0, ld);
    const uint32_t qo = q < S ? (uint32_t)(((long)(lane & 31) * ld + 8 * g) * 2) : OOB;
#pragma unroll
    for (int c = 0; c < DH / 16; ++c)
      rf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rq, qo, 32 * c, 0));
  }
  // role A: lse2 of this lane's query; role B: delta = rowsum(dO * O), from
  // the two halves of the row (lanes l and l + 32), also stored for the dK / dV
  // kernel, which runs after this one
  float lsd;
  if (role == 0) {
    lsd = q < S ? a.f.lse[hs + q] * LOG2E : 0.f;
  } else {
    const __amdgpu_buffer_rsrc_t ro = rows_rsrc(a.f.o + (long)b * S * a.f.ldo + (long)h * DH, pq0, a.f.ldo);
    const uint32_t oo = q < S ? (uint32_t)(((long)(lane & 31) * a.f.ldo + 8 * g) * 2) : OOB;
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < DH / 16; ++c) {
      const bf16x8 ov = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(ro, oo, 32 * c, 0));
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = __builtin_fmaf(bf2f(rf[c][e]), bf2f(ov[e]), acc);
    }
    lsd = halves_sum(acc);
    if (g == 0 && q < S) a.delta[hs + q] = lsd;
  }
  floatx16 acc[DH / 32];  // dQ^T (role B): dims 32 ot + acc_row(r, g), query = lane
#pragma unroll
  for (int t = 0; t < DH / 32; ++t) acc[t] = zero16();
  const int G = lane >> 4, ll = lane & 15;
  int tofs[4];
#pragma unroll
  for (int ot = 0; ot < 4; ++ot) {
    const int r = 4 * (G >> 1) + (ll >> 2);
    const int c = 4 * ot + 2 * (G & 1) + ((ll >> 1) & 1);
    tofs[ot] = r * DH + 8 * (c ^ swz_dual(r)) + 4 * (ll & 1);
  }

  const int kv_end = a.f.causal ? min(S, q0 + QPW) : S;
  const int nkb = (kv_end + BQ - 1) / BQ;
  auto stage_ptr = [&](int j) { return smem + (j % NSTG_Q) * STG_Q; };
  // four copy instructions per wave per block
  auto fetch = [&](int j) {
    const int kv = j * BQ;
    bf16* st = stage_ptr(j);
    copy_rows32(rows_rsrc(Kb, kv, a.f.ldk), a.f.ldk, S - kv, st, wave);
    copy_rows32(rows_rsrc(Vb, kv, a.f.ldv), a.f.ldv, S - kv, st + QT, wave);
  };

  fetch(0);
  if (nkb > 1) {
    fetch(1);
    wait_vm_lgkm0<4>();  // block 0 resident, block 1 may stay in flight
  } else {
    wait_vm_lgkm0<0>();
  }
  cta_barrier();

  for (int j = 0; j < nkb; ++j) {
    const int kv0 = j * BQ;
    const bf16* Ks = stage_ptr(j);
    const bf16* Vs = Ks + QT;
    float* xw = xbuf + (j & 1) * XB + pair * 16 * 64;
    const bool more2 = j + 2 < nkb;
    if (more2) fetch(j + 2);
    const bool active = !(a.f.causal && kv0 > pq0 + 31);
    floatx16 x = zero16();
    if (active) {
      const bf16* rows = role ? Vs : Ks;
      bf16x8 fr[PF_RQ + 1];
#pragma unroll
      for (int c = 0; c < PF_RQ; ++c) fr[c] = row_frag(rows, lane & 31, c, g);
#pragma unroll
      for (int c = 0; c < DH / 16; ++c) {
        if (c + PF_RQ < DH / 16) fr[(c + PF_RQ) % (PF_RQ + 1)] = row_frag(rows, lane & 31, c + PF_RQ, g);
        x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[c % (PF_RQ + 1)], rf[c], x, 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (role == 0) {
        // P^T = exp2(S^T log2e - lse2); zero for keys past S or (causal) past the query
        const int lim = min(S, a.f.causal ? q + 1 : S) - kv0 - 4 * g;  // keys with acc_row < lim valid
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kr = 8 * (r >> 2) + (r & 3);  // acc_row - 4 g
          float pr = __builtin_amdgcn_exp2f(x[r] * sc - lsd);
          pr = kr < lim ? pr : 0.f;
          xw[r * 64 + lane] = pr;
        }
      }
    }
    // own copies of block j + 1 landed (block j + 2's may stay in flight), P^T written
    if (more2) wait_vm_lgkm0<4>();
    else wait_vm_lgkm0<0>();
    cta_barrier();  // P^T of every pair and block j + 1 visible; block j - 1 done everywhere
    if (active && role == 1) {
#pragma unroll
      for (int r = 0; r < 16; ++r) x[r] = xw[r * 64 + lane] * (x[r] - lsd);
      bf16x8 xb[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int e = 0; e < 8; ++e) xb[hh][e] = f2bf(x[8 * hh + e]);
      auto tread = [&](int i) {  // i = 8 hh + ot
        const bf16* tb = Ks + 16 * (i >> 3) * DH;
        const int to = tofs[i & 3] + ((i & 7) >> 2) * 128;
        const bf16x4 lo = ds_read_tr((const lds_bf16x4*)lds(tb + to));
        const bf16x4 hi = ds_read_tr((const lds_bf16x4*)lds(tb + ((to ^ 16) + 8 * DH)));
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      };
#pragma unroll
      for (int i = 0; i < 2 * (DH / 32); ++i)
        acc[i & 7] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tread(i), xb[i >> 3], acc[i & 7], 0, 0, 0);
    }
  }
  if (role == 1 && q < S) {
    bf16* out = a.dq + ((long)b * S + q) * a.lddq + (long)h * DH;
#pragma unroll
    for (int ot = 0; ot < DH / 32; ++ot)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        bf16x4 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = f2bf(acc[ot][4 * r4 + e] * a.f.scale);
        *reinterpret_cast<bf16x4*>(out + 32 * ot + acc_row(4 * r4, g)) = y;
      }
  }
}

}  // namespace

bool attn256_fwd_eligible(const AttnArgs& a) {
  auto ok = [](const void* p, long ld) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 8 == 0; };
  return a.dh == DH && ok(a.q, a.ldq) && ok(a.k, a.ldk) && ok(a.v, a.ldv) &&
         (reinterpret_cast<uintptr_t>(a.o) & 7) == 0 && a.ldo % 4 == 0 &&
         (long)KB * a.ldk * 2 < (1L << 30) && (long)KB * a.ldv * 2 < (1L << 30);
}

bool attn256_bwd_eligible(const AttnBwdArgs& a) {
  auto ok = [](const void* p, long ld) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 8 == 0; };
  auto ok8 = [](const void* p, long ld) { return (reinterpret_cast<uintptr_t>(p) & 7) == 0 && ld % 4 == 0; };
  return attn256_fwd_eligible(a.f) && ok(a.dout, a.lddo) && ok8(a.dk, a.lddk) && ok8(a.dv, a.lddv) &&
         ok(a.f.o, a.f.ldo) && (long)QPW * a.f.ldo * 2 < (1L << 30) && a.delta != nullptr &&
         (long)KPW * a.f.ldk * 2 < (1L << 30) && (long)KPW * a.f.ldv * 2 < (1L << 30) &&
         (long)QPW * a.f.ldq * 2 < (1L << 30) && (long)QPW * a.lddo * 2 < (1L << 30) &&
         (reinterpret_cast<uintptr_t>(a.dq) & 7) == 0 && a.lddq % 4 == 0;
}

hipError_t launch_attn256_bwd_dkdv(const AttnBwdArgs& a, hipStream_t s) {
  dim3 grid((unsigned)(((a.f.S + KPW - 1) / KPW) * a.f.B * a.f.H));
  hipLaunchKernelGGL(attn256_bwd_dkdv_kernel, grid, dim3(NT8), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn256_bwd_dq(const AttnBwdArgs& a, hipStream_t s) {
  dim3 grid((unsigned)(((a.f.S + QPW - 1) / QPW) * a.f.B * a.f.H));
  hipLaunchKernelGGL(attn256_bwd_dq_kernel, grid, dim3(NT8), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn256_fwd(const AttnArgs& a, hipStream_t s) {
  dim3 grid((unsigned)(((a.S + QPB - 1) / QPB) * a.B * a.H));
  hipLaunchKernelGGL(attn256_fwd_kernel, grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}
