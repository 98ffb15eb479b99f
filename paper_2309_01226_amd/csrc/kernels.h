// Host-side launchers of the gfx950 kernels.  Every launcher enqueues work on
// the given stream and returns hipSuccess or the launch error; none of them
// synchronises or allocates.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;

// ---------------------------------------------------------------- AdamW constants
// The scalar constants are formed on the host in double precision:
//   p <- p - lr_wd * p;  m <- b1 m + omb1 g;  v <- b2 v + omb2 g^2;
//   p <- p - step * m / (sqrt(v) / bc2s + eps)
// with lr_wd = lr * wd, omb = 1 - beta, step = lr / (1 - beta1^t),
// bc2s = sqrt(1 - beta2^t).
struct AdamWConsts {
  float lr_wd, b1, omb1, b2, omb2, step, bc2s, eps;
};

// ---------------------------------------------------------------- GEMM
// C[m, n] = sum_k A(m, k) * B(n, k) on bf16 operands, fp32 accumulation.
//   A layout 0: A(m, k) = A[m * lda + k]      layout 1: A(m, k) = A[k * lda + m]
//   B layout 0: B(n, k) = B[n * ldb + k]      layout 1: B(n, k) = B[k * ldb + n]
enum GemmLayout { LAY_K = 0, LAY_MN = 1 };
enum GemmEpilogue {
  EPI_F32 = 0,        // out_f32[m, n] = C + bias
  EPI_RESID_F32 = 1,  // out_f32[m, n] = resid[m, n] + C + bias   (resid may alias out)
  EPI_BF16 = 2,       // out_bf16[m, n] = C + bias; and out2[m, n - gelu_col0] = GELU(C + bias)
  EPI_DGELU_BF16 = 3, // out_bf16[m, n] = C * GELU'(aux[m, n])
  EPI_ADAMW = 4,      // C is the gradient of a weight: one AdamW step on it (opt_* below)
};

struct GemmArgs {
  const bf16* A;
  const bf16* B;
  int M, N, K;
  long lda, ldb;
  void* out;
  long ldo;
  const float* bias;  // bias[n - bias_col0] added for n >= bias_col0; null = none
  int bias_col0;
  const float* resid;
  long ldr;
  bf16* out2;         // EPI_BF16: GELU outputs for n >= gelu_col0; null = none
  long ldo2;
  int gelu_col0;
  const bf16* aux;    // EPI_DGELU_BF16: GELU pre-activation
  long ldaux;
  int gelu_erf;       // 0 = tanh form, 1 = erf form
  // EPI_ADAMW: C[m, n] is the gradient of the weight W [M, N] (row pitch N)
  // whose fp32 master values, moments and bf16 copy start at opt_p, opt_m,
  // opt_v, opt_sh.  The epilogue applies one AdamW step (opt_c) to W, writes
  // the updated bf16 values there and, transposed, at opt_sht[n * opt_trows +
  // m] (rows M .. opt_trows - 1 of that copy as zeros), and writes C itself
  // as fp32 to out (pitch ldo) only when out is not null.
  float* opt_p;
  float* opt_m;
  float* opt_v;
  bf16* opt_sh;
  bf16* opt_sht;
  long opt_trows;
  AdamWConsts opt_c;
  // Split-K (256 x 256 kernel, EPI_F32, both operands K-contiguous, no bias):
  // splitk > 1 cuts K into slices of splitk_kc (a multiple of 64); slice s
  // writes its fp32 partial product to out + s * split_stride.
  int splitk;
  int splitk_kc;
  long split_stride;
  // Optional caller-owned fp32 workspace of splitk_ws_elems elements; with it,
  // launch_gemm runs fp32-output products that have too few 256 x 256 tiles
  // to fill the chip as split-K plus a reduction (gemm_splitk below).
  float* splitk_ws;
  long splitk_ws_elems;
  // Most K slices the split-K plan may use (0: 16).  Products with very few
  // output tiles and very long K (the convolution weight gradients, K =
  // pixels) fill the chip only with more.
  int splitk_max;
  // EPI_DGELU_BF16 in the 256 x 256 kernel: when not null, also the column
  // sums of the bf16 results over each block of 128 rows, block b at
  // colsum_part[b * N + n] (cdiv(M, 128) rows; launch_colsum_partials then
  // adds them in order).  Needs gemm256_eligible to hold with it set.
  float* colsum_part;
  // Keeps launch_gemm from splitting the rows of a mostly empty last round
  // (gemm_tail_split): a weight gradient whose AdamW step may instead be
  // fused into this kernel's epilogue must sum in the same order either way.
  int no_tail_split;
};

hipError_t launch_gemm(const GemmArgs& a, int alay, int blay, int epi, hipStream_t s);
// The 256 x 256 four-stage kernel (gemm256.hip) for large aligned problems;
// launch_gemm dispatches to it when gemm256_eligible holds.
bool gemm256_eligible(const GemmArgs& a, int alay, int blay, int epi);
hipError_t launch_gemm256(const GemmArgs& a, int alay, int blay, int epi, hipStream_t s);
// K slices launch_gemm uses for an fp32-output [M, N] product of depth K when
// a workspace is given (1: none; *kc: slice depth), and the workspace that
// then takes (fp32 elements; 0 when not split).  A product is split when it
// has fewer than 256 tiles of 256 x 256 and K >= 1024: into enough slices to
// give every CU a tile where K allows, each at least 512 deep, at most smax.
int gemm_splitk(int M, int N, int K, int* kc, int smax = 16);
long gemm_splitk_ws_elems(int M, int N, int K, int smax = 16);
// An fp32-output product with more than 256 tiles whose last round of 256
// workgroups would run mostly empty: the first *M1 rows (whole rounds) run
// unsplit, the remaining rows as *S K slices of depth *kc plus a reduction,
// when the same estimate as gemm_splitk says that is faster.  launch_gemm
// takes this plan when the workspace holds S * (M - M1) * N elements (the
// figure gemm_tail_ws_elems gives; 0 when the plan does not apply).
bool gemm_tail_split(int M, int N, int K, int smax, int* M1, int* S, int* kc);
long gemm_tail_ws_elems(int M, int N, int K, int smax = 16);
// out[m, n] = sum over s of ws[s * stride + m * N + n] (s in order) + bias[n -
// bias_col0] (n >= bias_col0; null: none) + resid[m * ldr + n] (null: none).
hipError_t launch_splitk_reduce(const float* ws, int S, long stride, int M, int N, float* out,
                                long ldo, const float* bias, int bias_col0, const float* resid,
                                long ldr, hipStream_t s);

// ---------------------------------------------------------------- LayerNorm
// y = (x - mean) * rstd * g + b over rows of length d; x fp32, y bf16.
// mean / rstd saved per row (fp32).  Row r of x is x + rows_idx(r) * ldx where
// rows_idx(r) = r * row_stride (row_stride lets the ViT head pick CLS rows).
hipError_t launch_layernorm_fwd(const float* x, long ldx, long row_stride, const float* g,
                                const float* b, bf16* y, long ldy, float* mean, float* rstd,
                                int rows, int d, float eps, hipStream_t s);
// dx = rstd * (gy - mean(gy) - xhat * mean(gy * xhat)), gy = dy * g; written as
// dres[r] += dx (fp32 residual gradient, row stride as in the forward).
// Per-row partials of dg / db go to part_g / part_b [n_part, d] and are then
// reduced by launch_colsum_partials (deterministic, no atomics).
hipError_t launch_layernorm_bwd(const float* dy, long lddy, const float* x, long ldx,
                                long row_stride, const float* g, const float* mean,
                                const float* rstd, float* dres, long ldres, float* part_g,
                                float* part_b, int rows, int d, int n_part, hipStream_t s,
                                bf16* dres_bf = nullptr, long ldbf = 0, float* part_o = nullptr);
// dres_bf (row_stride 1 only; null: none): also writes the updated dres rows
// rounded to bf16 at dres_bf + r * ldbf.  part_o (null: none): a third array
// of n_part partial rows, the column sums of the updated dres.
// Partial-sum rows (workgroups) the LayerNorm backward uses for `rows` rows
// of d: the dg / db partials take 2 * ln_bwd_parts(rows, d) * d floats (at
// most 2 * min(rows, 1024) * d).
int ln_bwd_parts(int rows, int d);
hipError_t launch_colsum_partials(const float* part, int n_part, int d, float* out,
                                  hipStream_t s);
// dg = colsum of part[0 : n_part], db = colsum of part[n_part : 2 n_part]
// (rows of d), and with dbias also dbias = colsum of part[2 n_part : 3 n_part],
// one launch.
hipError_t launch_ln_bwd_colsums(const float* part, int n_part, int d, float* dg, float* db,
                                 hipStream_t s, float* dbias = nullptr);
// out[c] = sum_r X[r, c] for a bf16 or fp32 matrix, deterministic two-pass.
hipError_t launch_colsum_bf16(const bf16* X, long ldx, int rows, int cols, float* part,
                              int n_part, float* out, hipStream_t s);
hipError_t launch_colsum_f32(const float* X, long ldx, int rows, int cols, float* part,
                             int n_part, float* out, hipStream_t s);

// ---------------------------------------------------------------- attention
struct AttnArgs {
  const bf16* q;   // q(b, h, s, :) = q[(b * S + s) * ldq + h * dh]
  const bf16* k;
  const bf16* v;
  long ldq, ldk, ldv;
  bf16* o;         // o(b, h, s, :) = o[(b * S + s) * ldo + h * dh]
  long ldo;
  float* lse;      // [B, H, S] log-sum-exp of the scaled scores (natural log)
  int B, H, S, dh;
  int causal;
  float scale;
};
struct AttnBwdArgs {
  AttnArgs f;
  const bf16* dout;  long lddo;
  float* delta;      // [B, H, S] rowsum(dO * O)
  bf16* dq; bf16* dk; bf16* dv;
  long lddq, lddk, lddv;
};
hipError_t launch_attention_fwd(const AttnArgs& a, hipStream_t s);
// 256-wide heads (attn256.hip); launch_attention_fwd dispatches to it.
bool attn256_fwd_eligible(const AttnArgs& a);
hipError_t launch_attn256_fwd(const AttnArgs& a, hipStream_t s);
hipError_t launch_attention_bwd(const AttnBwdArgs& a, hipStream_t s);
// 256-wide heads (attn256.hip): the dK / dV and dQ kernels; launch_attention_bwd
// dispatches to them after computing delta.
bool attn256_bwd_eligible(const AttnBwdArgs& a);
hipError_t launch_attn256_bwd_dkdv(const AttnBwdArgs& a, hipStream_t s);
hipError_t launch_attn256_bwd_dq(const AttnBwdArgs& a, hipStream_t s);
// 64- and 80-wide heads (attn_small.hip): forward, and dK / dV then dQ after
// launch_attention_bwd has computed delta.
bool attn_small_fwd_eligible(const AttnArgs& a);
bool attn_small_bwd_eligible(const AttnBwdArgs& a);
hipError_t launch_attn_small_fwd(const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_small_bwd(const AttnBwdArgs& a, hipStream_t s);

// ---------------------------------------------------------------- elementwise
// GPT-J rotary on interleaved pairs of the first rd dims of every q and k head,
// in place on the bf16 [T, ld] buffer (q at column 0, k at column d).  cs: the
// table of launch_rope_table for this S and rd, or null to compute the angles
// inline (same values).
hipError_t launch_rotary(bf16* qk, long ld, int B, int S, int H, int dh, int rd, int inverse,
                         hipStream_t s, const float2* cs = nullptr);
// cs[pos * (rd / 2) + i] = (cos, sin) of pos * 10000^(-2i/rd), pos < S.
hipError_t launch_rope_table(float2* cs, int S, int rd, hipStream_t s);
// h0[t, :] = wte[tok[t], :] (+ wpe[t % S, :])
hipError_t launch_embed_fwd(const int32_t* tok, const float* wte, const float* wpe, float* h,
                            int T, int S, int d, int V, hipStream_t s);
// dwte[v, :] = sum over t with tok[t] == v of dh[t, :], in increasing t (deterministic).
// Sorts (token, position) keys in `work` (int32, >= T entries); T <= 16384, V < 65536.
hipError_t launch_embed_bwd(const int32_t* tok, const float* dh, float* dwte, int T, int d,
                            int V, int32_t* work, hipStream_t s);
// ViT: images [B, C, I, I] fp32 -> patches [B * np, C * p * p] bf16, (c, kh, kw) order.
hipError_t launch_patchify(const float* img, bf16* out, int B, int C, int I, int p, int ldo,
                           hipStream_t s);
// ViT: h[b, 0] = cls + pos[0]; h[b, 1 + i] = z[b * np + i] + pos[1 + i]  (z holds bias).
hipError_t launch_vit_assemble(const float* z, const float* cls, const float* pos, float* h,
                               int B, int np, int d, hipStream_t s);
// ViT backward: dz[b * np + i, :] = bf16(dh[b * (np + 1) + 1 + i, :])
hipError_t launch_vit_patch_grad(const float* dh, bf16* dz, int B, int np, int d, hipStream_t s);
// fp32 -> bf16 copy of a strided matrix (rows x cols)
hipError_t launch_f32_to_bf16(const float* x, long ldx, bf16* y, long ldy, int rows, int cols,
                              hipStream_t s);
// dst[c, r] = src[r, c], bf16; rows, cols, strides multiples of 8, 16-byte
// aligned pointers (hipErrorInvalidValue otherwise).
hipError_t launch_transpose_bf16(const bf16* src, long lds, bf16* dst, long ldd, int rows,
                                int cols, hipStream_t s);
// Cross-entropy fwd+bwd over fp32 logits [N, V]: per-row loss (0 for ignored
// rows), dz = (softmax - onehot) * inv_n as bf16, count of valid rows.
// inv_n: device pointer to 1 / (number of labels != -1).
hipError_t launch_xent(const float* z, long ldz, const int32_t* labels, int N, int V,
                       float* row_loss, bf16* dz, long lddz, const float* inv_n, hipStream_t s);
// out[0] = inv_n[0] * sum of row_loss[0..n), summed in a fixed order.
hipError_t launch_loss_finalize(const float* row_loss, int n, const float* inv_n, float* out,
                                hipStream_t s);
// inv_n[0] = 1 / max(1, number of labels >= 0)
hipError_t launch_count_valid(const int32_t* labels, int n, float* inv_n, hipStream_t s);
// Synthetic profiling batches from a hash of (seed, index): tokens x [B, S]
// uniform in [0, V) with y the next token of the same stream; images of n
// values uniform in [-1, 1) with labels y [B] uniform in [0, classes).
hipError_t launch_synth_tokens(int32_t* x, int32_t* y, int B, int S, int V, uint32_t seed,
                               hipStream_t s);
hipError_t launch_synth_images(float* img, long n, int32_t* y, int B, int classes, uint32_t seed,
                               hipStream_t s);
// Fused AdamW over n contiguous fp32 parameters with bf16 shadow refresh.
AdamWConsts adamw_consts(double lr, double beta1, double beta2, double eps, double wd, long t);
hipError_t launch_adamw(float* p, const float* g, float* m, float* v, bf16* shadow, long n,
                        const AdamWConsts& c, hipStream_t s);
// One piece of the trainable parameters for the segmented AdamW below.
// Flat segment (toff < 0): n = rows elements at off.  Matrix segment: the
// [rows, cols] row-major matrix at off, updated in 64 x 64 tiles whose bf16
// values are also written transposed, shadow_t[toff + c * trows + r]; rows
// rows .. trows - 1 of the transposed copy are written as zeros.
// first_block: index of the segment's first workgroup (64 x 64 tiles, or
// chunks of 8192 elements); the table is sorted by it.
struct AdamWSeg {
  int64_t off, toff;
  int32_t rows, trows, cols, first_block;
};
constexpr int kAdamWChunk = 8192;
int adamw_seg_blocks(const AdamWSeg& g);
// Runs over nseg segments (device table) with total_blocks workgroups.
hipError_t launch_adamw_segments(float* p, const float* g, float* m, float* v, bf16* shadow,
                                 bf16* shadow_t, const AdamWSeg* segs, int nseg,
                                 int total_blocks, const AdamWConsts& c, hipStream_t s);
// Counter-based N(0, std^2) init of n fp32 values (Philox-style hash of
// (seed, tensor id, index) fed to Box-Muller); also writes the bf16 shadow.
hipError_t launch_init_normal(float* p, bf16* shadow, long n, uint64_t seed, uint32_t stream_id,
                              float std, hipStream_t s);
hipError_t launch_fill(float* p, bf16* shadow, long n, float value, hipStream_t s);
hipError_t launch_zero(void* p, long bytes, hipStream_t s);
hipError_t launch_sum_rows_batched(const float* dh, float* out, int B, int S, int d,
                                   hipStream_t s);

// ---------------------------------------------------------------- ResNet (conv.hip)
// NHWC activations ([N, H, W, C] = the matrix [N * H * W, C]).
// col[(n Ho + i) Wo + j, (a k + b) C + c] = x[n, i s - pad + a, j s - pad + b, c]
// (zero outside); bf16, C % 8 == 0, ldc == k k C.
hipError_t launch_im2col(const bf16* x, bf16* col, long ldc, int N, int H, int W, int C, int k,
                         int s, int pad, int Ho, int Wo, hipStream_t st);
// The same matrix transposed, colT [k k C, N Ho Wo] (row stride ldt): the
// token-contiguous operand of a convolution's weight-gradient product.
// C % 8 == 0, N Ho Wo % 8 == 0, ldt % 8 == 0, 16-byte aligned.
hipError_t launch_im2col_t(const bf16* x, bf16* colT, long ldt, int N, int H, int W, int C, int k,
                           int s, int pad, int Ho, int Wo, hipStream_t st);
// The same from fp32 NCHW images; columns k k C .. ldc - 1 are written as zeros.
hipError_t launch_im2col_nchw(const float* img, bf16* col, long ldc, int N, int C, int H, int W,
                              int k, int s, int pad, int Ho, int Wo, hipStream_t st);
// dx (+)= the sum over taps of dcol (the transpose of im2col, gathered per
// input element in tap order); fp32, C % 4 == 0.
hipError_t launch_col2im(const float* dcol, long ldc, float* dx, int N, int H, int W, int C, int k,
                         int s, int pad, int Ho, int Wo, int accumulate, hipStream_t st);
// Batch-norm statistics of x [P, C] per channel (training mode, biased
// variance): mean, rstd = 1 / sqrt(var + eps).  part: fp32 scratch of
// 2 * bn_parts(P, C) * C.
int bn_parts(long P, int C);
hipError_t launch_bn_stats(const float* x, long P, int C, float eps, float* part, float* mean,
                           float* rstd, hipStream_t st);
// y = (x - mean) rstd g + b (ReLU when relu) as bf16 (y, may be null) and fp32 (yf, may be null).
hipError_t launch_bn_apply(const float* x, long P, int C, const float* mean, const float* rstd,
                           const float* g, const float* b, int relu, bf16* y, float* yf,
                           hipStream_t st);
// out = ReLU(BN_a(xa) + BN_s(xs)) (ms null: + xs itself), fp32 and bf16.
hipError_t launch_bn_add_relu(const float* xa, const float* ma, const float* ra, const float* ga,
                              const float* ba, const float* xs, const float* ms, const float* rs,
                              const float* gs, const float* bs, long P, int C, float* out,
                              bf16* outb, hipStream_t st);
// Batch-norm backward with g = dy (mask_kind 0), dy where the bf16 mask > 0
// (1) or where the fp32 mask > 0 (2): dg = sum g xhat, db = sum g (written),
// dx = rstd gamma (g - db / P - xhat dg / P) as bf16.  part as for the stats.
hipError_t launch_bn_bwd(const float* dy, int mask_kind, const void* mask, const float* x,
                         const float* mean, const float* rstd, const float* gam, long P, int C,
                         float* part, float* dg, float* db, bf16* dx, hipStream_t st);
// dz = dy where out > 0, else 0 (n % 4 == 0).
hipError_t launch_relu_mask(const float* dy, const float* out, long n, float* dz, hipStream_t st);
// 3 x 3 max pool, stride 2, padding 1: fp32 / bf16 outputs and the winning
// tap (row-major index, first maximum); backward gathers dy by that tap.
hipError_t launch_maxpool_fwd(const float* x, int N, int H, int W, int C, int Ho, int Wo, float* y,
                              bf16* yb, uint8_t* arg, hipStream_t st);
hipError_t launch_maxpool_bwd(const float* dy, const uint8_t* arg, int N, int H, int W, int C,
                              int Ho, int Wo, float* dx, hipStream_t st);
// Global average pool over the HW rows of each image (bf16 features) and its backward.
hipError_t launch_avgpool_fwd(const float* x, int N, int HW, int C, bf16* feat, hipStream_t st);
hipError_t launch_avgpool_bwd(const float* dfeat, int N, int HW, int C, float* dx, hipStream_t st);
// dx[n, 2i, 2j] += dsub[n, i, j]: input gradient of a stride-2 1 x 1 convolution.
hipError_t launch_stride2_add(const float* dsub, int N, int Ho, int Wo, int C, int H, int W,
                              float* dx, hipStream_t st);
// Copy of a bf16 matrix [rows, cols] into [rows, ldd] with zero columns cols .. ldd - 1.
hipError_t launch_pad_cols_bf16(const bf16* src, int rows, int cols, bf16* dst, long ldd,
                                hipStream_t st);
