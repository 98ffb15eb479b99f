/* saturn_ops.h -- kernel-level C ABI of libsaturn.so.
 *
 * Each call enqueues one kernel of the fine-tuning step (the step that the
 * Saturn paper, arXiv 2309.01226, schedules for every model-selection task;
 * Sec. 3.1, Table 3) on `stream` (a hipStream_t, NULL = null stream) and
 * returns without waiting.  All tensor pointers are device pointers owned by
 * the caller; matrices are row-major with the given leading dimension (in
 * elements).  bf16 means IEEE bfloat16 storage (uint16).  The calls exist so
 * that every kernel can be checked and timed on its own; the model calls in
 * saturn.h use the same kernels.  Errors: SAT_EINVAL for bad sizes or null
 * pointers, SAT_EHIP when the launch fails.  Status codes as in saturn.h.
 */
#ifndef SATURN_OPS_H
#define SATURN_OPS_H

#include <stdint.h>

#include "saturn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Dense contraction C[m, n] = sum_k A(m, k) B(n, k) (bf16 operands, fp32
 * accumulation), the forward, input-gradient and weight-gradient products of
 * every linear layer.  Layout 0: A(m, k) = A[m*lda + k], B(n, k) = B[n*ldb + k];
 * layout 1: A(m, k) = A[k*lda + m], B(n, k) = B[k*ldb + n].
 * Epilogue 0: fp32 out = C + bias.  1: fp32 out = resid + C + bias (resid may
 * equal out).  2: bf16 out = C + bias, and, when out2 != NULL, bf16
 * out2[m, n - gelu_col0] = GELU(C + bias) for n >= gelu_col0.  3: bf16 out =
 * C * GELU'(aux[m, n]).  bias (fp32, may be NULL) applies to columns
 * n >= bias_col0 as bias[n - bias_col0].  gelu_erf: 0 tanh form, 1 erf form.
 * splitk_ws (fp32 device scratch of splitk_ws_elems elements, may be NULL):
 * with it, an epilogue-0/1 product on layout-0 operands that has fewer than
 * 256 output tiles of 256 x 256 and K >= 1024 runs split-K: K slices of at
 * least 512 write fp32 partials there, then one reduction adds them in slice
 * order with bias and residual.  Such a product with more than 256 tiles
 * whose last round of 256 tiles would run mostly empty instead runs its
 * first rows (whole rounds) unsplit and only the remaining rows split-K,
 * when that is estimated faster.  Results then differ from the unsplit
 * product by summation order only.  The scratch is used only when it holds
 * slices * (split rows) * N elements; the call makes no allocation. */
typedef struct {
  const void* A;
  const void* B;
  int32_t M, N, K;
  int64_t lda, ldb;
  int32_t a_layout, b_layout, epilogue;
  void* out;
  int64_t ldo;
  const float* bias;
  int32_t bias_col0;
  const float* resid;
  int64_t ldr;
  void* out2;
  int64_t ldo2;
  int32_t gelu_col0;
  const void* aux;
  int64_t ldaux;
  int32_t gelu_erf;
  float* splitk_ws;
  int64_t splitk_ws_elems;
} sat_gemm_desc;
sat_status sat_op_gemm(const sat_gemm_desc* d, void* stream);

/* sat_op_gemm for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops and harnesses that forbid hipMalloc.
 * Same descriptor and result as sat_op_gemm given a workspace large enough
 * for the product's split-K plan, except that d->splitk_ws must be NULL and
 * d->splitk_ws_elems 0: the split-K partials go to a scratch array of
 * SAT_GEMM_NOALLOC_WS_ELEMS fp32 elements (32 MiB) that the library holds on
 * every device it runs on until the process ends.  The call allocates
 * nothing.  A product whose split-K partials would exceed the scratch is
 * rejected with SAT_EINVAL before any launch, except one that would split
 * only the rows of its last round: that runs unsplit, with the result of
 * sat_op_gemm without a workspace.  All calls on one device share
 * that device's scratch: calls whose products split K and that may overlap
 * (different streams, or different host threads) race and must be ordered
 * by the caller. */
#define SAT_GEMM_NOALLOC_WS_ELEMS (8L * 1024 * 1024)
sat_status sat_op_gemm_noalloc(const sat_gemm_desc* d, void* stream);

/* LayerNorm forward over `rows` rows of length d: x fp32 (row r at
 * x + r*row_stride*ldx), y bf16 [rows, ldy], mean / rstd fp32 [rows]. */
sat_status sat_op_layernorm_fwd(const float* x, int64_t ldx, int64_t row_stride, const float* g,
                                const float* b, void* y, int64_t ldy, float* mean, float* rstd,
                                int32_t rows, int32_t d, float eps, void* stream);
/* LayerNorm backward: dres[r] += dx[r] (fp32, same row addressing as x);
 * dg, db fp32 [d] (overwritten).  work: fp32 scratch of 2*n_part*d floats,
 * n_part = min(rows, 1024). */
sat_status sat_op_layernorm_bwd(const float* dy, int64_t lddy, const float* x, int64_t ldx,
                                int64_t row_stride, const float* g, const float* mean,
                                const float* rstd, float* dres, int64_t ldres, float* dg,
                                float* db, float* work, int32_t rows, int32_t d, void* stream);

/* Flash-style attention forward.  q, k, v, o: bf16, element (b, h, s, j) at
 * ptr[(b*S + s)*ld + h*dh + j].  lse: fp32 [B, H, S] natural-log
 * log-sum-exp of the scaled scores.  scale multiplies q.k.  dh is one of 16,
 * 32, 64, 80, 128, 256; for 64, 80 and 256, q, k, v must be 16-byte aligned
 * with ld % 8 == 0, o 8-byte aligned with ldo % 4 == 0 and scale > 0
 * (SAT_EINVAL otherwise). */
sat_status sat_op_attention_fwd(const void* q, const void* k, const void* v, int64_t ldq,
                                int64_t ldk, int64_t ldv, void* o, int64_t ldo, float* lse,
                                int32_t B, int32_t H, int32_t S, int32_t dh, int32_t causal,
                                float scale, void* stream);
/* Attention backward from dO (bf16, addressed like o), the forward's o and
 * lse; writes dq, dk, dv (bf16, addressed like q, k, v).  delta: fp32
 * [B, H, S] scratch.  Head dims and alignment as for the forward; for 64, 80
 * and 256, o and dout must also be 16-byte aligned with ld % 8 == 0 and dq,
 * dk, dv 8-byte aligned with ld % 4 == 0. */
sat_status sat_op_attention_bwd(const void* q, const void* k, const void* v, int64_t ldq,
                                int64_t ldk, int64_t ldv, const void* o, int64_t ldo,
                                const float* lse, const void* dout, int64_t lddo, float* delta,
                                void* dq, void* dk, void* dv, int64_t lddq, int64_t lddk,
                                int64_t lddv, int32_t B, int32_t H, int32_t S, int32_t dh,
                                int32_t causal, float scale, void* stream);

/* Rotary on interleaved pairs of the first rd dims of every q and k head, in
 * place; qk bf16 [B*S, ld] with q at column 0 and k at column H*dh.
 * inverse = 1 applies the transpose rotation (backward).  ld and dh even, qk
 * 4-byte aligned (SAT_EINVAL otherwise). */
sat_status sat_op_rotary(void* qk, int64_t ld, int32_t B, int32_t S, int32_t H, int32_t dh,
                         int32_t rd, int32_t inverse, void* stream);

/* Softmax cross-entropy forward + backward over fp32 logits z [N, ldz]:
 * row_loss fp32 [N] (0 for label -1), dz bf16 [N, lddz] = (softmax - onehot)
 * * inv_n (0 rows for label -1), where inv_n = 1 / (number of labels != -1). */
sat_status sat_op_cross_entropy(const float* z, int64_t ldz, const int32_t* labels, int32_t N,
                                int32_t V, float* row_loss, void* dz, int64_t lddz, float* inv_n,
                                void* stream);

/* Fused AdamW over n fp32 values (torch semantics, decoupled decay) at step t
 * (t >= 1); refreshes the bf16 shadow when shadow != NULL. */
sat_status sat_op_adamw(float* p, const float* g, float* m, float* v, void* shadow, int64_t n,
                        double lr, double beta1, double beta2, double eps, double wd, int64_t t,
                        void* stream);

/* Token embedding forward h[t] = wte[tok[t]] (+ wpe[t % S]) and its
 * deterministic backward dwte[v] = sum over t with tok[t] == v of dh[t] in
 * increasing t, written for every v < V (zero rows for absent tokens).  Past
 * 16384 positions the sum is formed per chunk of 16384 positions, in order,
 * and the chunks' sums are added in order.
 * work: int32 scratch of min(T, 16384) entries.  Backward limit: V < 65536
 * (SAT_EINVAL otherwise). */
sat_status sat_op_embed_fwd(const int32_t* tok, const float* wte, const float* wpe, float* h,
                            int32_t T, int32_t S, int32_t d, int32_t V, void* stream);
sat_status sat_op_embed_bwd(const int32_t* tok, const float* dh, float* dwte, int32_t T,
                            int32_t d, int32_t V, int32_t* work, void* stream);

/* Column sum out[c] = sum_r X[r, c] of an fp32 [rows, ldx] matrix,
 * deterministic; work: fp32 scratch of min(rows, 256) * cols floats. */
sat_status sat_op_colsum(const float* X, int64_t ldx, int32_t rows, int32_t cols, float* out,
                         float* work, void* stream);

/* Transpose of a bf16 matrix: dst[c * ldd + r] = src[r * lds + c] for
 * r < rows, c < cols.  rows, cols, lds and ldd are multiples of 8 with
 * lds >= cols, ldd >= rows; both pointers device memory, 16-byte aligned
 * (SAT_EINVAL otherwise).  The runtime keeps transposed bf16 copies of the
 * weights for the input-gradient products dX = dY W (each a product over the
 * contiguous index of both operands). */
sat_status sat_op_transpose_bf16(const void* src, int64_t lds, void* dst, int64_t ldd,
                                 int32_t rows, int32_t cols, void* stream);

/* ---- the ResNet workload's own kernels (Table 3: the ResNet fine-tuned on
 * ImageNet-shaped images).  Activations are NHWC: [N, H, W, C] is the
 * row-major matrix [N * H * W, C]; Ho = (H + 2 pad - k) / stride + 1.
 *
 * im2col: col [N * Ho * Wo, k * k * C] bf16, col[(n Ho + i) Wo + j,
 * (a k + b) C + c] = x[n, i stride - pad + a, j stride - pad + b, c] (zero
 * outside the image), from x bf16; C a positive multiple of 8.  The operand of
 * a k x k convolution computed as one GEMM against the weight [Cout, k k C]. */
sat_status sat_op_im2col(const void* x, void* col, int32_t N, int32_t H, int32_t W, int32_t C,
                         int32_t k, int32_t stride, int32_t pad, void* stream);
/* The same matrix transposed: colT [k * k * C, N * Ho * Wo] bf16 with row
 * stride ldt (>= N Ho Wo, a multiple of 8), the token-contiguous operand of a
 * convolution's weight-gradient product.  N Ho Wo % 8 == 0, C % 8 == 0, x and
 * colT 16-byte aligned (SAT_EINVAL otherwise). */
sat_status sat_op_im2col_t(const void* x, void* colT, int64_t ldt, int32_t N, int32_t H, int32_t W,
                           int32_t C, int32_t k, int32_t stride, int32_t pad, void* stream);
/* col2im, the transpose of im2col: dx [N, H, W, C] fp32 = (accumulate: dx +)
 * the sum over the taps that read each input element of dcol [N * Ho * Wo,
 * k * k * C] fp32, in tap order; C a positive multiple of 4. */
sat_status sat_op_col2im(const float* dcol, float* dx, int32_t N, int32_t H, int32_t W, int32_t C,
                         int32_t k, int32_t stride, int32_t pad, int32_t accumulate, void* stream);
/* Batch norm in training mode over x [P, C] fp32 (statistics of the P rows,
 * biased variance): mean, rstd = 1 / sqrt(var + eps) [C]; y = (x - mean) rstd
 * g + b, with ReLU when relu, as bf16 (y, may be NULL) and fp32 (yf, may be
 * NULL, not both).  part: fp32 scratch of 2 * 1024 * C.  C % 4 == 0; every
 * fp32 array 16-byte aligned, y 8-byte aligned (SAT_EINVAL otherwise). */
sat_status sat_op_batchnorm_fwd(const float* x, int64_t P, int32_t C, const float* g,
                                const float* b, float eps, int32_t relu, float* part, float* mean,
                                float* rstd, void* y, float* yf, void* stream);
/* Its backward from dy [P, C] fp32, through a ReLU when mask_kind is 1 (dy
 * where the bf16 mask > 0) or 2 (fp32 mask > 0): dg = sum g' xhat, db = sum
 * g' (written), dx = rstd g (g' - db / P - xhat dg / P) as bf16.  Alignment as
 * for the forward (an fp32 mask 16-byte, a bf16 mask and dx 8-byte). */
sat_status sat_op_batchnorm_bwd(const float* dy, int32_t mask_kind, const void* mask,
                                const float* x, const float* mean, const float* rstd,
                                const float* g, int64_t P, int32_t C, float* part, float* dg,
                                float* db, void* dx, void* stream);
/* 3 x 3 max pool, stride 2, padding 1: y fp32, yb bf16 and the winning tap
 * arg (row-major index 0..8, the first maximum) [N, Ho, Wo, C]; the backward
 * routes dy to the winning taps: dx [N, H, W, C] fp32. */
sat_status sat_op_maxpool_fwd(const float* x, int32_t N, int32_t H, int32_t W, int32_t C, float* y,
                              void* yb, uint8_t* arg, void* stream);
sat_status sat_op_maxpool_bwd(const float* dy, const uint8_t* arg, int32_t N, int32_t H, int32_t W,
                              int32_t C, float* dx, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* SATURN_OPS_H */
