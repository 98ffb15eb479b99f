// Kernel-level C ABI (include/saturn_ops.h): argument checks, then one launch.
#include <algorithm>
#include <math.h>
#include <string.h>

#include <mutex>
#include <string>

#include "../../include/saturn_ops.h"
#include "abi_common.h"
#include "kernels.h"

static thread_local std::string g_last_error;

void sat_set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

extern "C" const char* sat_last_error(void) { return g_last_error.c_str(); }

static inline hipStream_t S(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Checks a descriptor and fills the launch arguments (everything but the
// split-K workspace).
static sat_status gemm_args(const sat_gemm_desc* d, GemmArgs* out, const char* fn) {
  SAT_CHECK_ARG(d != nullptr, "%s: null descriptor", fn);
  SAT_CHECK_ARG(d->A && d->B && d->out, "%s: null operand", fn);
  SAT_CHECK_ARG(d->M >= 0 && d->N >= 0 && d->K > 0, "%s: bad sizes M=%d N=%d K=%d", fn, d->M,
                d->N, d->K);
  SAT_CHECK_ARG(d->a_layout == 0 || d->a_layout == 1, "%s: bad a_layout", fn);
  SAT_CHECK_ARG(d->b_layout == 0 || d->b_layout == 1, "%s: bad b_layout", fn);
  SAT_CHECK_ARG(d->epilogue >= 0 && d->epilogue <= 3, "%s: bad epilogue", fn);
  SAT_CHECK_ARG(d->lda >= (d->a_layout == 0 ? d->K : d->M), "%s: lda too small", fn);
  SAT_CHECK_ARG(d->ldb >= (d->b_layout == 0 ? d->K : d->N), "%s: ldb too small", fn);
  SAT_CHECK_ARG(d->ldo >= d->N, "%s: ldo too small", fn);
  SAT_CHECK_ARG(d->epilogue != 1 || (d->resid && d->ldr >= d->N), "%s: resid", fn);
  SAT_CHECK_ARG(d->epilogue != 3 || (d->aux && d->ldaux >= d->N), "%s: aux", fn);
  SAT_CHECK_ARG(d->epilogue != 2 || d->out2 == nullptr ||
                    (d->gelu_col0 >= 0 && d->ldo2 >= d->N - d->gelu_col0),
                "%s: out2", fn);
  SAT_CHECK_ARG(d->splitk_ws_elems >= 0, "%s: negative splitk_ws_elems", fn);
  GemmArgs& a = *out;
  memset(&a, 0, sizeof a);
  a.A = (const bf16*)d->A;
  a.B = (const bf16*)d->B;
  a.M = d->M; a.N = d->N; a.K = d->K;
  a.lda = d->lda; a.ldb = d->ldb;
  a.out = d->out; a.ldo = d->ldo;
  a.bias = d->bias; a.bias_col0 = d->bias_col0;
  a.resid = d->resid; a.ldr = d->ldr;
  a.out2 = (bf16*)d->out2; a.ldo2 = d->ldo2; a.gelu_col0 = d->gelu_col0;
  a.aux = (const bf16*)d->aux; a.ldaux = d->ldaux;
  a.gelu_erf = d->gelu_erf;
  return SAT_OK;
}

extern "C" sat_status sat_op_gemm(const sat_gemm_desc* d, void* stream) {
  GemmArgs a;
  sat_status st = gemm_args(d, &a, "sat_op_gemm");
  if (st != SAT_OK) return st;
  a.splitk_ws = d->splitk_ws;
  a.splitk_ws_elems = d->splitk_ws ? d->splitk_ws_elems : 0;
  SAT_HIP(launch_gemm(a, d->a_layout, d->b_layout, d->epilogue, S(stream)));
  return SAT_OK;
}

// ---- sat_op_gemm_noalloc: the split-K workspace in a file-scope device array
//
// `scratch` is a host-side stand-in for the array in host code: its device
// address on the current device comes from hipGetSymbolAddress, looked up
// once per device on the first call there and kept in g_scratch_dev.  Every
// split-K slice writes all M x N of its partials before the reduction reads
// them, so the array needs no clearing between calls.
static __device__ __align__(256) float scratch[SAT_GEMM_NOALLOC_WS_ELEMS];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_dev[kMaxDevices];
}  // namespace

static sat_status scratch_on_current_device(float** out) {
  int dev = -1;
  SAT_HIP(hipGetDevice(&dev));
  SAT_CHECK_ARG(dev >= 0 && dev < kMaxDevices, "sat_op_gemm_noalloc: device %d beyond %d", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    SAT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    SAT_CHECK_ARG(p != nullptr && ((uintptr_t)p & 255) == 0,
                  "sat_op_gemm_noalloc: bad scratch address on device %d", dev);
    g_scratch_dev[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_dev[dev];
  return SAT_OK;
}

extern "C" sat_status sat_op_gemm_noalloc(const sat_gemm_desc* d, void* stream) {
  GemmArgs a;
  sat_status st = gemm_args(d, &a, "sat_op_gemm_noalloc");
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(d->splitk_ws == nullptr && d->splitk_ws_elems == 0,
                "sat_op_gemm_noalloc: splitk_ws must be NULL (the library's own scratch is used)");
  // the same split-K plan sat_op_gemm takes with a large enough workspace
  const bool may_split = (d->epilogue == 0 || d->epilogue == 1) && d->a_layout == 0 &&
                         d->b_layout == 0;
  // a product split for want of tiles must fit the scratch; one that would
  // only split the rows of its last round runs unsplit when those do not fit
  const long tail = may_split ? gemm_tail_ws_elems(d->M, d->N, d->K) : 0;
  const long need = may_split ? std::max(gemm_splitk_ws_elems(d->M, d->N, d->K),
                                         tail <= SAT_GEMM_NOALLOC_WS_ELEMS ? tail : 0L)
                              : 0;
  SAT_CHECK_ARG(need <= SAT_GEMM_NOALLOC_WS_ELEMS,
                "sat_op_gemm_noalloc: M=%d N=%d K=%d runs split-K with %ld fp32 partials, beyond "
                "the %ld-element scratch; use sat_op_gemm with a workspace",
                d->M, d->N, d->K, need, (long)SAT_GEMM_NOALLOC_WS_ELEMS);
  if (need > 0) {
    float* ws = nullptr;
    st = scratch_on_current_device(&ws);
    if (st != SAT_OK) return st;
    a.splitk_ws = ws;
    a.splitk_ws_elems = need;
  }
  SAT_HIP(launch_gemm(a, d->a_layout, d->b_layout, d->epilogue, S(stream)));
  return SAT_OK;
}

bool attention_supports_dh(int dh);

extern "C" sat_status sat_op_layernorm_fwd(const float* x, int64_t ldx, int64_t row_stride,
                                           const float* g, const float* b, void* y, int64_t ldy,
                                           float* mean, float* rstd, int32_t rows, int32_t d,
                                           float eps, void* stream) {
  SAT_CHECK_ARG(x && g && b && y && mean && rstd, "layernorm_fwd: null pointer");
  SAT_CHECK_ARG(rows >= 0 && d > 0 && d % 4 == 0 && d <= 8192, "layernorm_fwd: d=%d must be a positive multiple of 4 <= 8192", d);
  SAT_CHECK_ARG(ldx >= d && ldx % 4 == 0 && ldy >= d && ldy % 4 == 0 && row_stride >= 1,
                "layernorm_fwd: bad leading dimensions");
  SAT_HIP(launch_layernorm_fwd(x, ldx, row_stride, g, b, (bf16*)y, ldy, mean, rstd, rows, d, eps,
                               S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_layernorm_bwd(const float* dy, int64_t lddy, const float* x,
                                           int64_t ldx, int64_t row_stride, const float* g,
                                           const float* mean, const float* rstd, float* dres,
                                           int64_t ldres, float* dg, float* db, float* work,
                                           int32_t rows, int32_t d, void* stream) {
  SAT_CHECK_ARG(dy && x && g && mean && rstd && dres && dg && db && work,
                "layernorm_bwd: null pointer");
  SAT_CHECK_ARG(rows > 0 && d > 0 && d % 4 == 0 && d <= 4096, "layernorm_bwd: d=%d must be a positive multiple of 4 <= 4096", d);
  SAT_CHECK_ARG(lddy >= d && lddy % 4 == 0 && ldx >= d && ldx % 4 == 0 && ldres >= d &&
                    ldres % 4 == 0 && row_stride >= 1,
                "layernorm_bwd: bad leading dimensions");
  const int n_part = ln_bwd_parts(rows, d);
  SAT_HIP(launch_layernorm_bwd(dy, lddy, x, ldx, row_stride, g, mean, rstd, dres, ldres, work,
                               work + (long)n_part * d, rows, d, n_part, S(stream)));
  SAT_HIP(launch_ln_bwd_colsums(work, n_part, d, dg, db, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_attention_fwd(const void* q, const void* k, const void* v,
                                           int64_t ldq, int64_t ldk, int64_t ldv, void* o,
                                           int64_t ldo, float* lse, int32_t B, int32_t H,
                                           int32_t Sq, int32_t dh, int32_t causal, float scale,
                                           void* stream) {
  SAT_CHECK_ARG(q && k && v && o && lse, "attention_fwd: null pointer");
  SAT_CHECK_ARG(B >= 0 && H > 0 && Sq >= 0, "attention_fwd: bad sizes");
  SAT_CHECK_ARG(attention_supports_dh(dh), "attention_fwd: head dim %d not in {16,32,64,80,128,256}", dh);
  SAT_CHECK_ARG(ldq % 8 == 0 && ldk % 8 == 0 && ldv % 8 == 0 && ldq >= (int64_t)H * dh &&
                    ldk >= (int64_t)H * dh && ldv >= (int64_t)H * dh && ldo >= (int64_t)H * dh,
                "attention_fwd: leading dimensions must be multiples of 8 and >= H*dh");
  AttnArgs a;
  a.q = (const bf16*)q; a.k = (const bf16*)k; a.v = (const bf16*)v;
  a.ldq = ldq; a.ldk = ldk; a.ldv = ldv;
  a.o = (bf16*)o; a.ldo = ldo; a.lse = lse;
  a.B = B; a.H = H; a.S = Sq; a.dh = dh; a.causal = causal; a.scale = scale;
  SAT_CHECK_ARG(!(dh == 64 || dh == 80 || dh == 256) ||
                    (dh == 256 ? attn256_fwd_eligible(a) : attn_small_fwd_eligible(a)),
                "attention_fwd: head dim %d needs 16-byte aligned q, k, v, an 8-byte aligned o "
                "with ldo %% 4 == 0 and scale > 0", dh);
  SAT_HIP(launch_attention_fwd(a, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_attention_bwd(const void* q, const void* k, const void* v,
                                           int64_t ldq, int64_t ldk, int64_t ldv, const void* o,
                                           int64_t ldo, const float* lse, const void* dout,
                                           int64_t lddo, float* delta, void* dq, void* dk,
                                           void* dv, int64_t lddq, int64_t lddk, int64_t lddv,
                                           int32_t B, int32_t H, int32_t Sq, int32_t dh,
                                           int32_t causal, float scale, void* stream) {
  SAT_CHECK_ARG(q && k && v && o && lse && dout && delta && dq && dk && dv,
                "attention_bwd: null pointer");
  SAT_CHECK_ARG(B >= 0 && H > 0 && Sq >= 0, "attention_bwd: bad sizes");
  SAT_CHECK_ARG(attention_supports_dh(dh), "attention_bwd: head dim %d not in {16,32,64,80,128,256}", dh);
  SAT_CHECK_ARG(ldq % 8 == 0 && ldk % 8 == 0 && ldv % 8 == 0 && lddo % 8 == 0,
                "attention_bwd: leading dimensions must be multiples of 8");
  AttnBwdArgs a;
  a.f.q = (const bf16*)q; a.f.k = (const bf16*)k; a.f.v = (const bf16*)v;
  a.f.ldq = ldq; a.f.ldk = ldk; a.f.ldv = ldv;
  a.f.o = (bf16*)o; a.f.ldo = ldo; a.f.lse = (float*)lse;
  a.f.B = B; a.f.H = H; a.f.S = Sq; a.f.dh = dh; a.f.causal = causal; a.f.scale = scale;
  a.dout = (const bf16*)dout; a.lddo = lddo; a.delta = delta;
  a.dq = (bf16*)dq; a.dk = (bf16*)dk; a.dv = (bf16*)dv;
  a.lddq = lddq; a.lddk = lddk; a.lddv = lddv;
  SAT_CHECK_ARG(!(dh == 64 || dh == 80 || dh == 256) ||
                    (dh == 256 ? attn256_bwd_eligible(a) : attn_small_bwd_eligible(a)),
                "attention_bwd: head dim %d needs 16-byte aligned q, k, v, o, dout with leading "
                "dimensions %% 8 == 0, 8-byte aligned dq, dk, dv with leading dimensions %% 4 == 0 "
                "and scale > 0", dh);
  SAT_HIP(launch_attention_bwd(a, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_rotary(void* qk, int64_t ld, int32_t B, int32_t Sq, int32_t H,
                                    int32_t dh, int32_t rd, int32_t inverse, void* stream) {
  SAT_CHECK_ARG(qk != nullptr, "rotary: null pointer");
  SAT_CHECK_ARG(rd >= 0 && rd % 2 == 0 && rd <= dh, "rotary: rotary dim %d must be even and <= %d", rd, dh);
  SAT_CHECK_ARG(ld >= 2L * H * dh, "rotary: ld too small");
  SAT_CHECK_ARG(ld % 2 == 0 && dh % 2 == 0 && ((uintptr_t)qk & 3) == 0,
                "rotary: ld and head dim must be even and qk 4-byte aligned");
  SAT_HIP(launch_rotary((bf16*)qk, ld, B, Sq, H, dh, rd, inverse, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_cross_entropy(const float* z, int64_t ldz, const int32_t* labels,
                                           int32_t N, int32_t V, float* row_loss, void* dz,
                                           int64_t lddz, float* inv_n, void* stream) {
  SAT_CHECK_ARG(z && labels && row_loss && dz && inv_n, "cross_entropy: null pointer");
  SAT_CHECK_ARG(N >= 0 && V > 0 && ldz >= V && lddz >= V, "cross_entropy: bad sizes");
  SAT_HIP(launch_count_valid(labels, N, inv_n, S(stream)));
  SAT_HIP(launch_xent(z, ldz, labels, N, V, row_loss, (bf16*)dz, lddz, inv_n, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_adamw(float* p, const float* g, float* m, float* v, void* shadow,
                                   int64_t n, double lr, double beta1, double beta2, double eps,
                                   double wd, int64_t t, void* stream) {
  SAT_CHECK_ARG(p && g && m && v, "adamw: null pointer");
  SAT_CHECK_ARG(n >= 0 && t >= 1, "adamw: n >= 0 and t >= 1 required");
  SAT_HIP(launch_adamw(p, g, m, v, (bf16*)shadow, n, adamw_consts(lr, beta1, beta2, eps, wd, t),
                       S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_embed_fwd(const int32_t* tok, const float* wte, const float* wpe,
                                       float* h, int32_t T, int32_t Sq, int32_t d, int32_t V,
                                       void* stream) {
  SAT_CHECK_ARG(tok && wte && h, "embed_fwd: null pointer");
  SAT_CHECK_ARG(T >= 0 && Sq > 0 && d > 0 && d % 4 == 0 && V > 0, "embed_fwd: bad sizes");
  SAT_HIP(launch_embed_fwd(tok, wte, wpe, h, T, Sq, d, V, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_embed_bwd(const int32_t* tok, const float* dh, float* dwte,
                                       int32_t T, int32_t d, int32_t V, int32_t* work,
                                       void* stream) {
  SAT_CHECK_ARG(tok && dh && dwte && work, "embed_bwd: null pointer");
  SAT_CHECK_ARG(T > 0 && d > 0 && d % 4 == 0 && V > 0 && V < 65536,
                "embed_bwd: needs T > 0, d %% 4 == 0, 0 < V < 65536");
  SAT_HIP(launch_embed_bwd(tok, dh, dwte, T, d, V, work, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_colsum(const float* X, int64_t ldx, int32_t rows, int32_t cols,
                                    float* out, float* work, void* stream) {
  SAT_CHECK_ARG(X && out && work, "colsum: null pointer");
  SAT_CHECK_ARG(rows > 0 && cols >= 0 && ldx >= cols, "colsum: bad sizes");
  int n_part = rows < 256 ? rows : 256;
  SAT_HIP(launch_colsum_f32(X, ldx, rows, cols, work, n_part, out, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_transpose_bf16(const void* src, int64_t lds, void* dst, int64_t ldd,
                                            int32_t rows, int32_t cols, void* stream) {
  SAT_CHECK_ARG(src && dst, "transpose: null pointer");
  SAT_CHECK_ARG(rows >= 0 && cols >= 0 && rows % 8 == 0 && cols % 8 == 0,
                "transpose: rows and cols must be multiples of 8");
  SAT_CHECK_ARG(lds >= cols && ldd >= rows && lds % 8 == 0 && ldd % 8 == 0,
                "transpose: strides must cover the matrix and be multiples of 8");
  SAT_CHECK_ARG(((uintptr_t)src | (uintptr_t)dst) % 16 == 0, "transpose: pointers not 16-byte aligned");
  SAT_HIP(launch_transpose_bf16((const bf16*)src, lds, (bf16*)dst, ldd, rows, cols, S(stream)));
  return SAT_OK;
}

// ---- ResNet kernels (conv.hip)

static int conv_hw(int H, int k, int st, int pad) { return (H + 2 * pad - k) / st + 1; }

extern "C" sat_status sat_op_im2col(const void* x, void* col, int32_t N, int32_t H, int32_t W,
                                    int32_t C, int32_t k, int32_t stride, int32_t pad,
                                    void* stream) {
  SAT_CHECK_ARG(x && col, "im2col: null pointer");
  SAT_CHECK_ARG(N >= 1 && H >= 1 && W >= 1 && C >= 8 && C % 8 == 0 && k >= 1 && stride >= 1 &&
                    pad >= 0 && H + 2 * pad >= k && W + 2 * pad >= k,
                "im2col: bad sizes (C must be a positive multiple of 8)");
  const int Ho = conv_hw(H, k, stride, pad), Wo = conv_hw(W, k, stride, pad);
  SAT_HIP(launch_im2col((const bf16*)x, (bf16*)col, (long)k * k * C, N, H, W, C, k, stride, pad, Ho,
                        Wo, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_im2col_t(const void* x, void* colT, int64_t ldt, int32_t N, int32_t H,
                                      int32_t W, int32_t C, int32_t k, int32_t stride, int32_t pad,
                                      void* stream) {
  SAT_CHECK_ARG(x && colT, "im2col_t: null pointer");
  SAT_CHECK_ARG(N >= 1 && H >= 1 && W >= 1 && C >= 8 && C % 8 == 0 && k >= 1 && stride >= 1 &&
                    pad >= 0 && H + 2 * pad >= k && W + 2 * pad >= k,
                "im2col_t: bad sizes (C must be a positive multiple of 8)");
  const int Ho = conv_hw(H, k, stride, pad), Wo = conv_hw(W, k, stride, pad);
  const long P = (long)N * Ho * Wo;
  SAT_CHECK_ARG(P % 8 == 0 && ldt >= P && ldt % 8 == 0, "im2col_t: N Ho Wo and ldt must be multiples of 8, ldt >= N Ho Wo");
  SAT_CHECK_ARG(((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(colT)) & 15) == 0,
                "im2col_t: x and colT must be 16-byte aligned");
  SAT_HIP(launch_im2col_t((const bf16*)x, (bf16*)colT, ldt, N, H, W, C, k, stride, pad, Ho, Wo,
                          S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_col2im(const float* dcol, float* dx, int32_t N, int32_t H, int32_t W,
                                    int32_t C, int32_t k, int32_t stride, int32_t pad,
                                    int32_t accumulate, void* stream) {
  SAT_CHECK_ARG(dcol && dx, "col2im: null pointer");
  SAT_CHECK_ARG(N >= 1 && H >= 1 && W >= 1 && C >= 4 && C % 4 == 0 && k >= 1 && stride >= 1 &&
                    pad >= 0 && H + 2 * pad >= k && W + 2 * pad >= k,
                "col2im: bad sizes (C must be a positive multiple of 4)");
  const int Ho = conv_hw(H, k, stride, pad), Wo = conv_hw(W, k, stride, pad);
  SAT_HIP(launch_col2im(dcol, (long)k * k * C, dx, N, H, W, C, k, stride, pad, Ho, Wo, accumulate,
                        S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_batchnorm_fwd(const float* x, int64_t P, int32_t C, const float* g,
                                           const float* b, float eps, int32_t relu, float* part,
                                           float* mean, float* rstd, void* y, float* yf,
                                           void* stream) {
  SAT_CHECK_ARG(x && g && b && part && mean && rstd && (y || yf), "batchnorm_fwd: null pointer");
  SAT_CHECK_ARG(P >= 1 && C >= 4 && C % 4 == 0 && eps > 0.f, "batchnorm_fwd: bad sizes");
  auto al = [](const void* q, int n) { return q == nullptr || (reinterpret_cast<uintptr_t>(q) % n) == 0; };
  SAT_CHECK_ARG(al(x, 16) && al(g, 16) && al(b, 16) && al(part, 16) && al(mean, 16) && al(rstd, 16) &&
                    al(yf, 16) && al(y, 8),
                "batchnorm_fwd: fp32 arrays must be 16-byte aligned and y 8-byte aligned");
  SAT_HIP(launch_bn_stats(x, P, C, eps, part, mean, rstd, S(stream)));
  SAT_HIP(launch_bn_apply(x, P, C, mean, rstd, g, b, relu, (bf16*)y, yf, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_batchnorm_bwd(const float* dy, int32_t mask_kind, const void* mask,
                                           const float* x, const float* mean, const float* rstd,
                                           const float* g, int64_t P, int32_t C, float* part,
                                           float* dg, float* db, void* dx, void* stream) {
  SAT_CHECK_ARG(dy && x && mean && rstd && g && part && dg && db && dx, "batchnorm_bwd: null pointer");
  SAT_CHECK_ARG(mask_kind >= 0 && mask_kind <= 2 && (mask_kind == 0 || mask != nullptr),
                "batchnorm_bwd: mask_kind must be 0 (none), 1 (bf16) or 2 (fp32) with a mask");
  SAT_CHECK_ARG(P >= 1 && C >= 4 && C % 4 == 0, "batchnorm_bwd: bad sizes");
  auto al = [](const void* q, int n) { return q == nullptr || (reinterpret_cast<uintptr_t>(q) % n) == 0; };
  SAT_CHECK_ARG(al(dy, 16) && al(x, 16) && al(mean, 16) && al(rstd, 16) && al(g, 16) && al(part, 16) &&
                    al(dg, 16) && al(db, 16) && al(dx, 8) && al(mask, mask_kind == 2 ? 16 : 8),
                "batchnorm_bwd: fp32 arrays must be 16-byte aligned, dx and a bf16 mask 8-byte aligned");
  SAT_HIP(launch_bn_bwd(dy, mask_kind, mask, x, mean, rstd, g, P, C, part, dg, db, (bf16*)dx,
                        S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_maxpool_fwd(const float* x, int32_t N, int32_t H, int32_t W, int32_t C,
                                         float* y, void* yb, uint8_t* arg, void* stream) {
  SAT_CHECK_ARG(x && y && yb && arg, "maxpool_fwd: null pointer");
  SAT_CHECK_ARG(N >= 1 && H >= 2 && W >= 2 && C >= 1, "maxpool_fwd: bad sizes");
  SAT_HIP(launch_maxpool_fwd(x, N, H, W, C, conv_hw(H, 3, 2, 1), conv_hw(W, 3, 2, 1), y, (bf16*)yb,
                             arg, S(stream)));
  return SAT_OK;
}

extern "C" sat_status sat_op_maxpool_bwd(const float* dy, const uint8_t* arg, int32_t N, int32_t H,
                                         int32_t W, int32_t C, float* dx, void* stream) {
  SAT_CHECK_ARG(dy && arg && dx, "maxpool_bwd: null pointer");
  SAT_CHECK_ARG(N >= 1 && H >= 2 && W >= 2 && C >= 1, "maxpool_bwd: bad sizes");
  SAT_HIP(launch_maxpool_bwd(dy, arg, N, H, W, C, conv_hw(H, 3, 2, 1), conv_hw(W, 3, 2, 1), dx,
                             S(stream)));
  return SAT_OK;
}
