// Launch sequence of one fine-tuning step on the model's stream:
// embeddings -> blocks (LN, QKV, rotary, attention, out-projection, LN, MLP)
// -> final LN -> head -> cross-entropy, then the backward pass from the head
// down to block k (no work at all below it), then AdamW on the trainable
// suffix of the parameter arena.
#include <math.h>
#include <string.h>

#include "abi_common.h"
#include "kernels.h"
#include "model.h"
#include "step_common.h"

using namespace satstep;

namespace {

// Algorithmic bytes of the bandwidth kernels (each operand read once, each
// result written once): LayerNorm forward reads fp32 x and writes bf16 y plus
// the two per-row statistics; the backward reads dy, x and the residual
// gradient it accumulates into, writes that gradient back (and its bf16 copy),
// and reads the statistics; cross-entropy reads fp32 logits and the label and
// writes the bf16 logit gradient and the row loss.
double ln_fwd_bytes(long rows, int d) { return rows * (double)d * (4 + 2) + rows * 8.0 + d * 8.0; }
double ln_bwd_bytes(long rows, int d, bool bf) {
  return rows * (double)d * (4 + 4 + 4 + 4 + (bf ? 2 : 0)) + rows * 8.0 + d * 4.0;
}
double xent_bytes(long rows, long V) { return rows * (double)V * (4 + 2) + rows * 8.0; }

struct PIdx {
  const sat_model* M;
  int base;
  const ParamDesc& p(int i) const { return M->params[base + i]; }
};


// Index of the first parameter of block l and of the head group.
int embed_count(const sat_model* M) {
  if (M->D.arch == SAT_VIT) return 4;
  return M->D.arch == SAT_GPT2 ? 2 : 1;
}
int per_block(const sat_model* M) { return M->D.arch == SAT_GPTJ ? 8 : 12; }
int block_base(const sat_model* M, int l) { return embed_count(M) + l * per_block(M); }
int head_base(const sat_model* M) { return embed_count(M) + M->D.L * per_block(M); }

// Block parameter slots (GPT-2 / ViT order; GPT-J uses its own).
enum { B_LN1G = 0, B_LN1B, B_QKVW, B_QKVB, B_PROJW, B_PROJB, B_LN2G, B_LN2B, B_FC1W, B_FC1B, B_FC2W, B_FC2B };
enum { J_LN1G = 0, J_LN1B, J_QKVW, J_FC1W, J_FC1B, J_PROJW, J_FC2W, J_FC2B };

}  // namespace

const LayerActs& sat_layer_acts(const sat_model* M, int l) {
  const int k = M->D.k;
  if (M->D.ckpt) return M->acts[0];  // one set, rebuilt before each block's backward
  return (l < k) ? M->acts[0] : M->acts[l - k + (k > 0 ? 1 : 0)];
}

sat_status sat_run_init(sat_model* M) {
  const size_t NP = M->n_param_elems;
  hipStream_t s = M->stream;
  SAT_HIP(launch_zero(M->master, NP * 4, s));
  SAT_HIP(launch_zero(M->shadow, ((NP * 2 + 3) / 4) * 4, s));
  SAT_HIP(launch_zero(M->grad, NP * 4, s));
  SAT_HIP(launch_zero(M->mom, NP * 4, s));
  SAT_HIP(launch_zero(M->vel, NP * 4, s));
  if (!M->segs.empty())
    SAT_HIP(hipMemcpyAsync(M->segs_dev, M->segs.data(), M->segs.size() * sizeof(AdamWSeg),
                           hipMemcpyHostToDevice, s));
  if (!M->segs_rest.empty())
    SAT_HIP(hipMemcpyAsync(M->segs_rest_dev, M->segs_rest.data(),
                           M->segs_rest.size() * sizeof(AdamWSeg), hipMemcpyHostToDevice, s));
  for (size_t i = 0; i < M->params.size(); ++i) {
    const ParamDesc& p = M->params[i];
    long n = p.rows * p.cols;
    float* dst = M->master + p.off;
    bf16* sh = M->shadow + p.off;
    if (p.kind == 0)
      SAT_HIP(launch_init_normal(dst, sh, n, M->cfg.seed, (uint32_t)i, M->cfg.init_std, s));
    else
      SAT_HIP(launch_fill(dst, sh, n, p.kind == 2 ? 1.f : 0.f, s));
  }
  if (M->rope_cs) SAT_HIP(launch_rope_table(M->rope_cs, M->D.S, M->D.rd, s));
  return sat_refresh_transposed(M);
}

// Forward of block l from its input h_in[l] into its saved-activation set.
// recompute: the activations the backward of block l reads, rebuilt just
// before it (activation checkpointing) with the same kernels on the same
// input, so they are bitwise the values of the forward pass; the products
// whose results only feed the block's output (kept in h_in[l + 1]) are
// skipped, and nothing is counted in the per-kernel timing.
static sat_status block_forward(sat_model* M, int l, bool recompute) {
  const Dims& D = M->D;
  hipStream_t s = M->stream;
  const int T = D.T, d = D.d, m = D.m;
  const float eps = M->cfg.ln_eps;
  const int gelu_erf = D.arch == SAT_VIT ? 1 : 0;
  const bool gptj = D.arch == SAT_GPTJ;
  const int tk_qkv = recompute ? TK_ALL_GEMM : TK_QKV_FWD;
  const LayerActs& A = sat_layer_acts(M, l);
  const int pb = block_base(M, l);
  {
    Timed tm(M, TK_LN_FWD, ln_fwd_bytes(T, d));
    SAT_HIP(launch_layernorm_fwd(M->h_in[l], d, 1, master(M, pb + 0), master(M, pb + 1), A.a, d,
                                 A.mean1, A.rstd1, T, d, eps, s));
  }
  if (gptj) {
    // fused q | k | v | u = a [W_qkv; W_fc1]^T (+ fc1 bias on u), g = GELU(u)
    GemmArgs a = gargs(A.a, d, shadow(M, pb + J_QKVW), d, T, D.qkv_ld, d, A.qkv, D.qkv_ld);
    a.bias = master(M, pb + J_FC1B);
    a.bias_col0 = 3 * d;
    a.out2 = A.g;
    a.ldo2 = m;
    a.gelu_col0 = 3 * d;
    a.gelu_erf = 0;
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_BF16, tk_qkv));
    SAT_HIP(launch_rotary(A.qkv, D.qkv_ld, D.B, D.S, D.H, D.dh, D.rd, 0, s, M->rope_cs));
  } else {
    GemmArgs a = gargs(A.a, d, shadow(M, pb + B_QKVW), d, T, 3 * d, d, A.qkv, 3 * d);
    a.bias = master(M, pb + B_QKVB);
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_BF16, tk_qkv));
  }
  {
    AttnArgs at;
    at.q = A.qkv;
    at.k = A.qkv + d;
    at.v = A.qkv + 2 * d;
    at.ldq = at.ldk = at.ldv = D.qkv_ld;
    at.o = A.o;
    at.ldo = d;
    at.lse = A.lse;
    at.B = D.B;
    at.H = D.H;
    at.S = D.S;
    at.dh = D.dh;
    at.causal = D.arch != SAT_VIT;
    at.scale = 1.f / sqrtf((float)D.dh);
    if (recompute) {
      SAT_HIP(launch_attention_fwd(at, s));
    } else {
      Timed tm(M, TK_ATTN_FWD, 4.0 * D.B * D.H * (double)D.S * D.S * D.dh * (at.causal ? 0.5 : 1.0));
      SAT_HIP(launch_attention_fwd(at, s));
    }
  }
  if (gptj) {
    if (recompute) return SAT_OK;
    GemmArgs a = gargs(A.o, d, shadow(M, pb + J_PROJW), d, T, d, d, M->h_in[l + 1], d);
    a.resid = M->h_in[l];
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_RESID_F32));
    GemmArgs b = gargs(A.g, m, shadow(M, pb + J_FC2W), m, T, d, m, M->h_in[l + 1], d);
    b.resid = M->h_in[l + 1];
    b.bias = master(M, pb + J_FC2B);
    TRY(gemm(M, b, LAY_K, LAY_K, EPI_RESID_F32));
  } else {
    GemmArgs a = gargs(A.o, d, shadow(M, pb + B_PROJW), d, T, d, d, A.h_mid, d);
    a.resid = M->h_in[l];
    a.bias = master(M, pb + B_PROJB);
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_RESID_F32));
    {
      Timed tm(M, TK_LN_FWD, ln_fwd_bytes(T, d));
      SAT_HIP(launch_layernorm_fwd(A.h_mid, d, 1, master(M, pb + B_LN2G), master(M, pb + B_LN2B),
                                   A.c, d, A.mean2, A.rstd2, T, d, eps, s));
    }
    GemmArgs b = gargs(A.c, d, shadow(M, pb + B_FC1W), d, T, m, d, A.u, m);
    b.bias = master(M, pb + B_FC1B);
    b.out2 = A.g;
    b.ldo2 = m;
    b.gelu_col0 = 0;
    b.gelu_erf = gelu_erf;
    TRY(gemm(M, b, LAY_K, LAY_K, EPI_BF16));
    if (recompute) return SAT_OK;
    GemmArgs c = gargs(A.g, m, shadow(M, pb + B_FC2W), m, T, d, m, M->h_in[l + 1], d);
    c.resid = A.h_mid;
    c.bias = master(M, pb + B_FC2B);
    TRY(gemm(M, c, LAY_K, LAY_K, EPI_RESID_F32));
  }
  return SAT_OK;
}

sat_status sat_run_forward(sat_model* M, const void* inputs, const int32_t* labels) {
  if (M->D.arch == SAT_RESNET) return sat_resnet_forward(M, inputs, labels);
  const Dims& D = M->D;
  hipStream_t s = M->stream;
  const int T = D.T, d = D.d;
  const float eps = M->cfg.ln_eps;

  // ---- embeddings
  if (D.arch == SAT_VIT) {
    SAT_HIP(launch_patchify((const float*)inputs, M->patches, D.B, M->cfg.channels,
                            M->cfg.img_size, M->cfg.patch, D.pdp, s));
    GemmArgs a = gargs(M->patches, D.pdp, shadow(M, 0), D.pd, D.B * D.np, d, D.pd, M->zpatch, d);
    a.bias = master(M, 1);
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_F32));
    SAT_HIP(launch_vit_assemble(M->zpatch, master(M, 2), master(M, 3), M->h_in[0], D.B, D.np, d, s));
  } else {
    const float* wpe = (D.arch == SAT_GPT2) ? master(M, 1) : nullptr;
    SAT_HIP(launch_embed_fwd((const int32_t*)inputs, master(M, 0), wpe, M->h_in[0], T, D.S, d,
                             D.V, s));
  }

  // ---- blocks
  for (int l = 0; l < D.L; ++l) TRY(block_forward(M, l, false));

  // ---- final LN, head, cross-entropy
  const int hb = head_base(M);
  const int R = D.rows_head;
  const long rstride = (D.arch == SAT_VIT) ? D.S : 1;
  {
    Timed tm(M, TK_LN_FWD, ln_fwd_bytes(R, d));
    SAT_HIP(launch_layernorm_fwd(M->h_in[D.L], d, rstride, master(M, hb + 0), master(M, hb + 1),
                                 M->f, d, M->meanf, M->rstdf, R, d, eps, s));
  }
  GemmArgs a = gargs(M->f, d, shadow(M, hb + 2), d, R, D.V, d, M->logits, D.Vp);
  if (D.arch != SAT_GPT2) a.bias = master(M, hb + 3);
  TRY(gemm(M, a, LAY_K, LAY_K, EPI_F32));
  SAT_HIP(launch_count_valid(labels, R, M->scal + 1, s));
  {
    Timed tm(M, TK_XENT, xent_bytes(R, D.V));
    SAT_HIP(launch_xent(M->logits, D.Vp, labels, R, D.V, M->row_loss, M->dz, D.Vp, M->scal + 1, s));
  }
  SAT_HIP(launch_loss_finalize(M->row_loss, R, M->scal + 1, M->scal, s));
  return SAT_OK;
}

// dW[Mr, N] = sum over the T rows of Y[t, m] X[t, n] (Y, X bf16 row-major).
// With token-contiguous scratch (trans), both operands are first transposed
// into it (ycols >= Mr: the transposed width of Y, a multiple of 8), so the
// product reads K-contiguous operands; y_ready: tA already holds Y^T.
// pidx: the weight's parameter index.  When its AdamW step is fused, the
// product's epilogue applies the step to the weight (and writes the gradient
// only if the model keeps gradients).
// The product on token-contiguous operands yT [Mr, T] and xT [N, T], on
// stream st (the model's, or the weight-gradient stream).
static sat_status wgrad_t(sat_model* M, hipStream_t st, const bf16* yT, const bf16* xT, int Mr,
                          int N, int T, int pidx, int tk = TK_ALL_GEMM) {
  const ParamDesc& P = M->params[pidx];
  GemmArgs w = gargs(yT, T, xT, T, Mr, N, T, grad(M, pidx), P.cols);
  if (M->opt_fused && P.fused_opt) {
    if (!M->opt_keep_grads) w.out = nullptr;
    w.opt_p = M->master + P.off;
    w.opt_m = M->mom + P.off;
    w.opt_v = M->vel + P.off;
    w.opt_sh = M->shadow + P.off;
    w.opt_sht = M->shadow_t + P.toff;
    w.opt_trows = P.trows;
    w.opt_c = M->adamw_c;
    if (!gemm256_eligible(w, LAY_K, LAY_K, EPI_ADAMW)) {
      sat_set_error("internal: fused optimizer step of %s not eligible for the 256 x 256 kernel",
                    P.name.c_str());
      return SAT_EINVAL;
    }
    return gemm(M, w, LAY_K, LAY_K, EPI_ADAMW, tk, st);
  }
  // the same sums as the fused epilogue's (no row split of the last round),
  // so that the separate AdamW pass gives the fused step's parameters
  w.no_tail_split = 1;
  return gemm(M, w, LAY_K, LAY_K, EPI_F32, tk, st);
}

static sat_status wgrad(sat_model* M, bool trans, bool y_ready, const bf16* Y, long ldy,
                        int ycols, const bf16* X, long ldx, int Mr, int N, int T, int pidx,
                        int tk = TK_ALL_GEMM) {
  const ParamDesc& P = M->params[pidx];
  float* out = grad(M, pidx);
  const long ldo = P.cols;
  if (trans) {
    if (!y_ready) SAT_HIP(launch_transpose_bf16(Y, ldy, M->tA, T, T, ycols, M->stream));
    SAT_HIP(launch_transpose_bf16(X, ldx, M->tB, T, T, N, M->stream));
    return wgrad_t(M, M->stream, M->tA, M->tB, Mr, N, T, pidx, tk);
  }
  GemmArgs w = gargs(Y, ldy, X, ldx, Mr, N, T, out, ldo);
  return gemm(M, w, LAY_MN, LAY_MN, EPI_F32, tk);
}

// The fc1 bias gradient is the column sum of the fc2 input-gradient product's
// output.  Where the 256 x 256 kernel runs that product, its epilogue writes
// the column sums of every 128-row block into the partial buffer, which one
// launch of the partial-sum kernel then adds in order; otherwise the output is
// summed by the column-sum kernels afterwards.
static bool with_colsums(sat_model* M, GemmArgs& a) {
  a.colsum_part = sat_fc1_bias_in_epilogue(M->D) ? M->part : nullptr;
  if (!a.colsum_part) return false;
  if (((long)a.M + 127) / 128 * a.N > M->part_elems || !gemm256_eligible(a, LAY_K, LAY_K, EPI_DGELU_BF16))
    a.colsum_part = nullptr;
  return a.colsum_part != nullptr;
}

// Weight-gradient stream.  fork: what the model's stream has enqueued so far
// (the operand copies) precedes what the side stream enqueues next.  reuse:
// before the model's stream rewrites operand set i, the products that read it
// are done.  done: marks the end of the products of set i.  join: the model's
// stream waits for everything on the side stream.
static sat_status side_fork(sat_model* M) {
  SAT_HIP(hipEventRecord(M->ev_fork, M->stream));
  SAT_HIP(hipStreamWaitEvent(M->side, M->ev_fork, 0));
  return SAT_OK;
}
static sat_status side_reuse(sat_model* M, int i) {
  if (M->side_pending[i]) SAT_HIP(hipStreamWaitEvent(M->stream, M->ev_done[i], 0));
  M->side_pending[i] = false;
  return SAT_OK;
}
static sat_status side_done(sat_model* M, int i) {
  SAT_HIP(hipEventRecord(M->ev_done[i], M->side));
  M->side_pending[i] = true;
  return SAT_OK;
}
static sat_status side_join(sat_model* M) {
  SAT_HIP(hipEventRecord(M->ev_join, M->side));
  SAT_HIP(hipStreamWaitEvent(M->stream, M->ev_join, 0));
  M->side_pending[0] = M->side_pending[1] = false;
  return SAT_OK;
}

// LayerNorm backward into the residual gradient dh, which it also rounds into
// dh_bf, the bf16 copy the next products read.  dbias (may be null): the bias
// gradient of the residual product below, the column sums of the updated dh,
// reduced in the same pass.
static sat_status ln_bwd(sat_model* M, const float* dy, const float* x, long row_stride,
                         int gidx, const float* mean, const float* rstd, int rows,
                         float* dbias = nullptr) {
  const int d = M->D.d;
  const int np_ = ln_bwd_parts(rows, d);
  float* pg = M->part;
  float* pbb = M->part + (size_t)np_ * d;
  float* po = dbias ? M->part + (size_t)2 * np_ * d : nullptr;
  {
    Timed tm(M, TK_LN_BWD, ln_bwd_bytes(rows, d, true));
    SAT_HIP(launch_layernorm_bwd(dy, d, x, d, row_stride, master(M, gidx), mean, rstd, M->dh, d, pg,
                                 pbb, rows, d, np_, M->stream, M->dh_bf, d, po));
  }
  SAT_HIP(launch_ln_bwd_colsums(pg, np_, d, grad(M, gidx), grad(M, gidx + 1), M->stream, dbias));
  return SAT_OK;
}

// The bias gradients of the residual products (fc2; for GPT-2 / ViT also the
// out-projection) are the column sums of the residual gradient dh that the
// LayerNorm backward above them leaves.  For rows up to 2048 wide that pass
// reduces them as a third partial row (no separate read of dh).  For wider
// rows the extra registers and adds in it cost more than a separate column
// sum (GPT-J's 4096-wide rows: 0.6 ms per step slower).
static bool bias_in_ln_bwd(const sat_model* M) { return sat_bias_in_ln_bwd(M->D); }

// Where the LayerNorm backward above block l reduces block l's fc2 bias
// gradient: null when block l is frozen or the sum runs separately.
static float* fc2_bias_grad(sat_model* M, int l) {
  if (l < M->D.k || l < 0 || !bias_in_ln_bwd(M)) return nullptr;
  return grad(M, block_base(M, l) + (M->D.arch == SAT_GPTJ ? J_FC2B : B_FC2B));
}

sat_status sat_run_backward(sat_model* M, const void* inputs) {
  if (M->D.arch == SAT_RESNET) return sat_resnet_backward(M, inputs);
  const Dims& D = M->D;
  hipStream_t s = M->stream;
  const int T = D.T, d = D.d, m = D.m;
  const int gelu_erf = D.arch == SAT_VIT ? 1 : 0;
  const bool gptj = D.arch == SAT_GPTJ;
  const int hb = head_base(M);
  const int R = D.rows_head;
  const int npT = M->n_part;

  // ---- head
  {
    // Every input-gradient product of a weight runs before its weight-gradient
    // product, which may apply the weight's AdamW step in its epilogue.
    // K = Vp: the padding columns of dz are zero and the parameter arena has a
    // zero tail, so the extra products vanish and the 16-byte path applies.
    GemmArgs g = gargs(M->dz, D.Vp, shadow_t(M, hb + 2), D.Vp, R, d, D.Vp, M->dA, d);
    TRY(gemm(M, g, LAY_K, LAY_K, EPI_F32));
    TRY(wgrad(M, M->trans_head, false, M->dz, D.Vp, D.Vp, M->f, d, D.V, d, R, hb + 2));
    if (D.arch != SAT_GPT2)
      SAT_HIP(launch_colsum_bf16(M->dz, D.Vp, R, D.V, M->part, R < 256 ? R : 256,
                                 grad(M, hb + 3), s));
    SAT_HIP(launch_zero(M->dh, (long)T * d * 4, s));
    const long rstride = (D.arch == SAT_VIT) ? D.S : 1;
    // LN_f backward writes rows r * rstride of dh (CLS rows for ViT)
    // (the column sums of dh, zero outside those rows, are the top block's fc2
    // bias gradient)
    const int np_ = ln_bwd_parts(R, d);
    float* pg = M->part;
    float* pbb = M->part + (size_t)np_ * d;
    float* dbias_top = fc2_bias_grad(M, D.L - 1);
    float* po = dbias_top ? M->part + (size_t)2 * np_ * d : nullptr;
    {
      Timed tm(M, TK_LN_BWD, ln_bwd_bytes(R, d, rstride == 1));
      SAT_HIP(launch_layernorm_bwd(M->dA, d, M->h_in[D.L], d, rstride, master(M, hb + 0),
                                   M->meanf, M->rstdf, M->dh, d, pg, pbb, R, d, np_, s,
                                   rstride == 1 ? M->dh_bf : nullptr, d, po));
    }
    if (rstride != 1)  // ViT: only the CLS rows of dh were written
      SAT_HIP(launch_f32_to_bf16(M->dh, d, M->dh_bf, d, T, d, s));
    SAT_HIP(launch_ln_bwd_colsums(pg, np_, d, grad(M, hb + 0), grad(M, hb + 1), s, dbias_top));
  }

  // ---- blocks L-1 .. k
  // With the weight-gradient stream, block l's operand copies go to set l % 2
  // on the model's stream and its weight-gradient products run on the side
  // stream; every input-gradient product of a weight is enqueued before the
  // fork that releases the weight's (AdamW-fused) weight-gradient product.
  const bool ov = M->opt_overlap && M->trans_blocks && D.k < D.L;
  if (ov) TRY(sat_side_ensure(M));
  for (int l = D.L - 1; l >= D.k; --l) {
    if (ov) TRY(side_reuse(M, l & 1));
    WgradSet& W = M->wset[l & 1];
    if (D.ckpt) TRY(block_forward(M, l, true));
    const LayerActs& A = sat_layer_acts(M, l);
    const int pb = block_base(M, l);
    AttnBwdArgs ab;
    ab.f.q = A.qkv;
    ab.f.k = A.qkv + d;
    ab.f.v = A.qkv + 2 * d;
    ab.f.ldq = ab.f.ldk = ab.f.ldv = D.qkv_ld;
    ab.f.o = A.o;
    ab.f.ldo = d;
    ab.f.lse = A.lse;
    ab.f.B = D.B;
    ab.f.H = D.H;
    ab.f.S = D.S;
    ab.f.dh = D.dh;
    ab.f.causal = D.arch != SAT_VIT;
    ab.f.scale = 1.f / sqrtf((float)D.dh);
    ab.dout = M->dout;
    ab.lddo = d;
    ab.delta = M->delta;
    ab.dq = M->dqkv;
    ab.dk = M->dqkv + d;
    ab.dv = M->dqkv + 2 * d;
    ab.lddq = ab.lddk = ab.lddv = D.qkv_ld;
    const double attn_bwd_flops =
        8.0 * D.B * D.H * (double)D.S * D.S * D.dh * (ab.f.causal ? 0.5 : 1.0);

    // dh_bf: the bf16 copy of dh, written by the LayerNorm backward that last
    // updated dh (the head's, or the block above's)
    if (gptj) {
      const bool tr = M->trans_blocks;
      if (!bias_in_ln_bwd(M))
        SAT_HIP(launch_colsum_f32(M->dh, d, T, d, M->part, npT, grad(M, pb + J_FC2B), s));
      GemmArgs du = gargs(M->dh_bf, d, shadow_t(M, pb + J_FC2W), d, T, m, d, M->dqkv + 3 * d, D.qkv_ld);
      du.aux = A.qkv + 3 * d;
      du.ldaux = D.qkv_ld;
      du.gelu_erf = 0;
      const bool fc1b_fused = with_colsums(M, du);
      TRY(gemm(M, du, LAY_K, LAY_K, EPI_DGELU_BF16));
      if (fc1b_fused)
        SAT_HIP(launch_colsum_partials(M->part, (int)((T + 127) / 128), m, grad(M, pb + J_FC1B), s));
      GemmArgs go = gargs(M->dh_bf, d, shadow_t(M, pb + J_PROJW), d, T, d, d, M->dout, d);
      TRY(gemm(M, go, LAY_K, LAY_K, EPI_BF16));
      if (ov) {
        SAT_HIP(launch_transpose_bf16(M->dh_bf, d, W.dy1, T, T, d, s));
        SAT_HIP(launch_transpose_bf16(A.g, m, W.g, T, T, m, s));
        SAT_HIP(launch_transpose_bf16(A.o, d, W.o, T, T, d, s));
        TRY(side_fork(M));
        TRY(wgrad_t(M, M->side, W.dy1, W.g, d, m, T, pb + J_FC2W));
        TRY(wgrad_t(M, M->side, W.dy1, W.o, d, d, T, pb + J_PROJW));
      } else {
        TRY(wgrad(M, tr, false, M->dh_bf, d, d, A.g, m, d, m, T, pb + J_FC2W));
        TRY(wgrad(M, tr, true, M->dh_bf, d, d, A.o, d, d, d, T, pb + J_PROJW));
      }
      {
        Timed tm(M, TK_ATTN_BWD, attn_bwd_flops);
        SAT_HIP(launch_attention_bwd(ab, s));
      }
      SAT_HIP(launch_rotary(M->dqkv, D.qkv_ld, D.B, D.S, D.H, D.dh, D.rd, 1, s, M->rope_cs));
      GemmArgs ga = gargs(M->dqkv, D.qkv_ld, shadow_t(M, pb + J_QKVW), D.qkv_ld, T, d, D.qkv_ld,
                          M->dA, d);
      TRY(gemm(M, ga, LAY_K, LAY_K, EPI_F32));
      if (ov) {
        SAT_HIP(launch_transpose_bf16(M->dqkv, D.qkv_ld, W.qkv, T, T, D.qkv_ld, s));
        SAT_HIP(launch_transpose_bf16(A.a, d, W.a, T, T, d, s));
        TRY(side_fork(M));
        TRY(wgrad_t(M, M->side, W.qkv, W.a, D.qkv_ld, d, T, pb + J_QKVW, TK_QKV_WGRAD));
        TRY(side_done(M, l & 1));
      } else {
        TRY(wgrad(M, tr, false, M->dqkv, D.qkv_ld, D.qkv_ld, A.a, d, D.qkv_ld, d, T, pb + J_QKVW,
                  TK_QKV_WGRAD));
      }
      if (!fc1b_fused)
        SAT_HIP(launch_colsum_bf16(M->dqkv + 3 * d, D.qkv_ld, T, m, M->part, npT,
                                   grad(M, pb + J_FC1B), s));
      TRY(ln_bwd(M, M->dA, M->h_in[l], 1, pb + J_LN1G, A.mean1, A.rstd1, T,
                 fc2_bias_grad(M, l - 1)));
    } else {
      const bool tr = M->trans_blocks;
      if (!bias_in_ln_bwd(M))
        SAT_HIP(launch_colsum_f32(M->dh, d, T, d, M->part, npT, grad(M, pb + B_FC2B), s));
      GemmArgs du = gargs(M->dh_bf, d, shadow_t(M, pb + B_FC2W), d, T, m, d, M->du, m);
      du.aux = A.u;
      du.ldaux = m;
      du.gelu_erf = gelu_erf;
      const bool fc1b_fused = with_colsums(M, du);
      TRY(gemm(M, du, LAY_K, LAY_K, EPI_DGELU_BF16));
      if (fc1b_fused)
        SAT_HIP(launch_colsum_partials(M->part, (int)((T + 127) / 128), m, grad(M, pb + B_FC1B), s));
      GemmArgs gc = gargs(M->du, m, shadow_t(M, pb + B_FC1W), m, T, d, m, M->dA, d);
      TRY(gemm(M, gc, LAY_K, LAY_K, EPI_F32));
      if (ov) {
        SAT_HIP(launch_transpose_bf16(M->dh_bf, d, W.dy1, T, T, d, s));
        SAT_HIP(launch_transpose_bf16(A.g, m, W.g, T, T, m, s));
        SAT_HIP(launch_transpose_bf16(M->du, m, W.du, T, T, m, s));
        SAT_HIP(launch_transpose_bf16(A.c, d, W.c, T, T, d, s));
        TRY(side_fork(M));
        TRY(wgrad_t(M, M->side, W.dy1, W.g, d, m, T, pb + B_FC2W));
        TRY(wgrad_t(M, M->side, W.du, W.c, m, d, T, pb + B_FC1W));
      } else {
        TRY(wgrad(M, tr, false, M->dh_bf, d, d, A.g, m, d, m, T, pb + B_FC2W));
        TRY(wgrad(M, tr, false, M->du, m, m, A.c, d, m, d, T, pb + B_FC1W));
      }
      if (!fc1b_fused)
        SAT_HIP(launch_colsum_bf16(M->du, m, T, m, M->part, npT, grad(M, pb + B_FC1B), s));
      TRY(ln_bwd(M, M->dA, A.h_mid, 1, pb + B_LN2G, A.mean2, A.rstd2, T,
                 bias_in_ln_bwd(M) ? grad(M, pb + B_PROJB) : nullptr));
      if (!bias_in_ln_bwd(M))
        SAT_HIP(launch_colsum_f32(M->dh, d, T, d, M->part, npT, grad(M, pb + B_PROJB), s));
      GemmArgs go = gargs(M->dh_bf, d, shadow_t(M, pb + B_PROJW), d, T, d, d, M->dout, d);
      TRY(gemm(M, go, LAY_K, LAY_K, EPI_BF16));
      if (ov) {
        SAT_HIP(launch_transpose_bf16(M->dh_bf, d, W.dy2, T, T, d, s));
        SAT_HIP(launch_transpose_bf16(A.o, d, W.o, T, T, d, s));
        TRY(side_fork(M));
        TRY(wgrad_t(M, M->side, W.dy2, W.o, d, d, T, pb + B_PROJW));
      } else {
        TRY(wgrad(M, tr, false, M->dh_bf, d, d, A.o, d, d, d, T, pb + B_PROJW));
      }
      {
        Timed tm(M, TK_ATTN_BWD, attn_bwd_flops);
        SAT_HIP(launch_attention_bwd(ab, s));
      }
      GemmArgs ga = gargs(M->dqkv, 3 * d, shadow_t(M, pb + B_QKVW), 3 * d, T, d, 3 * d, M->dA, d);
      TRY(gemm(M, ga, LAY_K, LAY_K, EPI_F32));
      if (ov) {
        SAT_HIP(launch_transpose_bf16(M->dqkv, 3 * d, W.qkv, T, T, 3 * d, s));
        SAT_HIP(launch_transpose_bf16(A.a, d, W.a, T, T, d, s));
        TRY(side_fork(M));
        TRY(wgrad_t(M, M->side, W.qkv, W.a, 3 * d, d, T, pb + B_QKVW, TK_QKV_WGRAD));
        TRY(side_done(M, l & 1));
      } else {
        TRY(wgrad(M, tr, false, M->dqkv, 3 * d, 3 * d, A.a, d, 3 * d, d, T, pb + B_QKVW,
                  TK_QKV_WGRAD));
      }
      SAT_HIP(launch_colsum_bf16(M->dqkv, 3 * d, T, 3 * d, M->part, npT, grad(M, pb + B_QKVB), s));
      TRY(ln_bwd(M, M->dA, M->h_in[l], 1, pb + B_LN1G, A.mean1, A.rstd1, T,
                 fc2_bias_grad(M, l - 1)));
    }
  }

  if (ov) TRY(side_join(M));

  // ---- embeddings (only when nothing is frozen)
  if (D.k == 0) {
    if (D.arch == SAT_VIT) {
      SAT_HIP(launch_sum_rows_batched(M->dh, grad(M, 3), D.B, D.S, d, s));
      SAT_HIP(hipMemcpyAsync(grad(M, 2), grad(M, 3), (size_t)d * 4, hipMemcpyDeviceToDevice, s));
      SAT_HIP(launch_vit_patch_grad(M->dh, M->dzpatch, D.B, D.np, d, s));
      const int rows = D.B * D.np;
      if (M->trans_blocks && rows % 8 == 0 && d % 8 == 0) {
        // a reduction over every patch of the batch into a 1280 x 588 weight: on
        // token-contiguous copies it runs split-K over the whole chip
        SAT_HIP(launch_transpose_bf16(M->dzpatch, d, M->tA, rows, rows, d, s));
        SAT_HIP(launch_transpose_bf16(M->patches, D.pdp, M->tB, rows, rows, D.pdp, s));
        TRY(wgrad_t(M, s, M->tA, M->tB, d, D.pd, rows, 0));
      } else {
        GemmArgs wp = gargs(M->dzpatch, d, M->patches, D.pdp, d, D.pd, rows, grad(M, 0), D.pd);
        TRY(gemm(M, wp, LAY_MN, LAY_MN, EPI_F32));
      }
      SAT_HIP(launch_colsum_bf16(M->dzpatch, d, rows, d, M->part, rows < 256 ? rows : 256,
                                 grad(M, 1), s));
    } else {
      SAT_HIP(launch_embed_bwd((const int32_t*)inputs, M->dh, grad(M, 0), T, d, D.V, M->sortbuf, s));
      if (D.arch == SAT_GPT2) SAT_HIP(launch_sum_rows_batched(M->dh, grad(M, 1), D.B, D.S, d, s));
    }
  }
  return SAT_OK;
}

sat_status sat_refresh_transposed(sat_model* M, int only) {
  for (size_t i = 0; i < M->params.size(); ++i) {
    const ParamDesc& p = M->params[i];
    if (p.toff == SIZE_MAX) continue;
    if (only >= 0) {
      // the block [off, off + trows * cols) may span several parameters
      const ParamDesc& q = M->params[only];
      if (q.off + (size_t)q.rows * q.cols <= p.off || q.off >= p.off + (size_t)p.trows * p.cols)
        continue;
    }
    SAT_HIP(launch_transpose_bf16(M->shadow + p.off, p.cols, M->shadow_t + p.toff, p.trows,
                                  (int)p.trows, (int)p.cols, M->stream));
  }
  return SAT_OK;
}

sat_status sat_adamw_begin(sat_model* M) {
  M->t += 1;
  const sat_config& c = M->cfg;
  M->adamw_c = adamw_consts(c.lr, c.beta1, c.beta2, c.eps, c.weight_decay, M->t);
  M->last_step_fused = M->opt_fused;
  M->last_step_kept = M->opt_keep_grads;
  return SAT_OK;
}

sat_status sat_run_adamw(sat_model* M) {
  const bool fused = M->opt_fused;
  const std::vector<AdamWSeg>& segs = fused ? M->segs_rest : M->segs;
  Timed tm(M, TK_ADAMW, fused ? M->seg_rest_bytes : M->seg_bytes);
  SAT_HIP(launch_adamw_segments(M->master, M->grad, M->mom, M->vel, M->shadow, M->shadow_t,
                                fused ? M->segs_rest_dev : M->segs_dev, (int)segs.size(),
                                fused ? M->seg_rest_blocks : M->seg_blocks, M->adamw_c,
                                M->stream));
  return SAT_OK;
}
