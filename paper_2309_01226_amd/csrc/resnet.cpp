// Bottleneck-ResNet fine-tuning step (the paper's second image model, Table 3
// and Sec. 5 "Workloads": a ResNet of about 200 M parameters fine-tuned on
// ImageNet-shaped images): parameter table, memory plan and the launch
// sequence of forward, backward and AdamW on the model's stream.
//
// Every convolution is one MFMA GEMM over NHWC activations (rows = output
// pixels, columns = channels): a 1 x 1 convolution multiplies the activation
// matrix itself, a 3 x 3 (or the 7 x 7 stem) the im2col matrix of its input,
// a stride-2 1 x 1 projection the every-other-pixel subsample.  Its input
// gradient is one GEMM against the transposed bf16 weight copy, scattered
// back by col2im where the convolution is not 1 x 1; its weight gradient is
// one GEMM over the pixels (K = N H W) on token-contiguous copies of both
// operands, split over K so that the few output tiles still fill the chip.
// Batch norm runs in training mode: statistics of the batch, then a fused
// normalise (+ ReLU, + shortcut add) pass; its backward reduces the two
// per-channel sums, then applies the closed-form input gradient.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <memory>
#include <string>
#include <vector>

#include "abi_common.h"
#include "kernels.h"
#include "model.h"
#include "step_common.h"

using namespace satstep;

namespace {

constexpr int kSplitMax = 256;  // K slices of the pixel-long weight-gradient products

struct RBn {
  int g = -1;  // parameter index of the gain (the shift follows it)
  float* mean = nullptr;
  float* rstd = nullptr;
};

struct RBlock {
  int idx, stride;
  bool proj;
  int cin, mid, cout, H, W, Ho, Wo;
  long Pin, Pout;
  int w1, w2, w3, wd;  // parameter indices of the convolution weights (wd: -1 without projection)
  RBn n1, n2, n3, nd;
  float* c1 = nullptr;  // conv outputs before batch norm (fp32)
  float* c2 = nullptr;
  float* c3 = nullptr;
  float* cd = nullptr;
  bf16* a1 = nullptr;   // ReLU(BN) outputs feeding the next convolution (bf16)
  bf16* a2 = nullptr;
};

}  // namespace

struct ResNetPlan {
  int N = 0, C = 0, img = 0, width = 0, classes = 0, Vp = 0, F = 0;
  int Hs = 0, Hp = 0, Hf = 0;  // stem conv output, after max pool, last stage
  long Ps = 0, Pp = 0;
  int stem_w = -1, stem_kp = 0;
  RBn stem_n;
  int fc_w = -1;
  std::vector<RBlock> blocks;
  std::vector<float*> x;  // x[i]: input of block i; x[n_blocks]: last block output
  std::vector<bf16*> xb;  // their bf16 copies
  std::vector<long> x_rows;
  std::vector<int> x_cols;
  float* stem_c = nullptr;
  float* stem_act = nullptr;
  uint8_t* pool_arg = nullptr;
  bf16* stem_wpad = nullptr;
  bf16* col = nullptr;
  bf16* feat = nullptr;
  // backward workspace
  float* g0 = nullptr;
  float* g1 = nullptr;
  float* gdo = nullptr;
  float* da = nullptr;
  float* dcol = nullptr;
  float* dsub = nullptr;
  bf16* dc = nullptr;
  bf16* dcd = nullptr;
  bf16* tA = nullptr;
  bf16* tB = nullptr;
  float* part = nullptr;
  float* dfeat = nullptr;
};

namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int conv_out(int H, int k, int s, int pad) { return (H + 2 * pad - k) / s + 1; }

void add_param(std::vector<ParamDesc>& P, size_t& off, const std::string& name, long rows,
               long cols, int group, int kind) {
  ParamDesc p;
  p.name = name;
  p.rows = rows;
  p.cols = cols;
  p.off = off;
  p.group = group;
  p.kind = kind;
  p.trainable = false;
  p.toff = SIZE_MAX;
  p.trows = 0;
  p.fused_opt = false;
  P.push_back(p);
  off = align_up(off + (size_t)rows * cols, 64);
}

// The block table of a configuration (geometry only).
std::vector<RBlock> block_table(const sat_config& c, int Hp) {
  std::vector<RBlock> out;
  int cin = c.res_width, H = Hp, idx = 0;
  for (int s = 0; s < 4; ++s) {
    const int mid = c.res_width << s;
    for (int j = 0; j < c.res_blocks[s]; ++j) {
      RBlock b;
      b.idx = idx++;
      b.stride = (j == 0 && s > 0) ? 2 : 1;
      b.proj = j == 0;
      b.cin = cin;
      b.mid = mid;
      b.cout = 4 * mid;
      b.H = b.W = H;
      b.Ho = b.Wo = conv_out(H, 3, b.stride, 1);
      b.Pin = (long)c.batch * H * H;
      b.Pout = (long)c.batch * b.Ho * b.Wo;
      b.w1 = b.w2 = b.w3 = b.wd = -1;
      out.push_back(b);
      cin = b.cout;
      H = b.Ho;
    }
  }
  return out;
}

int stem_hw(const sat_config& c) { return conv_out(c.img_size, 7, 2, 3); }
int pool_hw(const sat_config& c) { return conv_out(stem_hw(c), 3, 2, 1); }

}  // namespace

sat_status sat_resnet_validate(const sat_config* c) {
  int total = 0;
  for (int s = 0; s < 4; ++s) {
    SAT_CHECK_ARG(c->res_blocks[s] >= 1, "res_blocks[%d] must be >= 1", s);
    total += c->res_blocks[s];
  }
  SAT_CHECK_ARG(c->n_layers == total, "n_layers %d must equal the sum of res_blocks (%d)",
                c->n_layers, total);
  SAT_CHECK_ARG(c->res_width >= 8 && c->res_width % 8 == 0 && c->res_width <= 512,
                "res_width must be a multiple of 8 in [8, 512]");
  SAT_CHECK_ARG(c->channels >= 1 && c->channels <= 16, "channels must be in [1, 16]");
  SAT_CHECK_ARG(c->img_size >= 8 && c->img_size <= 1024, "img_size must be in [8, 1024]");
  SAT_CHECK_ARG(c->vocab >= 2, "classes (vocab) must be >= 2");
  SAT_CHECK_ARG(c->batch >= 1, "batch must be >= 1");
  SAT_CHECK_ARG(c->frozen_layers >= 0 && c->frozen_layers <= c->n_layers,
                "frozen_layers %d not in [0, n_layers]", c->frozen_layers);
  SAT_CHECK_ARG(c->checkpoint == 0, "activation checkpointing is not offered for RESNET");
  SAT_CHECK_ARG(c->rotary_dim == 0, "rotary_dim must be 0 for RESNET");
  // the stem's pixel count is the largest GEMM row count and the K of the
  // stem's weight gradient: it must fit the GEMMs' 32-bit indexing
  const long Ps = (long)c->batch * stem_hw(*c) * stem_hw(*c);
  SAT_CHECK_ARG(Ps * 256 < (1L << 30), "batch * image too large (%ld stem pixels)", Ps);
  SAT_CHECK_ARG(c->lr >= 0.0 && c->beta1 >= 0.0 && c->beta1 < 1.0 && c->beta2 >= 0.0 &&
                    c->beta2 < 1.0 && c->eps > 0.0 && c->weight_decay >= 0.0,
                "invalid AdamW hyper-parameters");
  SAT_CHECK_ARG(c->ln_eps > 0.f && c->init_std >= 0.f, "invalid ln_eps / init_std");
  return SAT_OK;
}

void sat_resnet_dims(const sat_config& c, Dims* d) {
  memset(d, 0, sizeof *d);
  d->arch = SAT_RESNET;
  d->L = c.n_layers;
  d->k = c.frozen_layers;
  d->V = c.vocab;
  d->Vp = (int)align_up(c.vocab, 8);
  d->B = c.batch;
  d->S = 1;
  d->T = c.batch;
  d->rows_head = c.batch;
  d->d = 4 * (c.res_width << 3);  // feature width entering the head
  for (int s = 0; s < 4; ++s) d->res_blocks[s] = c.res_blocks[s];
  d->res_width = c.res_width;
  d->img = c.img_size;
  d->channels = c.channels;
}

void sat_resnet_build_params(const sat_config& c, const Dims& D, std::vector<ParamDesc>& P,
                             size_t* n_total) {
  P.clear();
  size_t off = 0;
  const int w = c.res_width;
  add_param(P, off, "stem.conv.w", w, 49L * c.channels, -1, 0);
  add_param(P, off, "stem.bn.g", w, 1, -1, 2);
  add_param(P, off, "stem.bn.b", w, 1, -1, 1);
  for (const RBlock& b : block_table(c, pool_hw(c))) {
    const std::string p = "b" + std::to_string(b.idx) + ".";
    add_param(P, off, p + "conv1.w", b.mid, b.cin, b.idx, 0);
    add_param(P, off, p + "bn1.g", b.mid, 1, b.idx, 2);
    add_param(P, off, p + "bn1.b", b.mid, 1, b.idx, 1);
    add_param(P, off, p + "conv2.w", b.mid, 9L * b.mid, b.idx, 0);
    add_param(P, off, p + "bn2.g", b.mid, 1, b.idx, 2);
    add_param(P, off, p + "bn2.b", b.mid, 1, b.idx, 1);
    add_param(P, off, p + "conv3.w", b.cout, b.mid, b.idx, 0);
    add_param(P, off, p + "bn3.g", b.cout, 1, b.idx, 2);
    add_param(P, off, p + "bn3.b", b.cout, 1, b.idx, 1);
    if (b.proj) {
      add_param(P, off, p + "down.w", b.cout, b.cin, b.idx, 0);
      add_param(P, off, p + "down.bn.g", b.cout, 1, b.idx, 2);
      add_param(P, off, p + "down.bn.b", b.cout, 1, b.idx, 1);
    }
  }
  add_param(P, off, "fc.w", D.V, D.d, D.L, 0);
  add_param(P, off, "fc.b", D.V, 1, D.L, 1);
  for (auto& p : P) p.trainable = (p.group < 0) ? (D.k == 0) : (p.group >= D.k);
  // transposed copies of the trainable weights of blocks and head (B operand
  // of every input-gradient product); the stem's input gradient is never formed
  size_t toff = 0;
  for (auto& p : P) {
    if (!p.trainable || p.group < 0 || p.cols == 1) continue;
    p.trows = p.name == "fc.w" ? D.Vp : p.rows;
    p.toff = toff;
    toff = align_up(toff + (size_t)p.trows * p.cols, 64);
  }
  // Zero tail: the transposed copy of the head weight covers the padded class
  // count, so its refresh reads up to 7 rows past the last weight matrix.
  *n_total = align_up(off + 8L * D.d, 64);
}

// Lays out the ResNet activations and workspace after the parameter sections.
void sat_resnet_carve(sat_model* M, SatCarver& c) {
  if (!M->rn) M->rn = std::make_shared<ResNetPlan>();
  ResNetPlan& R = *M->rn;
  const sat_config& cfg = M->cfg;
  const Dims& D = M->D;
  R.N = cfg.batch;
  R.C = cfg.channels;
  R.img = cfg.img_size;
  R.width = cfg.res_width;
  R.classes = D.V;
  R.Vp = D.Vp;
  R.F = D.d;
  R.Hs = stem_hw(cfg);
  R.Hp = pool_hw(cfg);
  R.Ps = (long)R.N * R.Hs * R.Hs;
  R.Pp = (long)R.N * R.Hp * R.Hp;
  R.stem_kp = (int)align_up(49 * R.C, 8);
  R.blocks = block_table(cfg, R.Hp);
  // parameter indices
  {
    int i = 0;
    R.stem_w = i;
    R.stem_n.g = i + 1;
    i += 3;
    for (RBlock& b : R.blocks) {
      b.w1 = i;
      b.n1.g = i + 1;
      b.w2 = i + 3;
      b.n2.g = i + 4;
      b.w3 = i + 6;
      b.n3.g = i + 7;
      i += 9;
      if (b.proj) {
        b.wd = i;
        b.nd.g = i + 1;
        i += 3;
      }
    }
    R.fc_w = i;
  }
  R.Hf = R.blocks.back().Ho;
  const int nb = (int)R.blocks.size();
  R.x.assign(nb + 1, nullptr);
  R.xb.assign(nb + 1, nullptr);
  R.x_rows.assign(nb + 1, 0);
  R.x_cols.assign(nb + 1, 0);
  long maxPC = R.Ps * R.width, col = R.Ps * R.stem_kp, dcol = 0, part = 0;
  auto bnp = [&](long P, int C) { part = std::max(part, 2L * bn_parts(P, C) * C); };
  bnp(R.Ps, R.width);
  // stem
  R.stem_c = c.take<float>(R.Ps * R.width);
  R.stem_act = c.take<float>(R.Ps * R.width);
  R.stem_n.mean = c.take<float>(R.width);
  R.stem_n.rstd = c.take<float>(R.width);
  R.pool_arg = c.take<uint8_t>(R.Pp * R.width);
  R.stem_wpad = c.take<bf16>((long)R.width * R.stem_kp);
  for (int i = 0; i <= nb; ++i) {
    const long P = i < nb ? R.blocks[i].Pin : R.blocks[nb - 1].Pout;
    const int C = i < nb ? R.blocks[i].cin : R.blocks[nb - 1].cout;
    R.x_rows[i] = P;
    R.x_cols[i] = C;
    R.x[i] = c.take<float>(P * C);
    R.xb[i] = c.take<bf16>(P * C);
    maxPC = std::max(maxPC, P * C);
  }
  for (RBlock& b : R.blocks) {
    b.c1 = c.take<float>(b.Pin * b.mid);
    b.a1 = c.take<bf16>(b.Pin * b.mid);
    b.c2 = c.take<float>(b.Pout * b.mid);
    b.a2 = c.take<bf16>(b.Pout * b.mid);
    b.c3 = c.take<float>(b.Pout * b.cout);
    if (b.proj) b.cd = c.take<float>(b.Pout * b.cout);
    for (RBn* n : {&b.n1, &b.n2, &b.n3, &b.nd}) {
      if (n == &b.nd && !b.proj) continue;
      const int C = (n == &b.n1 || n == &b.n2) ? b.mid : b.cout;
      n->mean = c.take<float>(C);
      n->rstd = c.take<float>(C);
    }
    maxPC = std::max({maxPC, b.Pin * b.mid, b.Pout * b.cout, b.Pout * b.cin});
    col = std::max(col, b.Pout * 9L * b.mid);
    dcol = std::max(dcol, b.Pout * 9L * b.mid);
    if (b.stride != 1) col = std::max(col, b.Pout * (long)b.cin);
    bnp(b.Pin, b.mid);
    bnp(b.Pout, b.mid);
    bnp(b.Pout, b.cout);
  }
  R.col = c.take<bf16>(col);
  R.feat = c.take<bf16>((long)R.N * R.F);
  // head
  M->logits = c.take<float>((long)R.N * R.Vp);
  M->dz = c.take<bf16>((long)R.N * R.Vp);
  M->row_loss = c.take<float>(R.N);
  M->scal = c.take<float>(8);
  // backward
  R.g0 = c.take<float>(maxPC);
  R.g1 = c.take<float>(maxPC);
  R.gdo = c.take<float>(maxPC);
  R.da = c.take<float>(maxPC);
  R.dsub = c.take<float>(maxPC);
  R.dcol = c.take<float>(std::max(dcol, 8L));
  R.dc = c.take<bf16>(maxPC);
  R.dcd = c.take<bf16>(maxPC);
  R.tA = c.take<bf16>(maxPC);
  R.tB = c.take<bf16>(std::max(col, maxPC));
  R.dfeat = c.take<float>((long)R.N * R.F);
  // column sums of the head bias gradient use the same partial buffer
  part = std::max(part, 2L * std::min(R.N, 256) * R.Vp);
  R.part = c.take<float>(part);
  M->part = R.part;
  // split-K workspace: the pixel-long weight-gradient products and the head
  long ws = gemm_splitk_ws_elems(R.N, R.classes, R.F);
  auto wneed = [&](int Mr, int Nc, long K) {
    ws = std::max(ws, gemm_splitk_ws_elems(Mr, Nc, (int)K, kSplitMax));
  };
  wneed(R.width, R.stem_kp, R.Ps);
  for (const RBlock& b : R.blocks) {
    wneed(b.mid, b.cin, b.Pin);
    wneed(b.mid, 9 * b.mid, b.Pout);
    wneed(b.cout, b.mid, b.Pout);
    if (b.proj) wneed(b.cout, b.cin, b.Pout);
  }
  M->splitk_ws_elems = ws;
  M->splitk_ws = ws > 0 ? c.take<float>(ws) : nullptr;
  // activations readable through sat_activation_read
  M->h_in = R.x;
  M->act_rows = R.x_rows;
  M->act_cols = R.x_cols;
}

double sat_resnet_flops(const Dims& D) {
  // 2 FLOPs per multiply-add of every forward convolution and the head,
  // twice that again for the input- and weight-gradient products of the
  // trainable part; a trainable stem adds its weight gradient only
  sat_config c;
  memset(&c, 0, sizeof c);
  for (int s = 0; s < 4; ++s) c.res_blocks[s] = D.res_blocks[s];
  c.res_width = D.res_width;
  c.img_size = D.img;
  c.channels = D.channels;
  c.batch = D.B;
  const double B = D.B;
  const int Hs = stem_hw(c);
  const double stem = 2.0 * B * Hs * Hs * 49.0 * D.channels * D.res_width;
  double fwd = stem, bwd = 0.0;
  for (const RBlock& b : block_table(c, pool_hw(c))) {
    const double f = 2.0 * (b.Pin * (double)b.cin * b.mid + b.Pout * 9.0 * b.mid * b.mid +
                            b.Pout * (double)b.mid * b.cout +
                            (b.proj ? b.Pout * (double)b.cin * b.cout : 0.0));
    fwd += f;
    if (b.idx >= D.k) bwd += 2.0 * f;
  }
  const double head = 2.0 * B * D.d * D.V;
  return fwd + head + bwd + 2.0 * head + (D.k == 0 ? stem : 0.0);
}

namespace {

const float* gam(const sat_model* M, const RBn& n) { return master(M, n.g); }
const float* bet(const sat_model* M, const RBn& n) { return master(M, n.g + 1); }

// out[Pout, cout] fp32 = A[Pout, Kc] (bf16, row pitch lda) times weight w.
sat_status conv_gemm(sat_model* M, const bf16* A, long lda, int w, long P, int cout, int Kc,
                     float* out, int tk = TK_ALL_GEMM) {
  GemmArgs a = gargs(A, lda, shadow(M, w), Kc, (int)P, cout, Kc, out, cout);
  return gemm(M, a, LAY_K, LAY_K, EPI_F32, tk);
}

// Weight gradient [cout, ncols] = dY^T X over P pixels (dY [P, cout] bf16;
// X [P, >= ncols] bf16 with row pitch ldx): on token-contiguous copies of both
// operands (xcols columns of X transposed) so the product splits K, else
// straight on the row-major operands.
sat_status rwgrad(sat_model* M, const bf16* dY, int cout, const bf16* X, long ldx, int ncols,
                  int xcols, long P, float* out) {
  ResNetPlan& R = *M->rn;
  if (P % 8 == 0 && cout % 8 == 0 && xcols % 8 == 0 && ldx % 8 == 0) {
    SAT_HIP(launch_transpose_bf16(dY, cout, R.tA, P, (int)P, cout, M->stream));
    SAT_HIP(launch_transpose_bf16(X, ldx, R.tB, P, (int)P, xcols, M->stream));
    GemmArgs w = gargs(R.tA, P, R.tB, P, cout, ncols, (int)P, out, ncols);
    w.splitk_max = kSplitMax;
    return gemm(M, w, LAY_K, LAY_K, EPI_F32);
  }
  GemmArgs w = gargs(dY, cout, X, ldx, cout, ncols, (int)P, out, ncols);
  return gemm(M, w, LAY_MN, LAY_MN, EPI_F32);
}

// dX [P, n] fp32 = dY [P, cout] (bf16) times weight w [cout, n] (through its
// transposed copy); resid (may equal out) is added when not null.
// The same with X already token-contiguous: XT [ncols, P] (row stride P).
sat_status rwgrad_t(sat_model* M, const bf16* dY, int cout, const bf16* XT, int ncols, long P,
                    float* out) {
  ResNetPlan& R = *M->rn;
  SAT_HIP(launch_transpose_bf16(dY, cout, R.tA, P, (int)P, cout, M->stream));
  GemmArgs w = gargs(R.tA, P, XT, P, cout, ncols, (int)P, out, ncols);
  w.splitk_max = kSplitMax;
  return gemm(M, w, LAY_K, LAY_K, EPI_F32);
}

sat_status dgrad(sat_model* M, const bf16* dY, int cout, int w, long P, int n, float* out,
                 const float* resid) {
  const ParamDesc& p = M->params[w];
  GemmArgs a = gargs(dY, cout, shadow_t(M, w), p.trows, (int)P, n, cout, out, n);
  if (resid) {
    a.resid = resid;
    a.ldr = n;
    return gemm(M, a, LAY_K, LAY_K, EPI_RESID_F32);
  }
  return gemm(M, a, LAY_K, LAY_K, EPI_F32);
}

}  // namespace

sat_status sat_resnet_forward(sat_model* M, const void* inputs, const int32_t* labels) {
  ResNetPlan& R = *M->rn;
  hipStream_t s = M->stream;
  const float eps = M->cfg.ln_eps;
  // stem: 7 x 7 / 2 convolution, BN, ReLU, 3 x 3 / 2 max pool
  SAT_HIP(launch_im2col_nchw((const float*)inputs, R.col, R.stem_kp, R.N, R.C, R.img, R.img, 7, 2, 3,
                             R.Hs, R.Hs, s));
  SAT_HIP(launch_pad_cols_bf16(shadow(M, R.stem_w), R.width, 49 * R.C, R.stem_wpad, R.stem_kp, s));
  {
    GemmArgs a = gargs(R.col, R.stem_kp, R.stem_wpad, R.stem_kp, (int)R.Ps, R.width, R.stem_kp,
                       R.stem_c, R.width);
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_F32));
  }
  SAT_HIP(launch_bn_stats(R.stem_c, R.Ps, R.width, eps, R.part, R.stem_n.mean, R.stem_n.rstd, s));
  SAT_HIP(launch_bn_apply(R.stem_c, R.Ps, R.width, R.stem_n.mean, R.stem_n.rstd, gam(M, R.stem_n),
                          bet(M, R.stem_n), 1, nullptr, R.stem_act, s));
  SAT_HIP(launch_maxpool_fwd(R.stem_act, R.N, R.Hs, R.Hs, R.width, R.Hp, R.Hp, R.x[0], R.xb[0],
                             R.pool_arg, s));
  // blocks
  for (size_t i = 0; i < R.blocks.size(); ++i) {
    RBlock& b = R.blocks[i];
    TRY(conv_gemm(M, R.xb[i], b.cin, b.w1, b.Pin, b.mid, b.cin, b.c1));
    SAT_HIP(launch_bn_stats(b.c1, b.Pin, b.mid, eps, R.part, b.n1.mean, b.n1.rstd, s));
    SAT_HIP(launch_bn_apply(b.c1, b.Pin, b.mid, b.n1.mean, b.n1.rstd, gam(M, b.n1), bet(M, b.n1), 1,
                            b.a1, nullptr, s));
    SAT_HIP(launch_im2col(b.a1, R.col, 9L * b.mid, R.N, b.H, b.W, b.mid, 3, b.stride, 1, b.Ho, b.Wo,
                          s));
    TRY(conv_gemm(M, R.col, 9L * b.mid, b.w2, b.Pout, b.mid, 9 * b.mid, b.c2, TK_QKV_FWD));
    SAT_HIP(launch_bn_stats(b.c2, b.Pout, b.mid, eps, R.part, b.n2.mean, b.n2.rstd, s));
    SAT_HIP(launch_bn_apply(b.c2, b.Pout, b.mid, b.n2.mean, b.n2.rstd, gam(M, b.n2), bet(M, b.n2), 1,
                            b.a2, nullptr, s));
    TRY(conv_gemm(M, b.a2, b.mid, b.w3, b.Pout, b.cout, b.mid, b.c3));
    SAT_HIP(launch_bn_stats(b.c3, b.Pout, b.cout, eps, R.part, b.n3.mean, b.n3.rstd, s));
    if (b.proj) {
      const bf16* sub = R.xb[i];
      if (b.stride != 1) {
        SAT_HIP(launch_im2col(R.xb[i], R.col, b.cin, R.N, b.H, b.W, b.cin, 1, b.stride, 0, b.Ho,
                              b.Wo, s));
        sub = R.col;
      }
      TRY(conv_gemm(M, sub, b.cin, b.wd, b.Pout, b.cout, b.cin, b.cd));
      SAT_HIP(launch_bn_stats(b.cd, b.Pout, b.cout, eps, R.part, b.nd.mean, b.nd.rstd, s));
      SAT_HIP(launch_bn_add_relu(b.c3, b.n3.mean, b.n3.rstd, gam(M, b.n3), bet(M, b.n3), b.cd,
                                 b.nd.mean, b.nd.rstd, gam(M, b.nd), bet(M, b.nd), b.Pout, b.cout,
                                 R.x[i + 1], R.xb[i + 1], s));
    } else {
      SAT_HIP(launch_bn_add_relu(b.c3, b.n3.mean, b.n3.rstd, gam(M, b.n3), bet(M, b.n3), R.x[i],
                                 nullptr, nullptr, nullptr, nullptr, b.Pout, b.cout, R.x[i + 1],
                                 R.xb[i + 1], s));
    }
  }
  // head: global average pool, linear layer, cross-entropy
  const int nb = (int)R.blocks.size();
  SAT_HIP(launch_avgpool_fwd(R.x[nb], R.N, R.Hf * R.Hf, R.F, R.feat, s));
  {
    GemmArgs a = gargs(R.feat, R.F, shadow(M, R.fc_w), R.F, R.N, R.classes, R.F, M->logits, R.Vp);
    a.bias = master(M, R.fc_w + 1);
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_F32));
  }
  SAT_HIP(launch_count_valid(labels, R.N, M->scal + 1, s));
  {
    Timed tm(M, TK_XENT, (double)R.N * R.classes * 6.0);
    SAT_HIP(launch_xent(M->logits, R.Vp, labels, R.N, R.classes, M->row_loss, M->dz, R.Vp,
                        M->scal + 1, s));
  }
  SAT_HIP(launch_loss_finalize(M->row_loss, R.N, M->scal + 1, M->scal, s));
  return SAT_OK;
}

sat_status sat_resnet_backward(sat_model* M, const void* inputs) {
  ResNetPlan& R = *M->rn;
  hipStream_t s = M->stream;
  const int k = M->D.k;
  const int nb = (int)R.blocks.size();
  // head: dfeat = dz W, dW = dz^T feat, db = column sums of dz
  {
    const ParamDesc& p = M->params[R.fc_w];
    GemmArgs a = gargs(M->dz, R.Vp, shadow_t(M, R.fc_w), p.trows, R.N, R.F, R.classes, R.dfeat, R.F);
    TRY(gemm(M, a, LAY_K, LAY_K, EPI_F32));
    GemmArgs w = gargs(M->dz, R.Vp, R.feat, R.F, R.classes, R.F, R.N, grad(M, R.fc_w), R.F);
    TRY(gemm(M, w, LAY_MN, LAY_MN, EPI_F32));
    SAT_HIP(launch_colsum_bf16(M->dz, R.Vp, R.N, R.classes, R.part, R.N < 256 ? R.N : 256,
                               grad(M, R.fc_w + 1), s));
  }
  SAT_HIP(launch_avgpool_bwd(R.dfeat, R.N, R.Hf * R.Hf, R.F, R.g0, s));
  float* dy = R.g0;
  float* dx = R.g1;
  for (int i = nb - 1; i >= k; --i) {
    const RBlock& b = R.blocks[i];
    // through the ReLU after the shortcut add, then BN3 (and the projection's BN)
    SAT_HIP(launch_relu_mask(dy, R.x[i + 1], b.Pout * b.cout, R.gdo, s));
    SAT_HIP(launch_bn_bwd(R.gdo, 0, nullptr, b.c3, b.n3.mean, b.n3.rstd, gam(M, b.n3), b.Pout, b.cout,
                          R.part, grad(M, b.n3.g), grad(M, b.n3.g + 1), R.dc, s));
    if (b.proj)
      SAT_HIP(launch_bn_bwd(R.gdo, 0, nullptr, b.cd, b.nd.mean, b.nd.rstd, gam(M, b.nd), b.Pout,
                            b.cout, R.part, grad(M, b.nd.g), grad(M, b.nd.g + 1), R.dcd, s));
    // conv3 (1 x 1)
    TRY(dgrad(M, R.dc, b.cout, b.w3, b.Pout, b.mid, R.da, nullptr));
    TRY(rwgrad(M, R.dc, b.cout, b.a2, b.mid, b.mid, b.mid, b.Pout, grad(M, b.w3)));
    SAT_HIP(launch_bn_bwd(R.da, 1, b.a2, b.c2, b.n2.mean, b.n2.rstd, gam(M, b.n2), b.Pout, b.mid,
                          R.part, grad(M, b.n2.g), grad(M, b.n2.g + 1), R.dc, s));
    // conv2 (3 x 3, the block's stride): input gradient through col2im, weight
    // gradient against the im2col matrix rebuilt from a1
    TRY(dgrad(M, R.dc, b.mid, b.w2, b.Pout, 9 * b.mid, R.dcol, nullptr));
    SAT_HIP(launch_col2im(R.dcol, 9L * b.mid, R.da, R.N, b.H, b.W, b.mid, 3, b.stride, 1, b.Ho, b.Wo,
                          0, s));
    // (the im2col matrix written token-contiguous when the shapes allow)
    if (b.Pout % 8 == 0 && b.mid % 8 == 0) {
      SAT_HIP(launch_im2col_t(b.a1, R.tB, b.Pout, R.N, b.H, b.W, b.mid, 3, b.stride, 1, b.Ho, b.Wo, s));
      TRY(rwgrad_t(M, R.dc, b.mid, R.tB, 9 * b.mid, b.Pout, grad(M, b.w2)));
    } else {
      SAT_HIP(launch_im2col(b.a1, R.col, 9L * b.mid, R.N, b.H, b.W, b.mid, 3, b.stride, 1, b.Ho, b.Wo,
                            s));
      TRY(rwgrad(M, R.dc, b.mid, R.col, 9L * b.mid, 9 * b.mid, 9 * b.mid, b.Pout, grad(M, b.w2)));
    }
    SAT_HIP(launch_bn_bwd(R.da, 1, b.a1, b.c1, b.n1.mean, b.n1.rstd, gam(M, b.n1), b.Pin, b.mid,
                          R.part, grad(M, b.n1.g), grad(M, b.n1.g + 1), R.dc, s));
    // conv1 (1 x 1) and the shortcut; the input gradient only when something
    // below this block trains
    const bool need_dx = i > k || k == 0;
    if (need_dx) TRY(dgrad(M, R.dc, b.mid, b.w1, b.Pin, b.cin, dx, b.proj ? nullptr : R.gdo));
    TRY(rwgrad(M, R.dc, b.mid, R.xb[i], b.cin, b.cin, b.cin, b.Pin, grad(M, b.w1)));
    if (b.proj) {
      if (b.stride != 1) {
        if (need_dx) {
          TRY(dgrad(M, R.dcd, b.cout, b.wd, b.Pout, b.cin, R.dsub, nullptr));
          SAT_HIP(launch_stride2_add(R.dsub, R.N, b.Ho, b.Wo, b.cin, b.H, b.W, dx, s));
        }
        // the every-other-pixel subsample, token-contiguous when the shapes allow
        if (b.Pout % 8 == 0 && b.cin % 8 == 0) {
          SAT_HIP(launch_im2col_t(R.xb[i], R.tB, b.Pout, R.N, b.H, b.W, b.cin, 1, b.stride, 0, b.Ho,
                                  b.Wo, s));
          TRY(rwgrad_t(M, R.dcd, b.cout, R.tB, b.cin, b.Pout, grad(M, b.wd)));
        } else {
          SAT_HIP(launch_im2col(R.xb[i], R.col, b.cin, R.N, b.H, b.W, b.cin, 1, b.stride, 0, b.Ho,
                                b.Wo, s));
          TRY(rwgrad(M, R.dcd, b.cout, R.col, b.cin, b.cin, b.cin, b.Pout, grad(M, b.wd)));
        }
      } else {
        if (need_dx) TRY(dgrad(M, R.dcd, b.cout, b.wd, b.Pout, b.cin, dx, dx));
        TRY(rwgrad(M, R.dcd, b.cout, R.xb[i], b.cin, b.cin, b.cin, b.Pout, grad(M, b.wd)));
      }
    }
    std::swap(dy, dx);
  }
  if (k > 0) return SAT_OK;
  // stem: max pool, ReLU + BN, weight gradient against the rebuilt columns
  SAT_HIP(launch_maxpool_bwd(dy, R.pool_arg, R.N, R.Hs, R.Hs, R.width, R.Hp, R.Hp, dx, s));
  SAT_HIP(launch_bn_bwd(dx, 2, R.stem_act, R.stem_c, R.stem_n.mean, R.stem_n.rstd, gam(M, R.stem_n),
                        R.Ps, R.width, R.part, grad(M, R.stem_n.g), grad(M, R.stem_n.g + 1), R.dc, s));
  SAT_HIP(launch_im2col_nchw((const float*)inputs, R.col, R.stem_kp, R.N, R.C, R.img, R.img, 7, 2, 3,
                             R.Hs, R.Hs, s));
  // over the zero-padded columns (whole 4-column output vectors, so the
  // product splits K), then the 7 x 7 x C columns into the gradient arena
  TRY(rwgrad(M, R.dc, R.width, R.col, R.stem_kp, R.stem_kp, R.stem_kp, R.Ps, R.dsub));
  SAT_HIP(hipMemcpy2DAsync(grad(M, R.stem_w), (size_t)49 * R.C * 4, R.dsub, (size_t)R.stem_kp * 4,
                           (size_t)49 * R.C * 4, R.width, hipMemcpyDeviceToDevice, s));
  return SAT_OK;
}
