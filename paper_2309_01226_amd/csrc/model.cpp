// Model runtime: configuration checks, the per-model arena layout, parameter
// table, and the forward / backward / AdamW launch sequence of one
// fine-tuning step on the model's HIP stream.
//
// Arena (one per model, caller-provided or owned):
//   fp32 master parameters | bf16 shadow | bf16 transposed weights (trainable
//   matrices of dX = dY W) | fp32 gradients | fp32 m | fp32 v | activations
//   saved for backward | backward workspace.
// Parameters run bottom to top (embeddings, blocks 0..L-1, final LN, head),
// so the tensors frozen by k > 0 form a prefix and AdamW is a single flat
// kernel over the trainable suffix; frozen gradients and moments are never
// written.  Blocks below k share one scratch activation set.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

#include "../../include/saturn.h"
#include "abi_common.h"
#include "kernels.h"
#include "model.h"

bool attention_supports_dh(int dh);

namespace {

constexpr size_t kAlignElems = 64;  // parameter offsets (elements)
constexpr size_t kAlignBytes = 256; // arena sections

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

// ------------------------------------------------------------------ config

sat_status sat_validate_config(const sat_config* c) {
  SAT_CHECK_ARG(c != nullptr, "null config");
  SAT_CHECK_ARG(c->struct_size == sizeof(sat_config), "struct_size %u != sizeof(sat_config) %zu",
                c->struct_size, sizeof(sat_config));
  SAT_CHECK_ARG(c->arch >= SAT_GPT2 && c->arch <= SAT_RESNET, "unknown arch %d", c->arch);
  if (c->arch == SAT_RESNET) return sat_resnet_validate(c);
  for (int s = 0; s < 4; ++s)
    SAT_CHECK_ARG(c->res_blocks[s] == 0, "res_blocks must be 0 for transformer architectures");
  SAT_CHECK_ARG(c->n_layers >= 1, "n_layers must be >= 1");
  SAT_CHECK_ARG(c->d_model >= 8 && c->d_model % 8 == 0 && c->d_model <= 4096,
                "d_model must be a multiple of 8 in [8, 4096]");
  SAT_CHECK_ARG(c->n_heads >= 1 && c->d_model % c->n_heads == 0, "d_model %% n_heads != 0");
  int dh = c->d_model / c->n_heads;
  SAT_CHECK_ARG(attention_supports_dh(dh), "head dim %d not in {16, 32, 64, 80, 128, 256}", dh);
  SAT_CHECK_ARG(c->d_mlp >= 8 && c->d_mlp % 8 == 0, "d_mlp must be a positive multiple of 8");
  SAT_CHECK_ARG(c->vocab >= 2, "vocab / classes must be >= 2");
  SAT_CHECK_ARG(c->batch >= 1, "batch must be >= 1");
  SAT_CHECK_ARG(c->frozen_layers >= 0 && c->frozen_layers <= c->n_layers,
                "frozen_layers %d not in [0, n_layers]", c->frozen_layers);
  SAT_CHECK_ARG(c->checkpoint == 0 || c->checkpoint == 1, "checkpoint must be 0 or 1");
  SAT_CHECK_ARG(c->lr >= 0.f && c->beta1 >= 0.f && c->beta1 < 1.f && c->beta2 >= 0.f &&
                    c->beta2 < 1.f && c->eps > 0.f && c->weight_decay >= 0.f,
                "invalid AdamW hyper-parameters");
  SAT_CHECK_ARG(c->ln_eps > 0.f && c->init_std >= 0.f, "invalid ln_eps / init_std");
  if (c->arch == SAT_VIT) {
    SAT_CHECK_ARG(c->patch >= 1 && c->img_size >= c->patch && c->img_size % c->patch == 0,
                  "img_size must be a positive multiple of patch");
    SAT_CHECK_ARG(c->channels >= 1, "channels must be >= 1");
    SAT_CHECK_ARG(c->rotary_dim == 0, "rotary_dim must be 0 for VIT");
  } else {
    SAT_CHECK_ARG(c->seq_len >= 1, "seq_len must be >= 1");
    if (c->arch == SAT_GPTJ)
      SAT_CHECK_ARG(c->rotary_dim >= 0 && c->rotary_dim % 2 == 0 && c->rotary_dim <= dh,
                    "rotary_dim must be even and <= head dim");
    else
      SAT_CHECK_ARG(c->rotary_dim == 0, "rotary_dim must be 0 for GPT2");
    SAT_CHECK_ARG(c->frozen_layers > 0 || c->vocab < 65536,
                  "training the token embedding needs vocab < 65536");
  }
  return SAT_OK;
}

// ------------------------------------------------------------------ layout

void sat_model_dims(const sat_config& c, Dims* d) {
  if (c.arch == SAT_RESNET) {
    sat_resnet_dims(c, d);
    return;
  }
  memset(d, 0, sizeof *d);
  d->arch = c.arch;
  d->L = c.n_layers;
  d->d = c.d_model;
  d->H = c.n_heads;
  d->dh = c.d_model / c.n_heads;
  d->m = c.d_mlp;
  d->V = c.vocab;
  d->Vp = (int)align_up(c.vocab, 8);
  d->B = c.batch;
  d->k = c.frozen_layers;
  d->rd = c.rotary_dim;
  if (c.arch == SAT_VIT) {
    int g = c.img_size / c.patch;
    d->np = g * g;
    d->pd = c.channels * c.patch * c.patch;
    d->pdp = (d->pd + 7) / 8 * 8;
    d->S = d->np + 1;
  } else {
    d->np = 0;
    d->pd = 0;
    d->pdp = 0;
    d->S = c.seq_len;
  }
  d->T = d->B * d->S;
  d->rows_head = (c.arch == SAT_VIT) ? d->B : d->T;
  d->qkv_ld = (c.arch == SAT_GPTJ) ? 3 * d->d + d->m : 3 * d->d;
  d->ckpt = c.checkpoint != 0;
}

static void add_param(std::vector<ParamDesc>& P, size_t& off, const std::string& name, long rows,
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
  off = align_up(off + (size_t)rows * cols, kAlignElems);
}

// kind: 0 = normal init, 1 = zeros (bias), 2 = ones (LN gain)
void sat_build_params(const sat_config& c, const Dims& D, std::vector<ParamDesc>& P,
                      size_t* n_total) {
  if (c.arch == SAT_RESNET) {
    sat_resnet_build_params(c, D, P, n_total);
    return;
  }
  P.clear();
  size_t off = 0;
  const int d = D.d, m = D.m;
  if (c.arch == SAT_VIT) {
    add_param(P, off, "patch.w", d, D.pd, -1, 0);
    add_param(P, off, "patch.b", d, 1, -1, 1);
    add_param(P, off, "cls", d, 1, -1, 0);
    add_param(P, off, "pos", D.S, d, -1, 0);
  } else {
    add_param(P, off, "wte", D.V, d, -1, 0);
    if (c.arch == SAT_GPT2) add_param(P, off, "wpe", D.S, d, -1, 0);
  }
  for (int l = 0; l < D.L; ++l) {
    std::string p = "h" + std::to_string(l) + ".";
    if (c.arch == SAT_GPTJ) {
      add_param(P, off, p + "ln1.g", d, 1, l, 2);
      add_param(P, off, p + "ln1.b", d, 1, l, 1);
      add_param(P, off, p + "attn.qkv.w", 3 * d, d, l, 0);
      add_param(P, off, p + "mlp.fc1.w", m, d, l, 0);  // contiguous with attn.qkv.w
      add_param(P, off, p + "mlp.fc1.b", m, 1, l, 1);
      add_param(P, off, p + "attn.proj.w", d, d, l, 0);
      add_param(P, off, p + "mlp.fc2.w", d, m, l, 0);
      add_param(P, off, p + "mlp.fc2.b", d, 1, l, 1);
    } else {
      add_param(P, off, p + "ln1.g", d, 1, l, 2);
      add_param(P, off, p + "ln1.b", d, 1, l, 1);
      add_param(P, off, p + "attn.qkv.w", 3 * d, d, l, 0);
      add_param(P, off, p + "attn.qkv.b", 3 * d, 1, l, 1);
      add_param(P, off, p + "attn.proj.w", d, d, l, 0);
      add_param(P, off, p + "attn.proj.b", d, 1, l, 1);
      add_param(P, off, p + "ln2.g", d, 1, l, 2);
      add_param(P, off, p + "ln2.b", d, 1, l, 1);
      add_param(P, off, p + "mlp.fc1.w", m, d, l, 0);
      add_param(P, off, p + "mlp.fc1.b", m, 1, l, 1);
      add_param(P, off, p + "mlp.fc2.w", d, m, l, 0);
      add_param(P, off, p + "mlp.fc2.b", d, 1, l, 1);
    }
  }
  add_param(P, off, "lnf.g", d, 1, D.L, 2);
  add_param(P, off, "lnf.b", d, 1, D.L, 1);
  add_param(P, off, "head.w", D.V, d, D.L, 0);
  if (c.arch != SAT_GPT2) add_param(P, off, "head.b", D.V, 1, D.L, 1);
  for (auto& p : P) p.trainable = (p.group < 0) ? (D.k == 0) : (p.group >= D.k);
  // Transposed copies for the input-gradient products of trainable blocks and
  // of the head (B operand of dX = dY W, read along W's rows).
  size_t toff = 0;
  auto ends_with = [](const std::string& a, const char* b) {
    const size_t n = strlen(b);
    return a.size() >= n && a.compare(a.size() - n, n, b) == 0;
  };
  for (auto& p : P) {
    if (!p.trainable || p.group < 0) continue;
    long trows = 0;
    if (ends_with(p.name, "attn.qkv.w")) trows = c.arch == SAT_GPTJ ? D.qkv_ld : p.rows;
    else if (ends_with(p.name, "attn.proj.w") || ends_with(p.name, "mlp.fc2.w")) trows = p.rows;
    else if (ends_with(p.name, "mlp.fc1.w") && c.arch != SAT_GPTJ) trows = p.rows;
    else if (p.name == "head.w") trows = D.Vp;
    if (trows == 0) continue;
    p.toff = toff;
    p.trows = trows;
    toff = align_up(toff + (size_t)trows * p.cols, kAlignElems);
  }
  // Zero tail: the head's input-gradient product reads up to 7 rows past the
  // last weight matrix when the vocabulary is not a multiple of 8.
  off = align_up(off + (size_t)8 * (d > m ? d : m), kAlignElems);
  *n_total = off;
}

namespace {

// Whether the weight-gradient product of a [rows, cols] weight (K = k
// token-contiguous rows) runs in the 256 x 256 kernel, so that its AdamW step
// can be fused into the product's epilogue: enough tiles for every CU, whole
// 8-column vectors, and the transposed copy in pieces of 8 rows.  The operand
// and parameter sections are 256-byte aligned by construction.
bool fused_opt_ok(long rows, long cols, long trows, long k) {
  return k % 8 == 0 && cols % 8 == 0 && trows % 8 == 0 && trows >= rows &&
         ((rows + 255) / 256) * ((cols + 255) / 256) >= 256;
}

// AdamW segments over the trainable suffix: one matrix segment per weight
// with a transposed copy (the GPT-J q|k|v weight and the fc1 weight after it
// form one), flat segments for everything between them (biases, LN
// parameters, embeddings, alignment gaps and the arena's zero tail).  The
// full table serves the unfused optimizer; the rest table leaves out the
// matrices whose update is fused into their weight-gradient products.
void build_segments(sat_model* M) {
  const Dims& D = M->D;
  auto& P = M->params;
  for (auto& p : P) p.fused_opt = false;
  auto build = [&](bool skip_fused, std::vector<AdamWSeg>& segs, int& blocks, double& bytes) {
    segs.clear();
    blocks = 0;
    bytes = 0.0;
    auto push = [&](AdamWSeg g) {
      g.first_block = blocks;
      blocks += adamw_seg_blocks(g);
      segs.push_back(g);
      // 30 bytes per element (fp32 p, g, m, v read; p, m, v, bf16 copy
      // written), 2 per element of a transposed copy
      bytes += 30.0 * (double)g.rows * (g.toff < 0 ? 1 : g.cols) +
               (g.toff < 0 ? 0.0 : 2.0 * (double)g.trows * g.cols);
    };
    auto flat = [&](size_t a, size_t b) {
      while (a < b) {  // pieces below 2^31 elements
        const size_t n = std::min<size_t>(b - a, (size_t)1 << 30);
        push(AdamWSeg{(int64_t)a, -1, (int32_t)n, 0, 0, 0});
        a += n;
      }
    };
    size_t cur = M->n_param_elems;  // first trainable element
    for (const auto& p : P)
      if (p.trainable) cur = std::min(cur, p.off);
    for (size_t i = 0; i < P.size(); ++i) {
      ParamDesc& p = P[i];
      if (!p.trainable || p.toff == SIZE_MAX || p.off < cur) continue;
      long rows = p.rows;
      // parameters stored right after it with the same width belong to the block
      for (size_t j = i + 1; j < P.size() && rows < p.trows; ++j) {
        if (P[j].cols != p.cols || P[j].off != p.off + (size_t)rows * p.cols) break;
        rows += P[j].rows;
      }
      flat(cur, p.off);
      const long k = p.group == D.L ? D.rows_head : D.T;
      p.fused_opt = D.arch != SAT_RESNET && fused_opt_ok(rows, p.cols, p.trows, k);
      if (!(skip_fused && p.fused_opt))
        push(AdamWSeg{(int64_t)p.off, (int64_t)p.toff, (int32_t)rows, (int32_t)p.trows,
                      (int32_t)p.cols, 0});
      cur = p.off + (size_t)rows * p.cols;
    }
    flat(cur, M->n_param_elems);
  };
  build(false, M->segs, M->seg_blocks, M->seg_bytes);
  build(true, M->segs_rest, M->seg_rest_blocks, M->seg_rest_bytes);
}

// Lays out every buffer; with base == nullptr it only measures.
size_t carve(sat_model* M, char* base) {
  const Dims& D = M->D;
  SatCarver c;
  c.base = base;
  const size_t NP = M->n_param_elems;
  M->master = c.take<float>(NP);
  M->shadow = c.take<bf16>(NP);
  size_t n_t = 0;
  for (const auto& p : M->params)
    if (p.toff != SIZE_MAX) n_t = std::max(n_t, p.toff + (size_t)p.trows * p.cols);
  M->shadow_t = c.take<bf16>(n_t > 0 ? n_t : 8);
  build_segments(M);
  M->segs_dev = c.take<AdamWSeg>(M->segs.size() + 1);
  M->segs_rest_dev = c.take<AdamWSeg>(M->segs_rest.size() + 1);
  M->grad = c.take<float>(NP);
  M->mom = c.take<float>(NP);
  M->vel = c.take<float>(NP);
  if (D.arch == SAT_RESNET) {
    sat_resnet_carve(M, c);
    return align_up(c.off, kAlignBytes);
  }
  const long T = D.T, d = D.d, m = D.m;
  const bool gptj = D.arch == SAT_GPTJ;
  // residual stream entering every block and the final LN
  M->h_in.assign(D.L + 1, nullptr);
  for (int l = 0; l <= D.L; ++l) M->h_in[l] = c.take<float>(T * d);
  M->act_rows.assign(D.L + 1, T);
  M->act_cols.assign(D.L + 1, (int)d);
  // per-layer saved activations: blocks >= k get their own, frozen blocks share
  // one set; with activation checkpointing every block uses the same set
  const int nsets = D.ckpt ? 1 : (D.k > 0) ? D.L - D.k + 1 : D.L;
  M->acts.assign(nsets, LayerActs());
  for (int s = 0; s < nsets; ++s) {
    LayerActs& A = M->acts[s];
    A.a = c.take<bf16>(T * d);
    A.mean1 = c.take<float>(T);
    A.rstd1 = c.take<float>(T);
    A.qkv = c.take<bf16>(T * D.qkv_ld);
    A.o = c.take<bf16>(T * d);
    A.lse = c.take<float>((size_t)D.B * D.H * D.S);
    A.g = c.take<bf16>(T * m);
    if (!gptj) {
      A.h_mid = c.take<float>(T * d);
      A.c = c.take<bf16>(T * d);
      A.mean2 = c.take<float>(T);
      A.rstd2 = c.take<float>(T);
      A.u = c.take<bf16>(T * m);
    } else {
      A.h_mid = nullptr;
      A.c = nullptr;
      A.mean2 = A.rstd2 = nullptr;
      A.u = nullptr;  // u lives in qkv[:, 3d:]
    }
  }
  // split-K workspace: the largest need of the step's fp32-output products
  // (weight gradients with K = tokens, input gradients into the residual
  // width, the forward residual products, the head's products)
  {
    const int Ti = (int)T, di = (int)d, mi = (int)m, R = D.rows_head;
    long ws = 0;
    // (weight gradients, K = tokens, never split the rows of their last round)
    auto need = [&](int Mg, int Ng, int Kg, bool wgrad) {
      ws = std::max(ws, gemm_splitk_ws_elems(Mg, Ng, Kg));
      if (!wgrad) ws = std::max(ws, gemm_tail_ws_elems(Mg, Ng, Kg));
    };
    need(D.qkv_ld, di, Ti, true);
    need(di, di, Ti, true);
    need(mi, di, Ti, true);
    need(di, mi, Ti, true);
    need(Ti, di, D.qkv_ld, false);
    need(Ti, di, mi, false);
    need(Ti, di, di, false);
    need(D.V, di, R, true);
    need(R, di, D.Vp, false);
    need(R, D.V, di, false);
    if (D.arch == SAT_VIT) need(di, D.pd, D.B * D.np, true);  // the patch weight's gradient
    M->splitk_ws_elems = ws;
    M->splitk_ws = ws > 0 ? c.take<float>((size_t)ws) : nullptr;
  }
  // head
  const long R = D.rows_head;
  M->f = c.take<bf16>(R * d);
  M->meanf = c.take<float>(R);
  M->rstdf = c.take<float>(R);
  M->logits = c.take<float>(R * D.Vp);
  M->dz = c.take<bf16>(R * D.Vp);
  M->row_loss = c.take<float>(R);
  M->scal = c.take<float>(8);  // [0] loss, [1] 1 / n_valid
  // ViT input side
  if (D.arch == SAT_VIT) {
    M->patches = c.take<bf16>((size_t)D.B * D.np * D.pdp);
    M->zpatch = c.take<float>((size_t)D.B * D.np * d);
    M->dzpatch = c.take<bf16>((size_t)D.B * D.np * d);
  }
  // backward workspace
  M->dh = c.take<float>(T * d);
  M->dh_bf = c.take<bf16>(T * d);
  M->dA = c.take<float>(T * d);
  M->dqkv = c.take<bf16>(T * D.qkv_ld);
  M->du = gptj ? nullptr : c.take<bf16>(T * m);
  M->dout = c.take<bf16>(T * d);
  M->trans_blocks = T % 8 == 0;
  M->trans_head = R % 8 == 0;
  {
    long na = 0, nb = 0;
    if (M->trans_blocks) {
      na = std::max(na, (long)std::max<long>(std::max<long>(d, D.qkv_ld), m) * T);
      nb = std::max(nb, std::max(d, m) * T);
    }
    if (M->trans_head) {
      na = std::max(na, (long)D.Vp * R);
      nb = std::max(nb, d * R);
    }
    M->tA = na > 0 ? c.take<bf16>(na) : nullptr;
    M->tB = nb > 0 ? c.take<bf16>(nb) : nullptr;
  }
  // operands of the blocks' weight-gradient products on the side stream (two
  // sets), and that stream's split-K workspace
  for (int i = 0; i < 2; ++i) {
    WgradSet& W = M->wset[i];
    memset(&W, 0, sizeof W);
    if (!M->trans_blocks) continue;
    W.dy1 = c.take<bf16>(T * d);
    W.g = c.take<bf16>(T * m);
    W.o = c.take<bf16>(T * d);
    W.a = c.take<bf16>(T * d);
    W.qkv = c.take<bf16>(T * D.qkv_ld);
    if (!gptj) {
      W.dy2 = c.take<bf16>(T * d);
      W.c = c.take<bf16>(T * d);
      W.du = c.take<bf16>(T * m);
    }
  }
  M->splitk_ws2 = M->splitk_ws_elems > 0 ? c.take<float>((size_t)M->splitk_ws_elems) : nullptr;
  M->delta = c.take<float>((size_t)D.B * D.H * D.S);
  M->rope_cs = D.rd > 0 ? c.take<float2>((size_t)D.S * (D.rd / 2)) : nullptr;
  M->n_part = (int)(T < 256 ? T : 256);
  long wide = D.qkv_ld > D.Vp ? D.qkv_ld : D.Vp;
  if (D.arch == SAT_VIT && D.pd > wide) wide = D.pd;
  // column-sum partials: n_part rows of the widest bias; LayerNorm partials:
  // ln_bwd_parts(rows, d) rows of d, for dg and db (and the bias gradient of
  // the residual product below, when the LayerNorm backward reduces it)
  const size_t lnp = (size_t)(sat_bias_in_ln_bwd(D) ? 3 : 2) *
                     ln_bwd_parts((int)std::max<long>(T, D.rows_head), d) * d;
  M->part_elems = (long)std::max((size_t)2 * M->n_part * (wide > d ? wide : d), lnp);
  M->part = c.take<float>((size_t)M->part_elems);
  M->sortbuf = c.take<int32_t>(T > 16384 ? 16384 : (T > 0 ? T : 1));  // one chunk of sorted keys
  return align_up(c.off, kAlignBytes);
}

}  // namespace

size_t sat_model_layout(sat_model* M, char* base) { return carve(M, base); }

double sat_step_flops(const Dims& D) {
  if (D.arch == SAT_RESNET) return sat_resnet_flops(D);
  const double T = D.T, d = D.d, m = D.m;
  const double gemm_layer = 2.0 * T * (3 * d * d + d * d + 2 * d * m);
  const double causal = (D.arch == SAT_VIT) ? 1.0 : 0.5;
  const double attn_layer = 4.0 * D.B * D.H * (double)D.S * D.S * D.dh * causal;
  const double fwd_layer = gemm_layer + attn_layer;
  double f = D.L * fwd_layer;                              // forward
  f += (D.L - D.k) * 2.0 * fwd_layer;                      // dgrad + wgrad, attention backward
  const double head = 2.0 * D.rows_head * d * D.V;
  f += 3.0 * head;
  if (D.arch == SAT_VIT) {
    const double pe = 2.0 * D.B * D.np * (double)D.pd * d;
    f += pe + (D.k == 0 ? pe : 0.0);
  }
  return f;
}
