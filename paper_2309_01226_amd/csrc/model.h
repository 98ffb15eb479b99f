// Internal model state shared by the runtime translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <memory>
#include <string>
#include <vector>

#include "../../include/saturn.h"
#include "kernels.h"

typedef __bf16 bf16;

struct Dims {
  int arch;
  int L, d, H, dh, m, V, Vp, B, S, T, k, rd;
  int np, pd;      // ViT: patches per image, values per patch
  int pdp;         // ViT: pitch of a row of patch values (pd rounded up to 8)
  int rows_head;   // rows entering the head (T, or B for ViT)
  int qkv_ld;      // row pitch of the q|k|v (|u for GPT-J) buffer
  bool ckpt;       // activation checkpointing: one saved-activation set, recomputed per block
  // RESNET: blocks per stage, stem / stage-0 mid width, image side and channels
  int res_blocks[4];
  int res_width, img, channels;
};

struct ParamDesc {
  std::string name;
  long rows, cols;
  size_t off;      // element offset in the parameter arena
  int group;       // -1 embeddings, l = block, L = final LN + head
  int kind;        // 0 normal init, 1 zeros, 2 ones
  bool trainable;
  // Transposed bf16 copy [cols, trows] at this element offset of shadow_t
  // (SIZE_MAX: none).  trows >= rows: the GPT-J q|k|v|fc1 weights are one
  // [3d + m, d] matrix, the head's covers the padded vocabulary.
  size_t toff;
  long trows;
  // The AdamW step of this weight (with the parameters stored after it in
  // the same matrix segment) runs in the epilogue of its weight-gradient
  // product whenever the optimizer is fused (see sat_model::opt_fused).
  bool fused_opt;
};

struct LayerActs {
  bf16* a;          // LN1 output [T, d]
  float* mean1;
  float* rstd1;
  bf16* qkv;        // [T, qkv_ld]: q | k | v (GPT-J: | u, the MLP pre-activation)
  bf16* o;          // attention output [T, d]
  float* lse;       // [B, H, S]
  bf16* g;          // GELU output [T, m]
  float* h_mid;     // GPT-2 / ViT: residual after attention [T, d]
  bf16* c;          // LN2 output
  float* mean2;
  float* rstd2;
  bf16* u;          // GPT-2 / ViT: MLP pre-activation [T, m]
};

struct ResNetPlan;  // resnet.cpp

// Carves 256-byte aligned sections out of the arena; with base == nullptr it
// only measures.
struct SatCarver {
  size_t off = 0;
  char* base = nullptr;
  template <typename T>
  T* take(size_t count) {
    size_t o = (off + 255) / 256 * 256;
    off = o + count * sizeof(T);
    return base ? reinterpret_cast<T*>(base + o) : nullptr;
  }
};

struct TimingRec {
  hipEvent_t e0, e1;
  double flops;
};

// Token-contiguous copies of the operands of one block's weight-gradient
// products, read by those products on the weight-gradient stream (two sets,
// used by alternate blocks).  dy1: dY of fc2 (and of the out-projection in
// the parallel GPT-J block); dy2: dY of the out-projection in the sequential
// block (the residual gradient after the second LayerNorm's backward);
// g, o, a, c: inputs of fc2, out-projection, QKV, fc1; du: dY of fc1; qkv: dY
// of the QKV (GPT-J: QKV + fc1) product.
struct WgradSet {
  bf16 *dy1, *dy2, *g, *o, *a, *c, *du, *qkv;
};

struct sat_model {
  sat_config cfg;
  Dims D;
  hipStream_t stream;
  // Weight-gradient stream: with opt_overlap the block's weight-gradient
  // products (and the AdamW steps fused into them) run here, beside the
  // input-gradient chain of the blocks below.  Created on first use.
  hipStream_t side;
  hipEvent_t ev_fork;     // model stream -> side: the operands are ready
  hipEvent_t ev_done[2];  // side -> model stream: set i may be rewritten
  hipEvent_t ev_join;     // side -> model stream: every product done
  bool side_pending[2];
  bool opt_overlap;
  WgradSet wset[2];
  float* splitk_ws2;      // split-K workspace of the side stream
  int device;
  char* arena;
  size_t arena_bytes;
  bool own_arena;
  bool failed;
  int64_t t;
  std::vector<ParamDesc> params;
  size_t n_param_elems;
  size_t train_off;  // first trainable element
  // parameter-sized sections
  float* master;
  bf16* shadow;
  bf16* shadow_t;  // transposed copies of the trainable weights of dX = dY W
  // AdamW over the trainable parameters: segment table (host copy and device
  // copy in the arena) and the workgroup count of one launch.
  std::vector<AdamWSeg> segs;
  AdamWSeg* segs_dev;
  int seg_blocks;
  double seg_bytes;  // algorithmic bytes of one launch over the table
  // The same without the matrices whose update is fused into their
  // weight-gradient products (the table launched when the optimizer is fused).
  std::vector<AdamWSeg> segs_rest;
  AdamWSeg* segs_rest_dev;
  int seg_rest_blocks;
  double seg_rest_bytes;
  // Options (sat_model_set_option): fuse the AdamW step of eligible weights
  // into their weight-gradient products (default on); also write those
  // weights' gradients to the gradient arena (default off).
  bool opt_fused;
  bool opt_keep_grads;
  bool last_step_fused;   // the last train step updated fused weights in their products
  bool last_step_kept;    // ... and kept their gradients
  AdamWConsts adamw_c;    // constants of the step in progress
  float* grad;
  float* mom;
  float* vel;
  // activations; h_in[l] ([act_rows[l], act_cols[l]] fp32) is what
  // sat_activation_read returns for layer l
  std::vector<float*> h_in;
  std::vector<long> act_rows;
  std::vector<int> act_cols;
  std::shared_ptr<ResNetPlan> rn;  // RESNET: layout and buffers of the convolutional step
  std::vector<LayerActs> acts;
  bf16* f;
  float* meanf;
  float* rstdf;
  float* logits;
  bf16* dz;
  float* row_loss;
  float* scal;
  bf16* patches;
  float* zpatch;
  bf16* dzpatch;
  // backward workspace
  float* dh;
  bf16* dh_bf;
  float* dA;
  bf16* dqkv;
  bf16* du;
  bf16* dout;
  // Token-contiguous (transposed) copies of the operands of the weight-gradient
  // products dW = dY^T X: tA holds dY^T, tB holds X^T (null when the token
  // count is not a multiple of 8; those products then read the row-major copies).
  bf16* tA;
  bf16* tB;
  bool trans_blocks;  // tA / tB serve the blocks (T % 8 == 0)
  bool trans_head;    // ... and the head (rows_head % 8 == 0)
  // split-K workspace of the fp32-output products with too few tiles
  float* splitk_ws;
  long splitk_ws_elems;
  float* delta;
  float2* rope_cs;  // rotary (cos, sin) per (position, pair); null without rotary
  float* part;
  long part_elems;  // fp32 elements of part
  // Whether fp32-output products may split the rows of a mostly empty last
  // round of tiles (launch_gemm's tail split).  The ResNet keeps every row of
  // a product summed in one order, so a batch of copies of one image gives
  // identical activations.
  bool tail_split;
  int n_part;
  int32_t* sortbuf;
  // optional per-launch timing of one kernel class
  int timing_kind;
  std::vector<TimingRec> timing;
  size_t timing_used;
};

// The weight-gradient stream: created on first use, destroyed with the model.
sat_status sat_side_ensure(sat_model* m);
// Whether the LayerNorm backward also reduces the bias gradient of the residual
// product below it (rows up to 2048 wide; wider rows use a separate column sum).
inline bool sat_bias_in_ln_bwd(const Dims& D) { return D.d <= 2048; }
// Whether the fc2 input-gradient product sums the fc1 bias gradient in its
// epilogue: for the same widths (at 4096 it measured no faster, and the
// weight-gradient products beside it on the second stream slowed down).
inline bool sat_fc1_bias_in_epilogue(const Dims& D) { return D.d <= 2048; }
void sat_side_destroy(sat_model* m);

sat_status sat_validate_config(const sat_config* c);
void sat_model_dims(const sat_config& c, Dims* d);
void sat_build_params(const sat_config& c, const Dims& D, std::vector<ParamDesc>& P,
                      size_t* n_total);
size_t sat_model_layout(sat_model* M, char* base);
double sat_step_flops(const Dims& D);

// step.cpp
sat_status sat_run_forward(sat_model* M, const void* inputs, const int32_t* labels);
sat_status sat_run_backward(sat_model* M, const void* inputs);
// AdamW: begin (t += 1 and the step's constants, before the backward, whose
// fused weight-gradient products apply them), end (one launch over the
// segment table of everything not updated by those products).
sat_status sat_adamw_begin(sat_model* M);
sat_status sat_run_adamw(sat_model* M);
sat_status sat_run_init(sat_model* M);
// Rewrites shadow_t from shadow (all transposed weights, or parameter i only).
sat_status sat_refresh_transposed(sat_model* M, int only = -1);

const LayerActs& sat_layer_acts(const sat_model* M, int l);

// resnet.cpp: the bottleneck-ResNet architecture
sat_status sat_resnet_validate(const sat_config* c);
void sat_resnet_dims(const sat_config& c, Dims* d);
void sat_resnet_build_params(const sat_config& c, const Dims& D, std::vector<ParamDesc>& P,
                             size_t* n_total);
void sat_resnet_carve(sat_model* M, SatCarver& c);
double sat_resnet_flops(const Dims& D);
sat_status sat_resnet_forward(sat_model* M, const void* inputs, const int32_t* labels);
sat_status sat_resnet_backward(sat_model* M, const void* inputs);
