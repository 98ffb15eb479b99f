// Helpers shared by the launch sequences of the fine-tuning step
// (transformers in step.cpp, the ResNet in resnet.cpp): per-launch timing of
// one kernel class, GEMM argument setup and launch, status propagation.
#pragma once

#include <string.h>

#include "abi_common.h"
#include "kernels.h"
#include "model.h"

namespace satstep {

enum {
  TK_OFF = 0, TK_QKV_FWD = 1, TK_ALL_GEMM = 2, TK_ADAMW = 3, TK_ATTN_FWD = 4, TK_ATTN_BWD = 5,
  TK_LN_FWD = 6, TK_LN_BWD = 7, TK_XENT = 8, TK_QKV_WGRAD = 9
};

// Records HIP events around the launches of one kernel class (the model's
// timing kind) while in scope, on the stream those launches go to (default:
// the model's stream).
struct Timed {
  sat_model* M;
  hipStream_t st;
  TimingRec* rec = nullptr;
  Timed(sat_model* m, int kind, double work, hipStream_t stream = nullptr)
      : M(m), st(stream ? stream : m->stream) {
    if (m->timing_kind == TK_OFF) return;
    bool match = (m->timing_kind == kind) ||
                 (m->timing_kind == TK_ALL_GEMM &&
                  (kind == TK_QKV_FWD || kind == TK_ALL_GEMM || kind == TK_QKV_WGRAD));
    if (!match || m->timing_used >= m->timing.size()) return;
    rec = &m->timing[m->timing_used++];
    rec->flops = work;
    hipEventRecord(rec->e0, st);
  }
  ~Timed() {
    if (rec) hipEventRecord(rec->e1, st);
  }
};

inline GemmArgs gargs(const bf16* A, long lda, const bf16* B, long ldb, int Mr, int N, int K,
                      void* out, long ldo) {
  GemmArgs a;
  memset(&a, 0, sizeof a);
  a.A = A;
  a.lda = lda;
  a.B = B;
  a.ldb = ldb;
  a.M = Mr;
  a.N = N;
  a.K = K;
  a.out = out;
  a.ldo = ldo;
  a.ldr = ldo;
  return a;
}

// One GEMM launch; fp32-output products with too few tiles run split-K in
// the workspace of the stream they go to (the model's stream, or the
// weight-gradient stream with its own workspace).
inline sat_status gemm(sat_model* M, const GemmArgs& a, int alay, int blay, int epi,
                       int tk = TK_ALL_GEMM, hipStream_t stream = nullptr) {
  const bool side = stream != nullptr && stream == M->side;
  hipStream_t st = stream ? stream : M->stream;
  Timed t(M, tk, 2.0 * a.M * a.N * (double)a.K, st);
  GemmArgs b = a;
  b.splitk_ws = side ? M->splitk_ws2 : M->splitk_ws;
  b.splitk_ws_elems = M->splitk_ws_elems;
  if (!M->tail_split) b.no_tail_split = 1;
  SAT_HIP(launch_gemm(b, alay, blay, epi, st));
  return SAT_OK;
}

#define TRY(x)                        \
  do {                                \
    sat_status st_ = (x);             \
    if (st_ != SAT_OK) return st_;    \
  } while (0)

// Parameter accessors by table index.
inline const float* master(const sat_model* M, int i) { return M->master + M->params[i].off; }
inline const bf16* shadow(const sat_model* M, int i) { return M->shadow + M->params[i].off; }
inline float* grad(sat_model* M, int i) { return M->grad + M->params[i].off; }
// Transposed bf16 copy [cols, trows] of a weight (B operand of dX = dY W).
inline const bf16* shadow_t(const sat_model* M, int i) { return M->shadow_t + M->params[i].toff; }

}  // namespace satstep
