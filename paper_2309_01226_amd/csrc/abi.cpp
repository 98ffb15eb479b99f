// Model-level C ABI (include/saturn.h): validation, arena ownership, the
// train / eval entry points and the synchronous host accessors.
#include <math.h>
#include <string.h>

#include <new>

#include "abi_common.h"
#include "kernels.h"
#include "model.h"

namespace {

sat_status check_model(const sat_model* m) {
  SAT_CHECK_ARG(m != nullptr, "null model");
  if (m->failed) {
    sat_set_error("model is in a failed state after an earlier HIP error");
    return SAT_ESTATE;
  }
  return SAT_OK;
}

sat_status mark(sat_model* m, sat_status st) {
  if (st == SAT_EHIP) m->failed = true;
  return st;
}

sat_status param_index(const sat_model* m, int32_t i) {
  SAT_CHECK_ARG(i >= 0 && (size_t)i < m->params.size(), "parameter index %d out of range", i);
  return SAT_OK;
}

sat_status sync(sat_model* m) {
  hipError_t e = hipStreamSynchronize(m->stream);
  if (e != hipSuccess) {
    sat_set_error("hipStreamSynchronize: %s", hipGetErrorString(e));
    m->failed = true;
    return SAT_EHIP;
  }
  return SAT_OK;
}

sat_status copy_d2h(sat_model* m, void* host, const void* dev, size_t bytes) {
  SAT_HIP(hipMemcpyAsync(host, dev, bytes, hipMemcpyDeviceToHost, m->stream));
  return sync(m);
}
sat_status copy_h2d(sat_model* m, void* dev, const void* host, size_t bytes) {
  SAT_HIP(hipMemcpyAsync(dev, host, bytes, hipMemcpyHostToDevice, m->stream));
  return sync(m);
}

}  // namespace

extern "C" sat_status sat_model_arena_bytes(const sat_config* cfg, size_t* bytes) {
  sat_status st = sat_validate_config(cfg);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(bytes != nullptr, "null bytes pointer");
  sat_model tmp;
  tmp.cfg = *cfg;
  sat_model_dims(*cfg, &tmp.D);
  sat_build_params(*cfg, tmp.D, tmp.params, &tmp.n_param_elems);
  *bytes = sat_model_layout(&tmp, nullptr);
  return SAT_OK;
}

// The weight-gradient stream (default priority) and its events, created on
// the first backward that uses them (a model that never overlaps adds no
// stream to the device's hardware queues).
void sat_side_destroy(sat_model* m) {
  if (m->side) {
    hipStreamSynchronize(m->side);
    hipStreamDestroy(m->side);
    m->side = nullptr;
  }
  for (hipEvent_t* e : {&m->ev_fork, &m->ev_done[0], &m->ev_done[1], &m->ev_join})
    if (*e) {
      hipEventDestroy(*e);
      *e = nullptr;
    }
}

sat_status sat_side_ensure(sat_model* m) {
  if (m->side) return SAT_OK;
  hipError_t e = hipStreamCreateWithFlags(&m->side, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev_fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev_done[0], hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev_done[1], hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev_join, hipEventDisableTiming);
  if (e != hipSuccess) {
    sat_set_error("creating the weight-gradient stream failed: %s", hipGetErrorString(e));
    sat_side_destroy(m);
    return SAT_EHIP;
  }
  return SAT_OK;
}

extern "C" sat_status sat_model_create(const sat_config* cfg, void* arena, size_t arena_bytes,
                                       void* hip_stream, sat_model** out) {
  sat_status st = sat_validate_config(cfg);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(out != nullptr, "null output pointer");
  sat_model* m = new (std::nothrow) sat_model();
  if (!m) {
    sat_set_error("host allocation failed");
    return SAT_ENOMEM;
  }
  m->cfg = *cfg;
  sat_model_dims(*cfg, &m->D);
  sat_build_params(*cfg, m->D, m->params, &m->n_param_elems);
  m->train_off = m->n_param_elems;
  for (const auto& p : m->params)
    if (p.trainable && p.off < m->train_off) m->train_off = p.off;
  m->stream = reinterpret_cast<hipStream_t>(hip_stream);
  m->t = 0;
  m->failed = false;
  m->timing_kind = 0;
  m->timing_used = 0;
  m->opt_fused = true;
  m->opt_keep_grads = false;
  m->opt_overlap = true;
  m->tail_split = cfg->arch != SAT_RESNET;
  m->last_step_fused = false;
  m->last_step_kept = false;
  hipGetDevice(&m->device);
  size_t need = sat_model_layout(m, nullptr);
  if (arena == nullptr) {
    hipError_t e = hipMalloc(&m->arena, need);
    if (e != hipSuccess) {
      sat_set_error("hipMalloc(%zu) failed: %s", need, hipGetErrorString(e));
      delete m;
      return SAT_ENOMEM;
    }
    m->own_arena = true;
    m->arena_bytes = need;
  } else {
    if (arena_bytes < need) {
      sat_set_error("arena of %zu bytes is smaller than the %zu bytes this model needs",
                    arena_bytes, need);
      delete m;
      return SAT_ENOMEM;
    }
    if (reinterpret_cast<uintptr_t>(arena) & 255) {
      sat_set_error("arena must be 256-byte aligned");
      delete m;
      return SAT_EINVAL;
    }
    m->arena = static_cast<char*>(arena);
    m->own_arena = false;
    m->arena_bytes = arena_bytes;
  }
  sat_model_layout(m, m->arena);
  st = sat_run_init(m);
  if (st == SAT_OK) st = sync(m);
  if (st != SAT_OK) {
    if (m->own_arena) hipFree(m->arena);
    delete m;
    return st;
  }
  *out = m;
  return SAT_OK;
}

extern "C" sat_status sat_model_destroy(sat_model* m) {
  if (m == nullptr) return SAT_OK;
  hipStreamSynchronize(m->stream);
  sat_side_destroy(m);
  for (auto& r : m->timing) {
    hipEventDestroy(r.e0);
    hipEventDestroy(r.e1);
  }
  if (m->own_arena) hipFree(m->arena);
  delete m;
  return SAT_OK;
}

static sat_status read_loss(sat_model* m, float* loss_out) {
  float h = 0.f;
  sat_status st = copy_d2h(m, &h, m->scal, sizeof(float));
  if (st != SAT_OK) return st;
  if (!isfinite(h)) {
    sat_set_error("loss is not finite (%f)", h);
    *loss_out = h;
    return SAT_ENONFINITE;
  }
  *loss_out = h;
  return SAT_OK;
}

extern "C" sat_status sat_train_step(sat_model* m, const void* inputs, const int32_t* labels,
                                     float* loss_out) {
  sat_status st = check_model(m);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(inputs != nullptr && labels != nullptr, "null inputs or labels");
  st = mark(m, sat_run_forward(m, inputs, labels));
  if (st == SAT_OK) st = mark(m, sat_adamw_begin(m));
  if (st == SAT_OK) st = mark(m, sat_run_backward(m, inputs));
  if (st == SAT_OK) st = mark(m, sat_run_adamw(m));
  if (st != SAT_OK) return st;
  if (loss_out) return read_loss(m, loss_out);
  return SAT_OK;
}

extern "C" sat_status sat_eval_loss(sat_model* m, const void* inputs, const int32_t* labels,
                                    float* loss_out) {
  sat_status st = check_model(m);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(inputs != nullptr && labels != nullptr && loss_out != nullptr,
                "null inputs, labels or loss_out");
  st = mark(m, sat_run_forward(m, inputs, labels));
  if (st != SAT_OK) return st;
  return read_loss(m, loss_out);
}

extern "C" int32_t sat_num_params(const sat_model* m) {
  return m ? (int32_t)m->params.size() : 0;
}

extern "C" sat_status sat_param_info(const sat_model* m, int32_t i, const char** name,
                                     int64_t shape[2], int32_t* trainable) {
  SAT_CHECK_ARG(m != nullptr, "null model");
  sat_status st = param_index(m, i);
  if (st != SAT_OK) return st;
  const ParamDesc& p = m->params[i];
  if (name) *name = p.name.c_str();
  if (shape) {
    shape[0] = p.rows;
    shape[1] = p.cols;
  }
  if (trainable) *trainable = p.trainable ? 1 : 0;
  return SAT_OK;
}

extern "C" sat_status sat_param_read(sat_model* m, int32_t i, float* host) {
  sat_status st = check_model(m);
  if (st == SAT_OK) st = param_index(m, i);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(host != nullptr, "null host buffer");
  const ParamDesc& p = m->params[i];
  return copy_d2h(m, host, m->master + p.off, (size_t)p.rows * p.cols * 4);
}

extern "C" sat_status sat_param_write(sat_model* m, int32_t i, const float* host) {
  sat_status st = check_model(m);
  if (st == SAT_OK) st = param_index(m, i);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(host != nullptr, "null host buffer");
  const ParamDesc& p = m->params[i];
  long n = p.rows * p.cols;
  st = copy_h2d(m, m->master + p.off, host, (size_t)n * 4);
  if (st != SAT_OK) return st;
  SAT_HIP(launch_f32_to_bf16(m->master + p.off, n, m->shadow + p.off, n, 1, (int)n, m->stream));
  st = sat_refresh_transposed(m, i);
  if (st != SAT_OK) return st;
  return sync(m);
}

extern "C" sat_status sat_grad_read(sat_model* m, int32_t i, float* host) {
  sat_status st = check_model(m);
  if (st == SAT_OK) st = param_index(m, i);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(host != nullptr, "null host buffer");
  const ParamDesc& p = m->params[i];
  // a weight stored after a fused one in the same matrix (GPT-J fc1 after q|k|v)
  bool fused = p.fused_opt;
  for (int32_t j = i - 1; j >= 0 && !fused; --j) {
    const ParamDesc& q = m->params[j];
    if (q.toff == SIZE_MAX || q.cols != p.cols || q.off + (size_t)q.trows * q.cols <= p.off) break;
    fused = q.fused_opt;
  }
  if (fused && p.trainable && m->last_step_fused && !m->last_step_kept) {
    sat_set_error("the gradient of %s was not stored: its AdamW step ran in its weight-gradient "
                  "product (set SAT_OPT_KEEP_GRADS to keep it)", p.name.c_str());
    return SAT_ENOTSUP;
  }
  return copy_d2h(m, host, m->grad + p.off, (size_t)p.rows * p.cols * 4);
}

extern "C" sat_status sat_model_set_option(sat_model* m, int32_t option, int32_t value) {
  sat_status st = check_model(m);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(value == 0 || value == 1, "option value %d is not 0 or 1", value);
  switch (option) {
    case SAT_OPT_FUSED_ADAMW: m->opt_fused = value != 0; return SAT_OK;
    case SAT_OPT_KEEP_GRADS: m->opt_keep_grads = value != 0; return SAT_OK;
    case SAT_OPT_OVERLAP_WGRAD: m->opt_overlap = value != 0; return SAT_OK;
  }
  sat_set_error("unknown option %d", option);
  return SAT_EINVAL;
}

extern "C" sat_status sat_activation_read(sat_model* m, int32_t layer, float* host) {
  sat_status st = check_model(m);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(layer >= 0 && layer <= m->D.L, "layer %d not in [0, n_layers]", layer);
  SAT_CHECK_ARG(host != nullptr, "null host buffer");
  return copy_d2h(m, host, m->h_in[layer], (size_t)m->act_rows[layer] * m->act_cols[layer] * 4);
}

extern "C" sat_status sat_activation_shape(const sat_model* m, int32_t layer, int64_t shape[2]) {
  SAT_CHECK_ARG(m != nullptr && shape != nullptr, "null model or shape");
  SAT_CHECK_ARG(layer >= 0 && layer <= m->D.L, "layer %d not in [0, n_layers]", layer);
  shape[0] = m->act_rows[layer];
  shape[1] = m->act_cols[layer];
  return SAT_OK;
}

extern "C" sat_status sat_logits_read(sat_model* m, float* host) {
  sat_status st = check_model(m);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(host != nullptr, "null host buffer");
  const Dims& D = m->D;
  SAT_HIP(hipMemcpy2DAsync(host, (size_t)D.V * 4, m->logits, (size_t)D.Vp * 4, (size_t)D.V * 4,
                           D.rows_head, hipMemcpyDeviceToHost, m->stream));
  return sync(m);
}

extern "C" sat_status sat_state_read(sat_model* m, int32_t i, float* mom, float* vel,
                                     int64_t* t) {
  sat_status st = check_model(m);
  if (st == SAT_OK) st = param_index(m, i);
  if (st != SAT_OK) return st;
  const ParamDesc& p = m->params[i];
  size_t bytes = (size_t)p.rows * p.cols * 4;
  if (mom && (st = copy_d2h(m, mom, m->mom + p.off, bytes)) != SAT_OK) return st;
  if (vel && (st = copy_d2h(m, vel, m->vel + p.off, bytes)) != SAT_OK) return st;
  if (t) *t = m->t;
  return SAT_OK;
}

extern "C" sat_status sat_state_write(sat_model* m, int32_t i, const float* mom, const float* vel,
                                      int64_t t) {
  sat_status st = check_model(m);
  if (st == SAT_OK) st = param_index(m, i);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(t >= 0, "t must be >= 0");
  const ParamDesc& p = m->params[i];
  size_t bytes = (size_t)p.rows * p.cols * 4;
  if (mom && (st = copy_h2d(m, m->mom + p.off, mom, bytes)) != SAT_OK) return st;
  if (vel && (st = copy_h2d(m, m->vel + p.off, vel, bytes)) != SAT_OK) return st;
  m->t = t;
  return SAT_OK;
}

extern "C" sat_status sat_model_stats(const sat_model* m, int64_t* n_params, int64_t* n_trainable,
                                      double* step_flops) {
  SAT_CHECK_ARG(m != nullptr, "null model");
  int64_t np = 0, nt = 0;
  for (const auto& p : m->params) {
    np += p.rows * p.cols;
    if (p.trainable) nt += p.rows * p.cols;
  }
  if (n_params) *n_params = np;
  if (n_trainable) *n_trainable = nt;
  if (step_flops) *step_flops = sat_step_flops(m->D);
  return SAT_OK;
}

extern "C" sat_status sat_model_set_timing(sat_model* m, int32_t kind, int32_t max_launches) {
  sat_status st = check_model(m);
  if (st != SAT_OK) return st;
  SAT_CHECK_ARG(kind >= 0 && kind <= 9, "unknown timing kind %d", kind);
  SAT_CHECK_ARG(max_launches >= 0 && max_launches <= (1 << 20), "bad max_launches");
  st = sync(m);
  if (st != SAT_OK) return st;
  for (auto& r : m->timing) {
    hipEventDestroy(r.e0);
    hipEventDestroy(r.e1);
  }
  m->timing.clear();
  m->timing_used = 0;
  m->timing_kind = 0;
  if (kind == 0 || max_launches == 0) return SAT_OK;
  m->timing.resize(max_launches);
  for (auto& r : m->timing) {
    SAT_HIP(hipEventCreate(&r.e0));
    SAT_HIP(hipEventCreate(&r.e1));
    r.flops = 0.0;
  }
  m->timing_kind = kind;
  return SAT_OK;
}

extern "C" sat_status sat_model_timing_read(sat_model* m, double* total_ms, int64_t* launches,
                                            double* work) {
  sat_status st = check_model(m);
  if (st != SAT_OK) return st;
  st = sync(m);
  if (st != SAT_OK) return st;
  double ms = 0.0, w = 0.0;
  for (size_t i = 0; i < m->timing_used; ++i) {
    float e = 0.f;
    SAT_HIP(hipEventElapsedTime(&e, m->timing[i].e0, m->timing[i].e1));
    ms += e;
    w += m->timing[i].flops;
  }
  if (total_ms) *total_ms = ms;
  if (launches) *launches = (int64_t)m->timing_used;
  if (work) *work = w;
  m->timing_used = 0;
  return SAT_OK;
}
