// Profiler over the model ABI (include/saturn.h, sat_profile): the runtime
// estimate that the paper's Trial Runner produces for every task (Sec. 3.2):
// a few minibatches of the task's own fine-tuning step, averaged, and the
// epoch time extrapolated from that average, which is sound because every
// SGD step of a task does the same work.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "abi_common.h"
#include "kernels.h"
#include "model.h"

namespace {

struct DevBuf {
  void* p = nullptr;
  ~DevBuf() {
    if (p) hipFree(p);
  }
};

struct Events {
  std::vector<hipEvent_t> e;
  ~Events() {
    for (auto x : e)
      if (x) hipEventDestroy(x);
  }
};

}  // namespace

extern "C" sat_status sat_profile_batch(const sat_config* cfg, void* inputs, int32_t* labels,
                                        void* hip_stream) {
  SAT_CHECK_ARG(cfg != nullptr && inputs != nullptr && labels != nullptr,
                "null configuration or buffer");
  sat_status st = sat_validate_config(cfg);
  if (st != SAT_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  const uint32_t seed = (uint32_t)(cfg->seed ^ (cfg->seed >> 32)) ^ 0x51ED270Bu;
  hipError_t e;
  if (cfg->arch == SAT_VIT || cfg->arch == SAT_RESNET) {
    const long n_in = (long)cfg->batch * cfg->channels * cfg->img_size * cfg->img_size;
    e = launch_synth_images((float*)inputs, n_in, labels, cfg->batch, cfg->vocab, seed, s);
  } else {
    e = launch_synth_tokens((int32_t*)inputs, labels, cfg->batch, cfg->seq_len, cfg->vocab, seed, s);
  }
  if (e != hipSuccess) {
    sat_set_error("synthetic batch: %s", hipGetErrorString(e));
    return SAT_EHIP;
  }
  return SAT_OK;
}

extern "C" sat_status sat_profile(const sat_config* cfg, void* hip_stream, int32_t warmup,
                                  int32_t steps, int64_t samples_per_epoch,
                                  sat_profile_result* out) {
  SAT_CHECK_ARG(cfg != nullptr && out != nullptr, "null configuration or result");
  SAT_CHECK_ARG(out->struct_size == sizeof(sat_profile_result),
                "sat_profile_result.struct_size is %u, expected %zu", out->struct_size,
                sizeof(sat_profile_result));
  SAT_CHECK_ARG(warmup >= 0 && steps >= 1 && steps <= 100000, "warmup %d / steps %d out of range",
                warmup, steps);
  SAT_CHECK_ARG(samples_per_epoch >= 0, "negative samples_per_epoch");
  sat_status st = sat_validate_config(cfg);
  if (st != SAT_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);

  size_t arena = 0;
  st = sat_model_arena_bytes(cfg, &arena);
  if (st != SAT_OK) return st;
  sat_model* m = nullptr;
  st = sat_model_create(cfg, nullptr, 0, hip_stream, &m);
  if (st != SAT_OK) return st;

  // synthetic batch of the task's shape, generated on the device
  Dims D;
  sat_model_dims(*cfg, &D);
  const bool vit = cfg->arch == SAT_VIT || cfg->arch == SAT_RESNET;
  const long n_in = vit ? (long)cfg->batch * cfg->channels * cfg->img_size * cfg->img_size
                        : (long)cfg->batch * cfg->seq_len;
  const long n_lab = vit ? cfg->batch : (long)cfg->batch * cfg->seq_len;
  DevBuf in, lab;
  Events ev;
  auto fail = [&](sat_status code) {
    sat_model_destroy(m);
    return code;
  };
  hipError_t e = hipMalloc(&in.p, (size_t)n_in * 4);
  if (e == hipSuccess) e = hipMalloc(&lab.p, (size_t)n_lab * 4);
  if (e != hipSuccess) {
    sat_set_error("hipMalloc of the profiling batch failed: %s", hipGetErrorString(e));
    return fail(SAT_ENOMEM);
  }
  st = sat_profile_batch(cfg, in.p, (int32_t*)lab.p, hip_stream);
  if (st != SAT_OK) return fail(st);
  for (int i = 0; i < warmup; ++i) {
    st = sat_train_step(m, in.p, (const int32_t*)lab.p, nullptr);
    if (st != SAT_OK) return fail(st);
  }
  ev.e.assign((size_t)steps + 1, nullptr);
  for (auto& x : ev.e) {
    e = hipEventCreate(&x);
    if (e != hipSuccess) {
      sat_set_error("hipEventCreate: %s", hipGetErrorString(e));
      return fail(SAT_EHIP);
    }
  }
  // one event between consecutive steps on the model's stream
  e = hipEventRecord(ev.e[0], s);
  for (int i = 0; i < steps && e == hipSuccess; ++i) {
    st = sat_train_step(m, in.p, (const int32_t*)lab.p, nullptr);
    if (st != SAT_OK) return fail(st);
    e = hipEventRecord(ev.e[i + 1], s);
  }
  if (e == hipSuccess) e = hipEventSynchronize(ev.e[steps]);
  if (e != hipSuccess) {
    sat_set_error("profiling events: %s", hipGetErrorString(e));
    return fail(SAT_EHIP);
  }
  double sum = 0.0, mn = INFINITY, mx = 0.0;
  for (int i = 0; i < steps; ++i) {
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, ev.e[i], ev.e[i + 1]);
    if (e != hipSuccess) {
      sat_set_error("hipEventElapsedTime: %s", hipGetErrorString(e));
      return fail(SAT_EHIP);
    }
    sum += ms;
    mn = std::min(mn, (double)ms);
    mx = std::max(mx, (double)ms);
  }
  float loss = 0.f;
  st = sat_eval_loss(m, in.p, (const int32_t*)lab.p, &loss);
  if (st != SAT_OK && st != SAT_ENONFINITE) return fail(st);

  sat_profile_result r;
  memset(&r, 0, sizeof r);
  r.struct_size = sizeof r;
  r.steps = steps;
  r.step_ms_mean = sum / steps;
  r.step_ms_min = mn;
  r.step_ms_max = mx;
  const double rows = cfg->arch == SAT_RESNET ? (double)cfg->batch
                      : vit ? (double)cfg->batch * D.S : (double)cfg->batch * cfg->seq_len;
  r.tokens_per_s = rows / (r.step_ms_mean * 1e-3);
  r.step_tflop = sat_step_flops(D) / 1e12;
  r.achieved_tflops = r.step_tflop / (r.step_ms_mean * 1e-3);
  const int64_t steps_per_epoch =
      samples_per_epoch > 0 ? (samples_per_epoch + cfg->batch - 1) / cfg->batch : 0;
  r.steps_per_epoch = steps_per_epoch;
  r.epoch_ms = r.step_ms_mean * (double)steps_per_epoch;
  r.arena_bytes = arena;
  r.final_loss = loss;
  st = sat_model_destroy(m);
  if (st != SAT_OK) return st;
  *out = r;
  return SAT_OK;
}
