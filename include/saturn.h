/* saturn.h -- C ABI of the MI355X fine-tuning-step library (libsaturn.so).
 *
 * The Saturn paper (Nagrecha & Kumar, arXiv 2309.01226) schedules a set of
 * model-training tasks, each given by a model, its data and its own
 * hyper-parameters (Sec. 3.1 "Workload Specification", the Task / HParams
 * API), drawn from model selection: grid or random search over batch size and
 * learning rate, and layer-wise fine-tuning, i.e. choosing which layers to
 * train (Abstract; Sec. 2 "Model selection"; Table 3).  The work it orders is
 * the fine-tuning step of each task.  This library runs that step on one
 * gfx950 GPU: one opaque model per task, advanced by sat_train_step.
 *
 * Conventions for every call:
 *   - returns SAT_OK or a negative sat_status; out-parameters are written only
 *     on SAT_OK; sat_last_error() gives a message (thread-local);
 *   - no call aborts the process;
 *   - "device pointer" means memory of the model's GPU; "host pointer" means
 *     ordinary CPU memory;
 *   - distinct models may be driven from one host thread on distinct streams;
 *     a single model is not re-entrant.
 */
#ifndef SATURN_H
#define SATURN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sat_model sat_model; /* opaque, owned by the library */

typedef enum {
  SAT_OK = 0,
  SAT_EINVAL = -1,      /* invalid configuration or argument */
  SAT_ENOMEM = -2,      /* the arena is too small (or device allocation failed); the analogue of
                           a parallelism's search reporting an out-of-memory plan as a null
                           result (Sec. 3.1, Parallelism Library, the search function) */
  SAT_EHIP = -3,        /* a HIP runtime call failed */
  SAT_ESTATE = -4,      /* the model is in a failed state */
  SAT_ENONFINITE = -5,  /* the loss read back is NaN or infinite */
  SAT_ENOTSUP = -6      /* the operation does not apply to this model */
} sat_status;

typedef enum { SAT_GPT2 = 0, SAT_GPTJ = 1, SAT_VIT = 2, SAT_RESNET = 3 } sat_arch;

/* Per-task configuration: architecture, depth, width, batch size, learning
 * rate and frozen-layer count of one model (the hyper-parameters a model
 * selection task carries, Sec. 3.1).
 *   GPT2: pre-LN decoder, learned positions, bias on every linear, untied head
 *         without bias, tanh GELU, causal attention.
 *   GPTJ: one LN per block feeding attention and MLP in parallel, rotary on the
 *         first rotary_dim dims of every head, no q/k/v/out bias, head bias.
 *   VIT : pre-LN encoder over (img/patch)^2 patches + a CLS token, erf GELU,
 *         bidirectional attention, class head on the CLS row.
 *   RESNET: bottleneck ResNet (the paper's second image model, Table 3):
 *         7 x 7 / 2 stem convolution, batch norm, ReLU, 3 x 3 / 2 max pool;
 *         stages of res_blocks[s] bottleneck blocks (1 x 1, 3 x 3 with the
 *         stage's stride in its first block, 1 x 1 with 4x expansion, batch
 *         norm after each, projection shortcut in each stage's first block,
 *         ReLU after the add) with mid width res_width * 2^s; global average
 *         pool and a linear class head with bias.  Batch norm uses the
 *         statistics of the current batch (training mode; no running
 *         statistics), eps = ln_eps.  n_layers = the total block count;
 *         d_model, n_heads, d_mlp, seq_len, patch and rotary_dim are unused
 *         (0). */
typedef struct {
  uint32_t struct_size; /* must equal sizeof(sat_config) */
  int32_t arch;         /* sat_arch */
  int32_t n_layers, d_model, n_heads, d_mlp;
  int32_t vocab;        /* decoders: vocabulary size; VIT: number of classes */
  int32_t seq_len;      /* decoders: tokens per row; VIT: ignored (derived) */
  int32_t img_size, patch, channels; /* VIT only */
  int32_t rotary_dim;   /* GPTJ: even, <= head dim; others 0 */
  int32_t batch;        /* rows per step, fixed per model */
  int32_t frozen_layers;/* k in [0, n_layers]: k > 0 freezes the embeddings and blocks [0, k) */
  int32_t checkpoint;   /* activation checkpointing, 0 or 1: 1 keeps only each block's input
                          (the residual stream) and recomputes the block's forward activations
                          just before its backward, with the same kernels on the same input,
                          so results are bitwise those of 0; saves all but one block's saved
                          activations, and costs each block's forward except its last
                          products (GPT-J: out-projection and fc2; GPT2 / VIT: fc2) once more
                          per step, which the step's algorithmic FLOPs do not count. */
  double lr, beta1, beta2, eps, weight_decay; /* AdamW, decoupled decay on every trainable
                          tensor; double so that 1 - beta is exact to float precision */
  float init_std;       /* std of the N(0, std^2) initialisation of matrices and tables */
  float ln_eps;
  uint64_t seed;        /* counter-based initialisation seed */
  int32_t res_blocks[4];/* RESNET: blocks per stage (each >= 1, sum = n_layers); others 0 */
  int32_t res_width;    /* RESNET: stem width = stage-0 mid width, a multiple of 8 */
} sat_config;

/* Bytes of device memory a model of this configuration needs (parameters,
 * bf16 shadow, gradients, AdamW moments, activations, workspace).  This is the
 * memory side of a parallelism's search for one task on one GPU (Sec. 3.1,
 * Parallelism Library): a caller learns before creation whether the task fits.
 * Errors: SAT_EINVAL for an invalid configuration. */
sat_status sat_model_arena_bytes(const sat_config* cfg, size_t* bytes);

/* Create a model on the current HIP device: the model-initialisation half of a
 * Task, with its hyper-parameters taken from cfg (Sec. 3.1, Trainer API: a
 * task is a model-initialisation function, a data-loading function and its
 * hyper-parameters).  Data loading stays with the caller, who passes device
 * batches to sat_train_step.
 *   arena: device pointer of at least arena_bytes bytes, borrowed until
 *          sat_model_destroy; NULL makes the library allocate (and own) it.
 *   hip_stream: hipStream_t every kernel of this model is enqueued on (NULL =
 *          the null stream); borrowed.
 * Initialises parameters (matrices and tables ~ N(0, init_std^2) from `seed`,
 * biases 0, LN gains 1) and zeroes AdamW state; t = 0.
 * Errors: SAT_EINVAL (configuration), SAT_ENOMEM (arena_bytes too small or
 * allocation failure), SAT_EHIP. */
sat_status sat_model_create(const sat_config* cfg, void* arena, size_t arena_bytes,
                            void* hip_stream, sat_model** out);

/* One fine-tuning step: forward, backward down to block k, AdamW on the
 * trainable tensors (t += 1), all enqueued on the model's stream.  One SGD
 * iteration of a task, the unit a parallelism's execute function repeats to
 * train the task (Sec. 3.1, Parallelism Library) and the unit the Trial
 * Runner times (Sec. 3.2, Profiler); which layers train is the layer-wise
 * fine-tuning choice of model selection (Abstract; Sec. 2, Model selection).
 *   inputs: device pointer; decoders int32 tokens [batch, seq_len] in
 *           [0, vocab); VIT fp32 images [batch, channels, img, img].
 *   labels: device pointer, int32; decoders [batch, seq_len], VIT [batch];
 *           -1 = ignore, otherwise in [0, vocab).
 *   loss_out: host pointer or NULL.  Non-NULL: the call waits for the step and
 *           writes the mean loss over non-ignored labels.  NULL: the call
 *           returns as soon as the work is enqueued.
 * Out-of-range token ids or labels are not checked on the device.
 * Errors: SAT_EINVAL (null model or pointers), SAT_ESTATE, SAT_EHIP,
 * SAT_ENONFINITE (loss read back is not finite; the update was applied). */
sat_status sat_train_step(sat_model* m, const void* inputs, const int32_t* labels,
                          float* loss_out);

/* Forward only; writes the mean loss to the host pointer loss_out (waits for
 * the stream).  Changes no parameter or optimizer state.  The loss by which
 * model selection compares the trained configurations (Sec. 2, Model
 * selection: training and comparing model configurations).
 * Arguments as for sat_train_step; loss_out must not be NULL.
 * Errors: SAT_EINVAL (null model or pointers), SAT_ESTATE, SAT_EHIP,
 * SAT_ENONFINITE. */
sat_status sat_eval_loss(sat_model* m, const void* inputs, const int32_t* labels,
                         float* loss_out);

/* Release the model (and the arena when the library allocated it).  Waits for
 * the model's stream.  NULL is accepted.  Ends a task's use of its GPU memory,
 * which the schedule then gives to the next task (Sec. 3.3, Joint Optimizer and Executor). */
sat_status sat_model_destroy(sat_model* m);

/* ---- parameter table and test / resume accessors --------------------------
 * Tensors are numbered 0..n-1 bottom to top (embeddings, blocks 0..L-1, final
 * LN, head).  Linear weights are [out, in] (y = x W^T + b).  All host buffers
 * are fp32 (t: int64) of the tensor's element count; every accessor waits for
 * the model's stream. */
int32_t sat_num_params(const sat_model* m);
/* name: static string owned by the library; shape: [rows, cols] (cols = 1 for vectors). */
sat_status sat_param_info(const sat_model* m, int32_t i, const char** name, int64_t shape[2],
                          int32_t* trainable);
sat_status sat_param_read(sat_model* m, int32_t i, float* host);
/* Writes the fp32 master and refreshes the bf16 shadow. */
sat_status sat_param_write(sat_model* m, int32_t i, const float* host);
/* Gradient of the last sat_train_step; zeros for frozen tensors.
 * SAT_ENOTSUP when that step applied tensor i's AdamW step inside its
 * weight-gradient product with SAT_OPT_KEEP_GRADS off: that gradient was
 * never stored. */
sat_status sat_grad_read(sat_model* m, int32_t i, float* host);
/* Residual stream entering block `layer` (fp32 [batch * seq, d_model]) after
 * the last forward; layer = n_layers gives the stream entering the final LN.
 * RESNET: the input of block `layer` (fp32 NHWC [batch * H * W, C]); layer =
 * n_layers gives the last block's output.  sat_activation_shape gives the
 * [rows, cols] of that tensor. */
sat_status sat_activation_read(sat_model* m, int32_t layer, float* host);
sat_status sat_activation_shape(const sat_model* m, int32_t layer, int64_t shape[2]);
/* Logits of the last forward, fp32 [rows, vocab] (rows = batch * seq, VIT: batch). */
sat_status sat_logits_read(sat_model* m, float* host);
sat_status sat_state_read(sat_model* m, int32_t i, float* mom, float* vel, int64_t* t);
sat_status sat_state_write(sat_model* m, int32_t i, const float* mom, const float* vel, int64_t t);
/* Number of trainable parameters (elements) and algorithmic FLOPs of one step. */
sat_status sat_model_stats(const sat_model* m, int64_t* n_params, int64_t* n_trainable,
                           double* step_flops);

/* ---- options ---------------------------------------------------------------
 * SAT_OPT_FUSED_ADAMW (default 1): the AdamW step of every weight matrix
 *   whose weight-gradient product runs in the 256 x 256 GEMM kernel is applied
 *   in that product's epilogue (the same fp32 arithmetic on the same fp32
 *   gradient as the separate pass), so the gradient makes no round trip
 *   through the gradient arena.  0: every tensor is updated by the separate
 *   AdamW pass after the backward.
 * SAT_OPT_KEEP_GRADS (default 0): 1 also writes the gradients of those
 *   weights to the gradient arena, so that sat_grad_read returns them.
 * SAT_OPT_OVERLAP_WGRAD (default 1): the blocks' weight-gradient products
 *   (with the AdamW steps fused into them) run on a second stream that the
 *   library creates on the first such backward (default priority; destroyed
 *   with the model), beside the input-gradient chain of the
 *   blocks below; they read token-contiguous copies of their operands in two
 *   alternating sets, and the step joins that stream back into the model's
 *   stream before the backward ends, so a caller that synchronizes the
 *   model's stream sees the whole step.  Results are bitwise those with 0
 *   (the same kernels on the same operands).  Needs batch * seq_len % 8 == 0
 *   (otherwise ignored).
 * value is 0 or 1; the setting applies from the next train step.
 * Errors: SAT_EINVAL (null model, unknown option or value), SAT_ESTATE. */
typedef enum {
  SAT_OPT_FUSED_ADAMW = 1,
  SAT_OPT_KEEP_GRADS = 2,
  SAT_OPT_OVERLAP_WGRAD = 3
} sat_option;
sat_status sat_model_set_option(sat_model* m, int32_t option, int32_t value);

/* ---- measurement ---------------------------------------------------------
 * Per-launch timing of one kernel class with HIP events recorded on the
 * model's stream around each matching launch (at most max_launches between
 * two reads; later launches are not timed).  kind: 0 off, 1 the forward QKV
 * product (GPT-J: the fused QKV + fc1 product), 2 every GEMM, 3 the AdamW
 * update, 4 attention forward, 5 attention backward, 6 LayerNorm forward,
 * 7 LayerNorm backward (the row kernel, not the gain / shift column sums),
 * 8 softmax cross-entropy, 9 the weight-gradient product of the QKV weight
 * (GPT-J: of the fused QKV + fc1 weight; with SAT_OPT_FUSED_ADAMW, the product
 * whose epilogue applies that weight's AdamW step; its work is counted as the
 * product's FLOPs).  Waits for the stream. */
sat_status sat_model_set_timing(sat_model* m, int32_t kind, int32_t max_launches);
/* Sum of the timed launches' durations (ms), their count and their
 * algorithmic work (FLOPs; bytes for AdamW, LayerNorm and cross-entropy),
 * then resets the counters. */
sat_status sat_model_timing_read(sat_model* m, double* total_ms, int64_t* launches, double* work);

/* ---- profiling (the Trial Runner's runtime estimate, Sec. 3.2, Profiler:
 * epoch times extrapolated from the mean of a few minibatches, which holds
 * because every SGD step of a task does the same work) --------------------
 * Creates a model of cfg on the calling thread's current device (arena and a
 * synthetic batch of the task's shape allocated and freed by the call), runs
 * `warmup` untimed and `steps` timed train steps on hip_stream (borrowed; NULL
 * = the null stream), then destroys it.  The batch comes from a hash of
 * cfg->seed: decoder tokens uniform in [0, vocab) with next-token labels, ViT
 * images uniform in [-1, 1) with uniform class labels.  Step times come from
 * HIP events recorded between consecutive steps on the stream.  Because every
 * step of a task does the same work, the epoch time is extrapolated as the
 * mean step time times ceil(samples_per_epoch / batch) (0 samples: no epoch
 * estimate).  The call waits for the stream.
 * Errors: SAT_EINVAL (configuration, counts, struct_size), SAT_ENOMEM,
 * SAT_EHIP.  Out-params are written only on SAT_OK. */
typedef struct {
  uint32_t struct_size;  /* set by the caller: sizeof(sat_profile_result) */
  int32_t steps;         /* timed steps */
  double step_ms_mean, step_ms_min, step_ms_max;
  double tokens_per_s;   /* rows entering the loss per second (ViT: batch * (patches + 1)) */
  double step_tflop;     /* algorithmic FLOPs of one step, 1e12 */
  double achieved_tflops;
  int64_t steps_per_epoch;
  double epoch_ms;       /* extrapolated epoch time */
  uint64_t arena_bytes;  /* device memory of the model */
  float final_loss;      /* eval loss on the profiling batch after the last step */
} sat_profile_result;
sat_status sat_profile(const sat_config* cfg, void* hip_stream, int32_t warmup, int32_t steps,
                       int64_t samples_per_epoch, sat_profile_result* out);
/* The synthetic batch sat_profile trains on, written into caller device
 * buffers on hip_stream (no wait): decoders int32 tokens [batch, seq_len] and
 * labels [batch, seq_len], where row b is a stream of seq_len + 1 hashed
 * tokens in [0, vocab), inputs its first seq_len and labels its last seq_len
 * (labels[b, s] = inputs[b, s + 1] for s < seq_len - 1); VIT fp32 images
 * [batch, channels, img, img] uniform in [-1, 1) and int32 labels [batch] in
 * [0, vocab).  The Trial Runner's minibatches are the task's own data
 * (Sec. 3.2, Profiler); here they stand in for it with the task's shape.
 * Errors: SAT_EINVAL (configuration, null pointers), SAT_EHIP. */
sat_status sat_profile_batch(const sat_config* cfg, void* inputs, int32_t* labels, void* hip_stream);

const char* sat_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SATURN_H */
