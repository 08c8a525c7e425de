/*
 * unifiednn.h -- C ABI of the fused N-model training step on one MI355X (gfx950).
 *
 * The library trains N independent models that share one input batch as one
 * "hybrid" model: every call to un_step runs, for ALL models at once, the body
 * of the paper's hybrid training algorithm (UnifiedNN, Trainer section,
 * Algorithm 2): each sub-model's gradient of its own loss on the batch, then
 * each sub-model's SGD update theta^m <- theta^m - eta * g^m. The models are
 * merged only in the sense of the Model Unifier (Algorithm 1): their layer
 * graphs are a disjoint union with one global input; no value ever flows from
 * one model to another, and each model trains exactly as it would alone.
 *
 * Conventions shared by every call:
 *   - Every call returns a un_status; UN_OK is 0. On failure the message is
 *     available from un_last_error(ctx) until the next call on that context.
 *     No C++ exception crosses this boundary.
 *   - A validation failure (UN_ERR_INVALID, UN_ERR_RANGE, UN_ERR_BUFSIZE,
 *     UN_ERR_STATE, UN_ERR_UNSUPPORTED) changes no state. A HIP runtime failure
 *     returns UN_ERR_DEVICE and poisons the context: every later call except
 *     un_last_error and un_destroy returns UN_ERR_DEVICE.
 *   - Host pointers are owned by the caller; the library copies what it needs
 *     before returning, except where a call says it is asynchronous.
 *   - A context owns all of its device memory (one arena, allocated in
 *     un_create, freed in un_destroy) and one HIP stream.
 *   - One context must not be used from two threads at once.
 */
#ifndef UNIFIEDNN_H
#define UNIFIEDNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct un_ctx un_ctx;

typedef enum {
  UN_OK = 0,
  UN_ERR_INVALID = 1,     /* malformed argument or spec */
  UN_ERR_STATE = 2,       /* call made in the wrong order (e.g. step before load) */
  UN_ERR_OOM = 3,         /* the arena does not fit in device memory */
  UN_ERR_DEVICE = 4,      /* HIP runtime error; the context is poisoned */
  UN_ERR_RANGE = 5,       /* index or label out of range */
  UN_ERR_BUFSIZE = 6,     /* caller's buffer too small / wrong element count */
  UN_ERR_UNSUPPORTED = 7  /* well-formed, but a layer pattern this library does not fuse */
} un_status;

/* Arithmetic of the step.
 * UN_F32:            every tensor fp32; fp32 MFMA with fp32 accumulation.
 * UN_BF16_F32MASTER: activations, activation gradients and the weights the
 *                    GEMMs read are bf16 (round to nearest even); accumulation,
 *                    logits, the loss, dW/db and the master weights stay fp32. */
typedef enum { UN_F32 = 0, UN_BF16_F32MASTER = 1 } un_precision;

/* Layer ops of a sub-model, in the order of a PyTorch nn.Sequential (the paper
 * defines every sub-model as a sequential module, Design overview). */
typedef enum {
  UN_LINEAR = 0,   /* out = features;   weight [out, in], bias [out] */
  UN_CONV2D = 1,   /* out = channels, kernel k x k, stride 1, zero padding pad;
                      weight [out, in, k, k], bias [out]; cross-correlation */
  UN_RELU = 2,
  UN_MAXPOOL2 = 3, /* 2x2, stride 2, floor mode; ties: first max in row-major order */
  UN_FLATTEN = 4,  /* NCHW (c, h, w) order */
  /* A skip connection around the layers between the two markers (a residual
   * block): the layers run on the block's input x as usual and, at the END
   * marker, x is added to their result, before any ReLU that follows the END
   * marker. In PyTorch terms the markers wrap the enclosed layers in a module
   * whose forward returns inner(x) + x. The enclosed layers are one or more
   * [Linear, optional ReLU] or [Conv2d, optional ReLU] blocks (no ReLU
   * directly before the END marker, no MaxPool2 inside or right after), the
   * result has the shape of x, x is the output of a Linear or Conv2d block (a
   * block never starts at the network input or after a Flatten), the block
   * does not end at the logits layer and blocks do not nest; other patterns
   * return UN_ERR_UNSUPPORTED (shape mismatches UN_ERR_INVALID). The markers
   * have no parameters. */
  UN_RESIDUAL_BEGIN = 5,
  UN_RESIDUAL_END = 6,
  /* View flat features as a sequence of `out` tokens of F / out features each
   * (PyTorch's Unflatten(1, (out, F / out)); F must divide). A Linear layer on
   * a sequence acts on every token (PyTorch's Linear on [B, T, d]); Flatten
   * turns a sequence back into T * d features, token by token. Allowed on the
   * network input or on a Linear layer's flat output. Token features (the
   * result of UN_UNFLATTEN and every Linear on a sequence) must be a multiple
   * of 8. */
  UN_UNFLATTEN = 7,
  /* Single-head self-attention on a sequence [T, d] (PyTorch's
   * MultiheadAttention(d, 1 head) called on (x, x, x), no mask, no dropout):
   * [Q K V] = x W_in^T + b_in, A = softmax(Q K^T / sqrt(d)) V over the
   * tokens of each sample, y = A W_out^T + b_out. Parameters in state_dict
   * order: in_proj_weight [3d, d], in_proj_bias [3d], out_proj.weight
   * [d, d], out_proj.bias [d]. A ReLU may follow, and residual markers may
   * enclose it (x + attn(x)). T <= 64 and the per-sample working set
   * (4 T (d + 1) + 2 T (T + 1) floats) must fit 160 KiB of LDS. */
  UN_SELF_ATTENTION = 8
} un_op;

typedef struct {
  int32_t op;      /* un_op */
  int32_t out;     /* UN_LINEAR: out features; UN_CONV2D: out channels; UN_UNFLATTEN: tokens; else 0 */
  int32_t kernel;  /* UN_CONV2D only */
  int32_t pad;     /* UN_CONV2D only */
} un_layer;

typedef struct {
  int32_t n_layers;
  const un_layer* layers;   /* read during un_create only */
  int32_t num_classes;      /* must equal the last Linear layer's out */
  uint64_t init_seed;       /* seed of the library's own initialisation */
} un_model_spec;

/* The one shared input: x is [batch, in_c, in_h, in_w] (images) or, with
 * in_h = in_w = 1, [batch, in_c] (feature vectors). */
typedef struct {
  int32_t batch;
  int32_t in_c, in_h, in_w;
  int32_t precision;        /* un_precision */
} un_input_spec;

/* Build the hybrid model (Model Unifier, Algorithm 1): validate every spec,
 * plan the fused schedule and the one device arena, allocate it, and
 * initialise each model's parameters from its init_seed (Kaiming-uniform
 * weights U(+-sqrt(6/fan_in)), biases U(+-1/sqrt(fan_in)), drawn with a
 * counter-based generator; callers needing exact start values use
 * un_set_params). Supported layer patterns per model: zero or more
 * [Conv2d, optional ReLU, optional MaxPool2] blocks, a Flatten if any conv is
 * present, then one or more [Linear, optional ReLU] blocks, the last Linear
 * having no ReLU and out == num_classes; residual markers may enclose runs of
 * the Linear blocks or of the Conv2d blocks as UN_RESIDUAL_BEGIN describes.
 * Size restrictions (UN_ERR_UNSUPPORTED otherwise): when some model starts
 * with a Linear layer, in_c * in_h * in_w is a multiple of 8; a Linear layer
 * reading a flattened conv output reads a multiple of 8 features
 * (channels * height * width of that output); batch <= 2^20.
 * The context's device is the one current at this call; the context's own
 * stream is created on it.
 * On success *out owns the context. Errors: UN_ERR_INVALID, UN_ERR_UNSUPPORTED,
 * UN_ERR_OOM, UN_ERR_DEVICE (then *out is NULL). */
un_status un_create(const un_model_spec* specs, int32_t n_models,
                    const un_input_spec* in, un_ctx** out);

/* As un_create, for models that train on different datasets (Algorithm 2
 * gives every sub-model its own batches; each sub-model's hyper-parameters
 * include its input size and batch size, Model Unifier section). inputs[g]
 * (g < n_groups) describes input group g: its batch size and sample shape
 * (precision equal for all groups). Model i reads group group_of[i] (host
 * int32 [n_models]; may be NULL when n_groups == 1). Each group is one
 * dataset: its batch is copied to the device once (un_load_group_batch) and
 * read by all of its models, and the first hidden Linear layers of a group's
 * models still run as one GEMM. Models of different groups differ in batch
 * size and input shape freely. n_groups == 1 is un_create. Every group must
 * hold at least one model. Errors as un_create, and UN_ERR_RANGE (a group
 * index out of range). */
un_status un_create_grouped(const un_model_spec* specs, int32_t n_models, const un_input_spec* inputs,
                            int32_t n_groups, const int32_t* group_of, un_ctx** out);

/* Device memory a context for these models would take, computed on the host
 * without touching the device (the planner of un_create, dry): *arena_bytes is
 * exactly what un_create allocates (un_arena_bytes), *state_bytes (may be
 * NULL) what the first non-SGD optimizer adds (un_set_optimizer). The paper
 * sizes a hybrid as the maximum over its sub-models because its scheduler
 * trains them one at a time (Trainer section, memory requirement); a fused
 * step holds all N at once, so here it is one shared input plus the sum over
 * the models. Use it to admit models onto a GPU before creating anything.
 * Errors: as un_create's validation. */
un_status un_plan_bytes(const un_model_spec* specs, int32_t n_models, const un_input_spec* in,
                        size_t* arena_bytes, size_t* state_bytes);

/* un_plan_bytes for un_create_grouped's arguments. */
un_status un_plan_bytes_grouped(const un_model_spec* specs, int32_t n_models, const un_input_spec* inputs,
                                int32_t n_groups, const int32_t* group_of, size_t* arena_bytes,
                                size_t* state_bytes);

/* Copy one shared batch to the device, once for all N models (Memory
 * conservation section: a common dataset is loaded only once). x is host fp32
 * laid out as in un_input_spec, y is host int32 [batch]. Labels are checked on
 * the host: a label outside [0, num_classes) of any model returns UN_ERR_RANGE
 * and leaves the previously loaded batch in place. Synchronous. With several
 * input groups: UN_ERR_INVALID (use un_load_group_batch). */
un_status un_load_batch(un_ctx* ctx, const float* x, const int32_t* y);

/* un_load_batch for input group g of a un_create_grouped context: x [batch_g,
 * shape of group g] fp32, y int32 [batch_g], labels checked against the
 * models of group g. A step runs only once every group has a batch loaded;
 * loaded batches stay until replaced. Errors as un_load_batch, and
 * UN_ERR_RANGE (g). */
un_status un_load_group_batch(un_ctx* ctx, int32_t g, const float* x, const int32_t* y);

/* As un_load_batch, with x and y already in device memory (same layouts). The
 * buffers are read on the context's stream (un_get_stream): the caller orders
 * the work that writes them before this call (e.g. a stream or device
 * synchronisation, or by running that work on the context's stream). The
 * labels are range-checked after a device-to-host copy; the call returns when
 * the batch has been converted, after which x_dev and y_dev may be reused. */
un_status un_load_batch_device(un_ctx* ctx, const float* x_dev, const int32_t* y_dev);

/* Labels per model for the batches already loaded (Algorithm 2 gives every
 * sub-model its own batches; the inputs x stay those of the input groups).
 * y is host int32: model 0's labels, then model 1's, ..., each row as long as
 * its model's batch ([N][batch] with one input group), each label in
 * [0, num_classes of the model) or UN_ERR_RANGE (nothing changes). They
 * replace the labels of the groups' batches until the next un_load_batch /
 * un_load_group_batch, which goes back to the group labels. Synchronous.
 * UN_ERR_STATE before every group has a batch. */
un_status un_load_labels(un_ctx* ctx, const int32_t* y);

/* One fused training step of all N models on the loaded batch (Algorithm 2's
 * loop body for every sub-model): forward, per-model mean softmax
 * cross-entropy, backward, per-model SGD with learning rate lr.
 * If losses is non-NULL it receives, per model, the loss at the parameters
 * BEFORE this step's update (host fp32 [N]); the call then waits for the step.
 * With losses == NULL the step is only enqueued on the context's stream.
 * The update theta <- fma(-lr, g, theta) (fp32) is applied inside the
 * weight-gradient kernels; gradients are stored only when kept (un_keep_grads).
 * Errors: UN_ERR_STATE (no batch loaded), UN_ERR_INVALID (lr not finite). */
un_status un_step(un_ctx* ctx, float lr, float* losses);

/* As un_step with a learning rate per model: model i updates with lrs[i]
 * (host fp32 [N], each finite, else UN_ERR_INVALID and nothing runs). The
 * paper indexes the rate by the batch (Algorithm 2) and gives every sub-model
 * its own hyper-parameters; a schedule eta_t is this call with the step's
 * rates. The rates are copied when the call returns (the host array may be
 * reused at once); inactive models ignore theirs. */
un_status un_step_lr(un_ctx* ctx, const float* lrs, float* losses);

/* Active set of the following steps (Trainer section: a scheduler - first
 * come first serve, priority, shortest job first, round robin - decides which
 * sub-models train; a sub-model whose training is done is returned through the
 * Model Separator while the others go on). mask is host uint8 [N]; mask[i] != 0
 * keeps model i in the steps. A model outside the set is neither run nor
 * updated (its parameters stay bitwise as they are), un_step reports NaN as its
 * loss, and un_get_params returns it at any time. The active models compute
 * exactly what they compute in any other set. Re-plans the launch tables in
 * the context's arena (no allocation); waits for the stream; gradients kept
 * by earlier steps are no longer available. Default: all models active.
 * Errors: UN_ERR_INVALID (mask NULL or no model active). */
un_status un_set_active(un_ctx* ctx, const uint8_t* mask);

/* The trained parameters of model i (Model Separator section: the sub-model's
 * parameters copied back into the user's original layout): fp32, PyTorch
 * state_dict order (per parameterised layer: weight then bias; Linear
 * [out, in], Conv2d [out, in, k, k]; a Linear after Flatten indexes its input
 * in NCHW order). With dst == NULL only *n_elems is set. Waits for the stream.
 * Errors: UN_ERR_RANGE (i), UN_ERR_BUFSIZE (cap_elems too small). */
un_status un_get_params(un_ctx* ctx, int32_t i, float* dst, size_t cap_elems, size_t* n_elems);

/* Overwrite model i's parameters (same layout as un_get_params; n_elems must be
 * the exact count). Used to start from given values, e.g. to compare with a
 * reference trained elsewhere. Errors: UN_ERR_RANGE, UN_ERR_BUFSIZE. */
un_status un_set_params(un_ctx* ctx, int32_t i, const float* src, size_t n_elems);

/* Keep (1) or stop keeping (0) the gradients: the update is fused into the
 * weight-gradient kernels, so by default gradients are applied and never
 * stored. While enabled, un_step also stores every gradient (4 more bytes of
 * traffic per parameter) for un_get_grads. Default 0. */
un_status un_keep_grads(un_ctx* ctx, int32_t enable);

/* The gradient of model i computed by the last un_step (same layout and order
 * as un_get_params). Waits for the stream. Errors as un_get_params, and
 * UN_ERR_STATE before the first step, when that step did not keep gradients
 * (un_keep_grads), or after un_set_active; model i must have been active in
 * that step. */
un_status un_get_grads(un_ctx* ctx, int32_t i, float* dst, size_t cap_elems, size_t* n_elems);

/* Optimizer of one model (each sub-model has its own optimizer: Model
 * Unifier section; the paper's models use SGD, Adam for the transformer).
 * Element-wise, fp32, with g the gradient and lr the step's rate of the model:
 *   UN_OPT_SGD       w <- fma(-lr, g, w)                       (the default)
 *   UN_OPT_MOMENTUM  b <- fma(momentum, b, g);  w <- fma(-lr, b, w)
 *                    (b starts at 0: the first step is plain SGD)
 *   UN_OPT_ADAM      m <- fma(beta1, m, (1-beta1) g);  v <- fma(beta2, v, (1-beta2) g^2);
 *                    w <- w - (lr / (1 - beta1^t)) * m / (sqrt(v) / sqrt(1 - beta2^t) + eps)
 *                    (t = the model's update count, from 1; m, v start at 0)
 * These are torch.optim.SGD (momentum, no dampening, not Nesterov) and
 * torch.optim.Adam (no weight decay, no amsgrad) without weight decay. */
typedef enum { UN_OPT_SGD = 0, UN_OPT_MOMENTUM = 1, UN_OPT_ADAM = 2 } un_opt_kind;
typedef struct {
  int32_t kind;      /* un_opt_kind */
  float momentum;    /* UN_OPT_MOMENTUM: in [0, 1) */
  float beta1, beta2;/* UN_OPT_ADAM: in [0, 1) */
  float eps;         /* UN_OPT_ADAM: > 0 */
} un_optimizer;

/* Give model i a fresh optimizer: its state is zeroed and its update count
 * reset (as a new torch optimizer would). The first non-SGD optimizer of a
 * context allocates the state of all models (two fp32 values per parameter,
 * outside the arena) and rebuilds the step's tables. Waits for the stream.
 * Errors: UN_ERR_RANGE (i), UN_ERR_INVALID (kind or hyper-parameters),
 * UN_ERR_OOM. */
un_status un_set_optimizer(un_ctx* ctx, int32_t i, const un_optimizer* opt);

/* Model i's optimizer state for a checkpoint: k * n_params floats, k = 0
 * (SGD), 1 (momentum buffer) or 2 (Adam: first moments, then second
 * moments), each block in un_get_params layout and order; *step receives the
 * number of updates the model has taken under this optimizer. With dst ==
 * NULL only *n_elems and *step are set. Waits for the stream.
 * Errors: UN_ERR_RANGE, UN_ERR_BUFSIZE. */
un_status un_get_opt_state(un_ctx* ctx, int32_t i, float* dst, size_t cap_elems, size_t* n_elems, int64_t* step);

/* Restore model i's optimizer state and update count (layout as
 * un_get_opt_state for the model's current optimizer; n_elems exact), e.g.
 * to resume from a checkpoint. Errors: UN_ERR_RANGE, UN_ERR_BUFSIZE,
 * UN_ERR_INVALID (negative step, NULL src). */
un_status un_set_opt_state(un_ctx* ctx, int32_t i, const float* src, size_t n_elems, int64_t step);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): un_step
 * with the step's workspace - the split-K partial sums of conv weight
 * gradients and of Linear weight gradients with long contractions, and the
 * per-model loss partials, which a step writes and reads back within
 * itself - in one static device array of the library (32 MiB per device,
 * held until the process ends) instead of the context's arena. Results equal
 * un_step's bit for bit. Allocates nothing: the array is a file-scope
 * device variable whose address is looked up once per device. Every call on
 * one device shares that array (it keeps the last call's contents; nothing in
 * it needs to start at zero), so calls that overlap on one device - steps of
 * two contexts on two streams at once - race; serialise them.
 * Errors: as un_step, and UN_ERR_UNSUPPORTED (nothing runs) when this
 * context's workspace exceeds the array (wide CNN hybrids; use un_step). */
un_status un_step_scratch(un_ctx* ctx, float lr, float* losses);

/* Number of parameters of model i. */
un_status un_param_count(const un_ctx* ctx, int32_t i, size_t* n_elems);

/* Bytes of the device arena (the whole footprint of the hybrid model). */
un_status un_arena_bytes(const un_ctx* ctx, size_t* bytes);

/* Wait until all work enqueued on the context's stream has finished. */
un_status un_sync(un_ctx* ctx);

/* The context's HIP stream (a hipStream_t), so a caller can order its own work
 * or record events around steps. Owned by the context unless set by
 * un_set_stream. */
un_status un_get_stream(const un_ctx* ctx, void** hip_stream);

/* Run the context's work from now on on the caller's stream (a hipStream_t on
 * the context's device, e.g. a PyTorch stream), so that it is ordered with
 * the caller's other work without host synchronisation; NULL returns to the
 * context's own stream. The caller keeps the stream alive while the context
 * uses it. Waits for the work already enqueued on the previous stream.
 * Invalidates a captured step (un_graph_capture). */
un_status un_set_stream(un_ctx* ctx, void* hip_stream);

/* Capture one step (exactly what un_step(ctx, lr, NULL) enqueues) as a HIP
 * graph owned by the context, for callers whose steps are bounded by launch
 * latency: un_graph_step then replays it with one launch. The graph holds the
 * rate lr, the active set, the optimizers, un_keep_grads and the label mode
 * of this moment; un_set_active, un_set_optimizer state allocation,
 * un_set_stream, or a change of un_keep_grads or of the label mode
 * (un_load_labels / un_load_batch) make it stale. The batch, parameters and
 * labels it reads are the context's buffers: load new batches and set
 * parameters as usual between replays. Not available while a model has a
 * momentum or Adam optimizer (their per-step hyper-parameters would be frozen).
 * Errors: UN_ERR_STATE (no batch), UN_ERR_INVALID (lr), UN_ERR_UNSUPPORTED,
 * UN_ERR_DEVICE. */
un_status un_graph_capture(un_ctx* ctx, float lr);

/* Replay the captured step: the same result as the un_step call it recorded
 * (losses as un_step). Errors: UN_ERR_STATE (nothing captured, or stale). */
un_status un_graph_step(un_ctx* ctx, float* losses);

/* Kernel classes for per-kernel timing. */
typedef enum {
  UN_K_GEMM_FWD = 0,    /* grouped GEMM, forward levels */
  UN_K_GEMM_BWD = 1,    /* grouped GEMM, dgrad + wgrad levels */
  UN_K_CONV_FWD = 2,
  UN_K_CONV_DGRAD = 3,
  UN_K_CONV_WGRAD = 4,
  UN_K_CE = 5,          /* softmax cross-entropy */
  UN_K_SGD = 6,         /* weight copy refresh (SGD kernel without gradient) */
  UN_K_OTHER = 7,       /* split-K reduction with the fused update (conv, long-contraction Linear) */
  UN_K_ATTN = 8,        /* self-attention core, forward and backward */
  UN_K_COUNT = 9
} un_kernel_class;

/* Enable (1) or disable (0) per-kernel timing: while enabled, every launch is
 * bracketed by HIP events on the context's stream and its duration is added to
 * its class. Enabling resets the totals. */
un_status un_profile_enable(un_ctx* ctx, int32_t enable);

/* Totals since un_profile_enable(ctx, 1): summed milliseconds and launch count
 * of one kernel class. Waits for the stream. */
un_status un_profile_read(un_ctx* ctx, int32_t kernel_class, double* total_ms, int64_t* launches);

/* Free the context and its arena. NULL is accepted. */
void un_destroy(un_ctx* ctx);

/* Message of the last failed call on ctx (or of the last failed un_create when
 * ctx is NULL). Never NULL; owned by the library. */
const char* un_last_error(const un_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* UNIFIEDNN_H */
