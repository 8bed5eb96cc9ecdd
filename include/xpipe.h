/*
 * xpipe.h -- C ABI of libxpipe, one pipeline stage's training step under
 * XPipe's asynchronous pipelining with Adam-based weight prediction
 * (arXiv:1911.04610), on one AMD Instinct MI355X (gfx950).
 *
 * The step for one mini-batch of T micro-batches (Sec. III-A, III-B):
 *   xpipe_predict_weights(FWD, s_f)   bellwether prediction, Eq. 3, cached
 *   T x xpipe_stage_fwd(x_i)          forward on the cached forward prediction
 *   xpipe_predict_weights(BWD, s_b)   bellwether prediction, Eq. 3, cached
 *   T x xpipe_stage_bwd(x_i, dy_i)    recompute the forward, then the VJP;
 *                                     weight gradients accumulate (Sec. III-A)
 *   xpipe_adam_step(...)              update after the T-th backward (Eq. 4),
 *                                     optionally emitting the next predictions
 * s_f and s_b come from Eq. 1 and Eq. 2 (xpipe_version_difference).
 *
 * Conventions shared by every entry point:
 *   - Device buffers and the HIP stream are owned by the caller.  A stage
 *     handle keeps host-side descriptors and non-owning device pointers; it
 *     allocates no device memory.
 *   - Calls that touch the device enqueue work on the stage's stream and
 *     return; results (including the loss) are in device memory once the
 *     stream has been synchronised by the caller.
 *   - Arguments are checked on the host before anything is enqueued.  A
 *     failed check returns XPIPE_EINVAL (bad argument) or XPIPE_ESTATE (call
 *     out of order) and leaves the device untouched.  A failed launch
 *     returns XPIPE_EHIP.  xpipe_last_error() gives a message for the last
 *     non-OK status of the calling thread.  No C++ exception crosses the ABI.
 *   - Names follow the paper; its first moment v (decay gamma) and second
 *     moment m (decay lambda) of Eq. 4 are called m (beta1) and v (beta2)
 *     here, as in Adam.
 */
#ifndef XPIPE_H
#define XPIPE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  XPIPE_OK = 0,
  XPIPE_EINVAL = 1,       /* invalid argument, shape or layer list */
  XPIPE_ESTATE = 2,       /* call out of order (see each entry point) */
  XPIPE_EHIP = 3,         /* a HIP runtime call or kernel launch failed */
  XPIPE_EUNSUPPORTED = 4  /* valid but not supported by this library */
} xpipe_status;

/* Storage format of activations and activation gradients.  Master weights,
 * moments, gradient accumulator and predictions are fp32 in both.
 *   XPIPE_F32:  fp32 storage; every contraction and reduction is computed in
 *               fp64 (fp64 MFMA) and rounded once, on store.
 *   XPIPE_BF16: bf16 storage; convolutions and linear layers multiply bf16
 *               operands (the fp32 prediction rounded to nearest even) on
 *               MFMA with fp32 accumulation; other layers compute in fp64. */
typedef enum { XPIPE_F32 = 0, XPIPE_BF16 = 1 } xpipe_dtype;

typedef enum { XPIPE_FWD = 0, XPIPE_BWD = 1 } xpipe_dir;

/* Prediction direction of Eq. 3 (the paper prints eps inside the root and
 * bias corrections without the power t; see XPIPE_PRED_LITERAL). */
typedef enum {
  XPIPE_PRED_EQ3 = 0,     /* m_hat / sqrt(v_hat + eps), m_hat = m/(1-beta1^t), v_hat = v/(1-beta2^t) */
  XPIPE_PRED_ADAMDIR = 1, /* m_hat / (sqrt(v_hat) + eps): Adam's own update direction */
  XPIPE_PRED_LITERAL = 2, /* (m/(1-beta1)) / sqrt(v/(1-beta2) + eps): Eq. 4 as printed */
  XPIPE_PRED_SMOOTHED = 3 /* m/(1-beta1): the smoothed gradient of momentum SGD, the
                           * predictor of SpecTrain that Sec. II describes.  With beta1
                           * equal to the rule's momentum and m advanced by the same
                           * gradients from zero, m/(1-beta1) is the heavy-ball buffer
                           * buf of XPIPE_RULE_MOMENTUM_SGD, so W_hat = W - s lr buf
                           * (lr: the rule's). */
} xpipe_pred_mode;

/* Tie rule for the "round" of Eq. 1 and Eq. 2 (undefined in the paper). */
typedef enum {
  XPIPE_ROUND_HALF_UP = 0,   /* ties away from zero (default reading) */
  XPIPE_ROUND_HALF_EVEN = 1,
  XPIPE_ROUND_HALF_DOWN = 2
} xpipe_rounding;

/* Layer kinds of a stage (Sec. IV-C's VGG-16, ResNet-101, Inception-V3).
 * Activations are NHWC; a [n, C] tensor is NHWC with H = W = 1. */
typedef enum {
  XPIPE_LINEAR = 0,     /* y = x W^T + b; W [cout][cin]; input must have H = W = 1 */
  XPIPE_CONV = 1,       /* k x kw kernel, stride 1 or 2, zero padding (k/2, kw/2) or
                           none (pad = 1), cross-correlation; output
                           floor((H + 2 ph - k) / stride) + 1; W [cout][k][kw][cin] (KRSC) */
  XPIPE_BN = 2,         /* batch norm with the micro-batch's mean and biased
                           variance, eps 1e-5; params gamma[C], beta[C] */
  XPIPE_RELU = 3,       /* max(x, 0); derivative 0 at 0 */
  XPIPE_ADD = 4,        /* inputs[0] + inputs[1] (same shape) */
  XPIPE_MAXPOOL2 = 5,   /* 2x2 window, stride 2, floor; gradient to the first
                           maximum in row-major window order */
  XPIPE_AVGPOOL3 = 6,   /* 3x3 window, stride 1, zero padding 1, divisor 9 */
  XPIPE_GAP = 7,        /* mean over H and W: [n,H,W,C] -> [n,1,1,C] */
  XPIPE_CONCAT = 8,     /* channel concatenation of 2..4 inputs, in order */
  XPIPE_SOFTMAX_CE = 9, /* loss = sum over the micro-batch of -log softmax(x)[label],
                           divided by the mini-batch size N = T * micro_batch;
                           must be the last layer */
  XPIPE_MAXPOOL3S2 = 10 /* 3x3 window, stride 2, padding 1 (never chosen) or none
                           (pad = 1), output floor((H + 2p - 3) / 2) + 1; gradient to
                           the first maximum in row-major window order (ResNet-101's
                           stem, Inception-V3's stem and grid reductions) */
} xpipe_layer_kind;

#define XPIPE_MAX_INPUTS 4

typedef struct {
  int32_t kind;                       /* xpipe_layer_kind */
  int32_t n_inputs;                   /* 1, or 2 (ADD), or 2..4 (CONCAT) */
  int32_t inputs[XPIPE_MAX_INPUTS];   /* producer layer indices (< own index); -1 = stage input */
  int32_t cin, cout;                  /* LINEAR, CONV; BN uses cout as its channel count */
  int32_t k;                          /* CONV kernel height (odd, 1..7) */
  int32_t has_bias;                   /* LINEAR, CONV */
  int32_t classes;                    /* SOFTMAX_CE: number of classes (= its input channels) */
  int32_t stride;                     /* CONV: 1 or 2 (0 reads as 1); others 0 or 1 */
  int32_t kw;                         /* CONV kernel width (odd, 1..7; 0 reads as k) */
  int32_t pad;                        /* CONV, MAXPOOL3S2: 0 zero padding ("same": k/2, kw/2;
                                         1 for the pool), 1 none ("valid") */
} xpipe_layer_desc;

/* Optimizer and prediction hyper-parameters (Sec. IV-C: gamma 0.9,
 * lambda 0.999, eps 1e-8).  t is the number of completed updates. */
typedef struct {
  double lr, beta1, beta2, eps;
  int64_t t;
  int32_t mode;                       /* xpipe_pred_mode */
} xpipe_hparams;

typedef struct xpipe_stage* xpipe_stage_t;

/* Eq. 1 (dir = XPIPE_FWD): s = round((size + T - rank/2 - 2) / T);
 * Eq. 2 (dir = XPIPE_BWD): s = round((T + floor(rank/2) - 1) / T).
 * rounding selects the tie rule; ceil_half_rank != 0 reads Eq. 1's rank/2 as
 * ceil(rank/2).  Host only.  EINVAL unless size >= 1, T >= 1, 0 <= rank < size. */
xpipe_status xpipe_version_difference(int32_t size, int32_t T, int32_t rank, int32_t dir,
                                      int32_t rounding, int32_t ceil_half_rank, int32_t* s_out);

/* Validates a layer list for micro-batch shape [micro_batch, H, W, C] and
 * reports the flat parameter count (each tensor zero-padded to a multiple of
 * 64 elements) and the workspace size in bytes.  Host only. */
xpipe_status xpipe_stage_query(const xpipe_layer_desc* layers, int32_t n_layers,
                               int32_t micro_batch, int32_t H, int32_t W, int32_t C,
                               int32_t dtype, int64_t* n_params_padded, size_t* workspace_bytes);

/* Creates a stage.  W, m, v, grad, w_pred_fwd, w_pred_bwd are caller-owned
 * fp32 device buffers of n_params_padded elements (layout: layers in order,
 * weight then bias (CONV/LINEAR) or gamma then beta (BN), each tensor at a
 * 64-element-aligned offset, padding zero).  workspace is caller-owned device
 * memory of at least the queried size, 256-byte aligned.  T >= 1 is the
 * number of micro-batches per mini-batch.  hip_stream is a hipStream_t (NULL
 * = default stream).  grad is zeroed on the stream.  The workspace belongs
 * to the stage until destroy, and calls on one stage must not overlap in time
 * (they share it), which one stream guarantees.  Nothing is predicted yet:
 * call xpipe_predict_weights before the first forward. */
xpipe_status xpipe_stage_create(const xpipe_layer_desc* layers, int32_t n_layers,
                                int32_t micro_batch, int32_t T, int32_t H, int32_t W, int32_t C,
                                int32_t dtype, void* hip_stream,
                                float* W_, float* m, float* v, float* grad,
                                float* w_pred_fwd, float* w_pred_bwd,
                                void* workspace, size_t workspace_bytes, xpipe_stage_t* out);

/* Variant of xpipe_stage_create for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): same arguments and semantics, but no workspace argument.
 * The stage's workspace is the library's static device array of
 * XPIPE_STATIC_WORKSPACE_BYTES bytes (one per GPU, held from the library's
 * load until the process ends), so neither this call nor any later call on
 * the stage allocates or frees device memory, and none creates streams,
 * events or graphs: every kernel runs on hip_stream, in launch order, passes
 * are not recorded (xpipe_stage_set_graphs(st, 1) returns
 * XPIPE_EUNSUPPORTED), and grad is zeroed by a kernel, not a memset.
 * Results are bit-identical to a stage made by xpipe_stage_create.
 * Errors: XPIPE_EINVAL when the stage's workspace (xpipe_stage_query) exceeds
 * XPIPE_STATIC_WORKSPACE_BYTES, or as xpipe_stage_create; XPIPE_ESTATE while
 * another stage made by this call is alive on the current device (a stage
 * keeps state in its workspace between calls, and the array is shared);
 * XPIPE_EHIP when the array's device address cannot be resolved.  The array
 * keeps whatever the previous stage left in it; nothing in it needs to start
 * at zero.  Calls that overlap in time on one GPU (the stage driven from two
 * threads or streams at once) race on the array. */
#define XPIPE_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
xpipe_status xpipe_stage_create_static(const xpipe_layer_desc* layers, int32_t n_layers,
                                       int32_t micro_batch, int32_t T, int32_t H, int32_t W, int32_t C,
                                       int32_t dtype, void* hip_stream, float* W_, float* m, float* v,
                                       float* grad, float* w_pred_fwd, float* w_pred_bwd,
                                       xpipe_stage_t* out);

/* Number of parameter tensors, and offset/count (elements) of tensor idx. */
xpipe_status xpipe_stage_num_param_tensors(xpipe_stage_t st, int32_t* n);
xpipe_status xpipe_stage_param_layout(xpipe_stage_t st, int32_t tensor_idx,
                                      int64_t* offset, int64_t* count);

/* Stage output shape per micro-batch (for a stage ending in SOFTMAX_CE: the
 * logits, [micro_batch, 1, 1, classes]). */
xpipe_status xpipe_stage_output_shape(xpipe_stage_t st, int32_t* n, int32_t* H, int32_t* W,
                                      int32_t* C);

/* Bellwether prediction (Sec. III-B, Eq. 3 with Eq. 4's moments after hp->t
 * completed updates): w_pred_{fwd|bwd} = W - s * lr * dir(m, v).  s >= 0.
 * s = 0, or hp->t = 0 with any mode but LITERAL, gives W exactly.  The
 * result is cached for the mini-batch's other T-1 micro-batches. */
xpipe_status xpipe_predict_weights(xpipe_stage_t st, int32_t which, int32_t s,
                                   const xpipe_hparams* hp);

/* Forward of one micro-batch on the cached forward prediction.
 * x: [micro_batch, H, W, C] in the stage dtype (fp32 or bf16), read only.
 * y: stage output (logits for a loss stage), written.  labels: int32
 * [micro_batch] in [0, classes), required iff the stage ends in SOFTMAX_CE;
 * loss (fp32 scalar, may be NULL) receives this micro-batch's share of the
 * mini-batch loss.  ESTATE before the first forward prediction.  Enqueued on
 * the stage's stream, or on its forward stream once one is set
 * (xpipe_stage_set_fwd_stream). */
xpipe_status xpipe_stage_fwd(xpipe_stage_t st, const void* x, void* y, const int32_t* labels,
                             float* loss);

/* Backward of one micro-batch on the cached backward prediction: the forward
 * is recomputed from x (Sec. IV-C), then the vector-Jacobian product with dy
 * (stage-output gradient, same dtype and shape as y; NULL for a loss stage,
 * which uses labels).  Weight gradients are added into grad.  dx (input
 * gradient, shape of x) is written unless NULL.  ESTATE before the first
 * backward prediction. */
xpipe_status xpipe_stage_bwd(xpipe_stage_t st, const void* x, const void* dy,
                             const int32_t* labels, void* dx);

/* Adam update at the mini-batch boundary (Sec. III-A; Kingma and Ba's update
 * with Eq. 4's moments and bias correction for update number hp->t + 1, eps
 * outside the root), then grad = 0.  With emit_pred != 0 the same pass also
 * writes the next mini-batch's forward and backward predictions (version
 * differences s_fwd_next, s_bwd_next, moments after hp->t + 1 updates), so
 * the next mini-batch needs no xpipe_predict_weights.  With
 * emit_pred = XPIPE_KEEP_PRED the cached predictions stay valid (an interleaved
 * schedule reuses a mini-batch's prediction across an update); with 0 they
 * become invalid.  ESTATE when no backward ran since the last update. */
#define XPIPE_KEEP_PRED 2
xpipe_status xpipe_adam_step(xpipe_stage_t st, const xpipe_hparams* hp, int32_t s_fwd_next,
                             int32_t s_bwd_next, int32_t emit_pred);

/* Update rules of the paper's other settings, with the prediction still built
 * from Adam moments (Sec. III-B): momentum SGD with weight decay (Sec. IV-D's
 * experiments) and RMSProp with momentum (Sec. IV-D's robustness study).
 * The gradient the rule steps on is g = grad + weight_decay * W; the Adam
 * moments m, v (Eq. 4) advance by the same g in the same pass.
 *   MOMENTUM_SGD: buf = momentum * buf + g;  W -= lr * buf
 *   RMSPROP:      sq = alpha * sq + (1 - alpha) * g^2;
 *                 buf = momentum * buf + g / (sqrt(sq) + eps);  W -= lr * buf
 * (heavy-ball momentum without dampening; eps outside the root). */
typedef enum { XPIPE_RULE_MOMENTUM_SGD = 1, XPIPE_RULE_RMSPROP = 2 } xpipe_rule;

typedef struct {
  int32_t rule;          /* xpipe_rule */
  double lr;             /* the rule's step size */
  double momentum;       /* in [0, 1) */
  double weight_decay;   /* >= 0 */
  double alpha;          /* RMSProp: decay of the squared-gradient average, in [0, 1) */
  double eps;            /* RMSProp: > 0, added to the root */
} xpipe_rule_hparams;

/* The update at the mini-batch boundary with rule rp instead of Adam, then
 * grad = 0.  buf (momentum buffer) and, for RMSProp, sq (squared-gradient
 * average) are caller-owned fp32 device buffers of the stage's padded
 * parameter count, zero before the first update and carried between calls
 * (16-byte aligned; sq may be NULL for momentum SGD).  hp supplies the
 * prediction: beta1, beta2 and eps of the Adam moments, the prediction's lr
 * (the paper predicts with the rule's learning rate: pass the same value),
 * the mode, and t = completed updates before this one.  With emit_pred != 0
 * the same pass writes the next mini-batch's forward and backward predictions
 * from the updated W and moments (update count hp->t + 1).  ESTATE when no
 * backward ran since the last update. */
xpipe_status xpipe_rule_step(xpipe_stage_t st, const xpipe_rule_hparams* rp, const xpipe_hparams* hp,
                             float* buf, float* sq, int32_t s_fwd_next, int32_t s_bwd_next,
                             int32_t emit_pred);

xpipe_status xpipe_stage_destroy(xpipe_stage_t st);

/* ---------------------------------------------------------------- partition
 * The paper's model partition (Sec. IV-B): the layers are split across the
 * GPUs into consecutive stages with roughly equal numbers of layers, the later
 * GPUs taking slightly more.  Counted here are the layers with weights (LINEAR,
 * CONV): with L of them over K stages, stage k gets L / K and the last L % K
 * stages one more; a stage starts at its first weighted layer (activations,
 * pools, normalisations and joins stay with the stage of the layer they follow).
 * A cut is valid only where the previous stage's last layer is the one tensor
 * crossing it.  A cut that would split a branch or a skip connection (an
 * Inception module, a residual block) moves to the nearest valid cut at a
 * weighted layer, ties to the earlier one, keeping the cuts in order.
 * first[k] = index of stage k's first layer (first[0] = 0, first[K] = n;
 * K + 1 entries).  Layer inputs are re-indexed by the caller: the previous
 * stage's last layer becomes the stage input (-1).  EUNSUPPORTED when some cut
 * has no valid position left; EINVAL when K exceeds L.  Host only. */
xpipe_status xpipe_partition(const xpipe_layer_desc* layers, int32_t n_layers, int32_t stages, int32_t* first);

/* ---------------------------------------------------------------- schedule
 * The pipeline schedule of Sec. III-A (Fig. 1) as a unit-time model, host
 * only: on a `size`-GPU pipeline, GPU `rank` runs the forward pass of
 * micro-batch i (1-based) at unit 2i + rank and its backward at
 * 2i + 2 size - 1 - rank, which gives the warm-up, the one-forward-one-
 * backward steady phase and the drain, and reproduces the orders the text
 * walks through.  The weights are updated after the backward pass of every
 * T-th micro-batch.  For a bellwether (the first micro-batch of a mini-batch,
 * Sec. III-B) the event carries Eq. 1 / Eq. 2's version difference and the
 * counted one: the updates on this GPU after the pass, up to the unit in which
 * the mini-batch's T-th micro-batch completes its backward pass on GPU 0
 * (s_incl; s_excl leaves out the mini-batch's own update). */
typedef struct {
  int32_t time;          /* pipeline unit */
  int32_t kind;          /* XPIPE_FWD or XPIPE_BWD */
  int32_t micro;         /* micro-batch index, 1-based */
  int32_t mini;          /* mini-batch index, 1-based */
  int32_t bellwether;    /* 1 for the first micro-batch of its mini-batch */
  int32_t update_after;  /* 1 if the weights are updated right after this backward */
  int32_t version;       /* updates applied on this GPU before the pass */
  int32_t s_eq;          /* bellwether: Eq. 1 (forward) or Eq. 2 (backward) */
  int32_t s_excl, s_incl;/* bellwether: counted version differences */
} xpipe_sched_event;

/* Events of GPU `rank` for `minibatches` mini-batches of T micro-batches, in
 * time order: *count = 2 T minibatches.  With out = NULL only the count is
 * returned; otherwise capacity must hold them.  rounding / ceil_half_rank as
 * in xpipe_version_difference.  No device work. */
xpipe_status xpipe_schedule(int32_t size, int32_t T, int32_t rank, int32_t minibatches, int32_t rounding,
                            int32_t ceil_half_rank, xpipe_sched_event* out, int32_t capacity,
                            int32_t* count);

/* Host arrays (n_micro entries, indexed by micro-batch - 1) of device
 * pointers for xpipe_stage_run. */
typedef struct {
  int32_t n_micro;
  const void* const* x;           /* stage inputs (required) */
  const void* const* dy;          /* upstream gradients; NULL for a loss stage */
  const int32_t* const* labels;   /* NULL unless the stage ends in SOFTMAX_CE */
  void* const* y;                 /* forward outputs (required) */
  float* loss;                    /* device array [n_micro] of per-micro-batch losses, or NULL */
  void* const* dx;                /* input gradients, or NULL */
} xpipe_run_io;

/* Runs a schedule's events on one stage in order, as GPU `rank` would: a
 * bellwether's forward (backward) pass first predicts with its s_eq and caches
 * the result (xpipe_predict_weights), the other micro-batches of the mini-batch
 * reuse the cache even after an update in between (Sec. III-B), and the
 * update (Adam, or rule when not NULL, with buf / sq as in xpipe_rule_step)
 * follows every event with update_after, keeping both caches.  hp->t counts
 * the updates before the run; hp's lr is the prediction's.  draft != 0 takes
 * the variant of the draft text instead: a forward micro-batch that finds its
 * mini-batch's cached prediction older than the latest update predicts again
 * from the current weights with the bellwether's s reduced by the updates since
 * (at least 0), and the later ones reuse that. */
xpipe_status xpipe_stage_run(xpipe_stage_t st, const xpipe_sched_event* events, int32_t n_events,
                             const xpipe_run_io* io, const xpipe_hparams* hp,
                             const xpipe_rule_hparams* rule, float* buf, float* sq, int32_t draft);

/* Flat-buffer forms of the two bandwidth-bound kernels, on n fp32 elements
 * (any n >= 0).  The kernels stream 16-byte chunks from the base pointers:
 * every fp32 buffer must be 16-byte aligned (a bf16 output 8-byte aligned),
 * else the call returns XPIPE_EINVAL before anything is enqueued.  n need not
 * be a multiple of the chunk; the tail is handled element by element.
 * xpipe_predict_flat: out = W - s * lr * dir(m, v) (Eq. 3); out_bf16 (may be
 * NULL) receives the same values rounded to bf16 (uint16 bit patterns).
 * xpipe_adam_flat: W, m, v updated in place from G (update hp->t + 1); G is
 * zeroed when zero_grad != 0; when pred_fwd / pred_bwd are not NULL they
 * receive predictions with s_fwd / s_bwd from the updated state. */
xpipe_status xpipe_predict_flat(const float* W, const float* m, const float* v, float* out,
                                uint16_t* out_bf16, int64_t n, int32_t s, const xpipe_hparams* hp,
                                void* hip_stream);
xpipe_status xpipe_adam_flat(float* W, float* m, float* v, float* G, int64_t n,
                             const xpipe_hparams* hp, int32_t zero_grad,
                             float* pred_fwd, int32_t s_fwd, float* pred_bwd, int32_t s_bwd,
                             void* hip_stream);
/* xpipe_rule_flat: xpipe_rule_step's pass on flat buffers: W, buf, sq
 * (RMSProp only; may be NULL otherwise), m, v updated in place from G; G
 * zeroed when zero_grad != 0; predictions as in xpipe_adam_flat. */
xpipe_status xpipe_rule_flat(float* W, float* buf, float* sq, float* m, float* v, float* G, int64_t n,
                             const xpipe_rule_hparams* rp, const xpipe_hparams* hp, int32_t zero_grad,
                             float* pred_fwd, int32_t s_fwd, float* pred_bwd, int32_t s_bwd,
                             void* hip_stream);

/* Optional per-kernel timing (measurement support, not part of the method):
 * while enabled, hipEvents bracket every kernel the stage launches on its
 * stream.  xpipe_stage_timing_count waits for the recorded launches and
 * reports how many distinct kernels ran; xpipe_stage_timing_entry gives, for
 * entry i (0 <= i < count, sorted by name), the kernel name (a static string
 * owned by the library, valid until the stage is destroyed), the summed
 * duration in ms, the launch count and the algorithmic work (flops for the
 * GEMM kernels k_conv_gemm / k_wgrad, bytes moved for all others).
 * Enabling (or re-enabling) clears the accumulated entries. */
xpipe_status xpipe_stage_set_timing(xpipe_stage_t st, int32_t enable);

/* Recorded passes (on by default; the environment variable XPIPE_GRAPHS=0
 * turns them off at creation).  xpipe_stage_fwd and xpipe_stage_bwd capture
 * each distinct combination of their pointer arguments once into a HIP graph
 * (all launch lanes, same kernels and arguments as the eager launches) and
 * replay it on later calls, so a pass costs one graph launch on the host.  At
 * most 64 graphs are kept (least recently used are dropped).  Results are
 * identical with or without graphs.  A pointer argument must keep describing
 * the same buffer between calls that pass it (a freed and reallocated buffer
 * of the same size at the same address is fine).  Timing mode runs eagerly.
 * xpipe_stage_set_graphs turns recording on or off and drops the kept graphs. */
xpipe_status xpipe_stage_set_graphs(xpipe_stage_t st, int32_t enable);

/* Forward passes on a stream of their own.  In the pipeline's steady state a
 * stage alternates the forward of one micro-batch with the backward of
 * another (Sec. III-A); the two read different weight versions (the cached
 * forward and backward predictions, Sec. III-B) and share no activations
 * (the backward recomputes its forward), so they may run concurrently.
 * With a workspace given, xpipe_stage_fwd enqueues on a stream the stage
 * owns (one of its launch lanes, returned in *hip_stream when hip_stream is
 * not NULL; valid until the stage is destroyed) and keeps its activations and
 * scratch in `workspace` (caller-owned device memory of at least
 * xpipe_stage_query's workspace_bytes, 256-byte aligned, used by this stage
 * until this call is made again or the stage is destroyed).  Every other
 * call stays on the stage's stream.  Ordering kept by the library: a forward
 * starts after the last call that wrote the forward prediction
 * (xpipe_predict_weights(FWD), or an update with emit_pred = 1), and such a
 * call waits for the forwards enqueued before it.  The caller orders the
 * forward's inputs (x, labels) and outputs (y, loss) against the returned
 * stream itself.  Results are identical to forwards on the stage's stream.
 * workspace = NULL goes back to one stream (*hip_stream = NULL).  The call
 * synchronises both streams and drops the recorded passes.  While it is set,
 * the forward and the backward's recomputed forward each run as one chain of
 * launches (the BNs over a merged GEMM's slices applied by one launch), which
 * is faster beside the backward.  Timing mode runs the same launches on the
 * stage's stream.  EINVAL: workspace too small or misaligned; EUNSUPPORTED
 * for a stage of xpipe_stage_create_static. */
xpipe_status xpipe_stage_set_fwd_stream(xpipe_stage_t st, void* workspace, size_t workspace_bytes,
                                        void** hip_stream);
xpipe_status xpipe_stage_timing_count(xpipe_stage_t st, int32_t* n);
xpipe_status xpipe_stage_timing_entry(xpipe_stage_t st, int32_t i, const char** kernel, double* ms,
                                      int64_t* launches, double* work);

/* Measurement probes (not part of the method): the attainable peaks the
 * benchmark reports next to the published ones.
 * xpipe_probe_copy: dst[i] = src[i] for `bytes` bytes (a multiple of 16; both
 * 16-byte aligned, not overlapping), one 16-byte chunk per thread.
 * xpipe_probe_mfma: every wave of `waves` runs `iters` rounds of eight
 * independent v_mfma_f32_32x32x16_bf16 (32768 flops each) on register
 * operands and writes one float per wave to out[waves] (so the work is kept);
 * flops = waves * iters * 8 * 32768.  Both enqueue on hip_stream. */
xpipe_status xpipe_probe_copy(const void* src, void* dst, int64_t bytes, void* hip_stream);
/* xpipe_probe_stream: a bare stream of a pass's shape, the attainable HBM
 * rate the prediction and update passes are compared with: each of nsrc
 * (0..4) fp32 buffers of n elements is read once and each of ndst (1..6) is
 * written once (the element-wise sum of the sources), 16 bytes per thread and
 * buffer with the passes' non-temporal hints.  n a multiple of 4; every
 * buffer 16-byte aligned and non-overlapping; src / dst are host arrays of
 * device pointers.  Prediction: 3 reads, 1 write; Adam: 4 and 3; Adam fused
 * with zeroing the gradient and both predictions: 4 and 6. */
xpipe_status xpipe_probe_stream(const float* const* src, int32_t nsrc, float* const* dst, int32_t ndst,
                                int64_t n, void* hip_stream);

xpipe_status xpipe_probe_mfma(float* out, int32_t waves, int32_t iters, void* hip_stream);

/* xpipe_probe_graph: what a fork/join costs inside a recorded HIP graph, the
 * structure the stage's launch lanes become.  Two graphs are recorded and
 * each replayed 2 + 5 times on hip_stream (the last 5 timed): `reps` diamonds
 * of (one launch, then `width` branches on separate streams of `len`
 * launches each, joined back), and the same launches as one chain.  Every
 * launch is 256 workgroups of 256 threads doing `spin` dependent fp32
 * multiply-adds (0: an empty launch).  scratch: device memory of at least
 * 2048 floats (read and written).  us_out (host, 2 doubles): microseconds per
 * diamond with branches, then as one chain.  1 <= width <= 3, 1 <= len <= 8,
 * 1 <= reps <= 256, spin >= 0; creates and destroys its own streams (default
 * priority), events and graphs, runs after the work already enqueued on
 * hip_stream and returns when its own work has finished. */
xpipe_status xpipe_probe_graph(float* scratch, int32_t width, int32_t len, int32_t reps, int32_t spin,
                               double* us_out, void* hip_stream);

/* Message for the last non-OK status returned on the calling thread. */
const char* xpipe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* XPIPE_H */
