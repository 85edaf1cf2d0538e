/*
 * ekya.h - C ABI of the MI355X retraining / micro-profiling / inference library.
 *
 * The library runs, on one gfx950 GPU, the data-parallel hot path of Ekya
 * (Bhardwaj et al., "Ekya: Continuous Learning of Video Analytics Models on
 * Edge Compute Servers"): retraining the last k stages of a ResNet18 frame
 * classifier on a uniformly subsampled window of labelled frames (sections 3.1
 * and 4.3), micro-profiling many such retraining configurations for a few
 * epochs on small subsets (section 4.3, "Micro-profiling design"), and
 * batched inference at a configured resolution (sections 1 and 3.1,
 * inference configurations).
 *
 * Conventions shared by every call
 *  - Pointers marked "device" are HIP device pointers (e.g. torch tensors'
 *    data_ptr()); pointers marked "host" are CPU memory.  The caller owns every
 *    buffer and keeps it alive until the call returns (synchronous calls) or
 *    until `stream` has been synchronised (asynchronous calls).
 *  - The library owns only the memory behind an ekya_ctx: one workspace arena
 *    (every device buffer a call needs -- activations, gradients, optimizer
 *    state, frozen-prefix feature caches -- is planned inside it), internal
 *    streams and events.  Calls on one context run in turn on the GPU: each
 *    call's work is ordered after the previous call's.
 *  - Arguments are validated before any GPU work; on failure nothing is
 *    launched and the status names the problem (see ekya_last_error).
 *  - A context is used by one host thread at a time.
 *  - Frames are NHWC with 3 channels, element type per `precision`
 *    (EKYA_FP32: float, EKYA_BF16: bfloat16).  Labels are int32 in
 *    [0, n_classes).
 *  - Weights ("canonical layout"): one flat fp32 array holding the ResNet18
 *    parameters and BatchNorm running statistics in torchvision state_dict
 *    order (num_batches_tracked omitted): conv weights [K][C][R][S], BatchNorm
 *    weight, bias, running_mean, running_var, ..., fc.weight [classes][512],
 *    fc.bias.  ekya_weights_count gives its length (11,189,190 floats for 6
 *    classes).
 *  - Stages: k_trainable counts ResNet18 stages from the head over
 *    [stem, layer1, layer2, layer3, layer4, fc]: 1 = fc only, 2 = layer4 and
 *    fc, 3 = layer3 and above, ..., 6 = every stage.  Frozen stages run
 *    BatchNorm in eval mode and are computed once per frame (the frozen-prefix
 *    feature cache); trainable stages run BatchNorm in train mode and are
 *    updated by SGD with momentum.
 */
#ifndef EKYA_H_
#define EKYA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EKYA_OK = 0,
  EKYA_ERR_INVALID_ARG = 1, /* a pointer, size or option is out of range */
  EKYA_ERR_NOMEM = 2,       /* the workspace could not be allocated, or a fixed one is too small */
  EKYA_ERR_HIP = 3,         /* a HIP runtime call or kernel launch failed */
  EKYA_ERR_NONFINITE = 4,   /* a training loss became NaN or infinite */
  EKYA_ERR_UNSUPPORTED = 5  /* valid request this build does not implement */
} ekya_status;

typedef enum { EKYA_FP32 = 0, EKYA_BF16 = 1 } ekya_precision;

#define EKYA_MAX_EPOCHS 64
#define EKYA_MAX_HIDDEN 4096

typedef struct ekya_ctx ekya_ctx;

/* Retraining configuration (the paper's retraining configuration, section
 * 3.1: layers to retrain, data fraction, epochs, batch size; learning rate
 * and momentum of plain SGD). */
typedef struct {
  double subsample_frac; /* (0, 1]: round-half-up(frac * n_frames), at least 1, frames are used */
  int epochs;            /* 1 .. EKYA_MAX_EPOCHS */
  float lr;              /* > 0 */
  float momentum;        /* [0, 1) (0.9 in the configurations studied) */
  int batch;             /* >= 1; the last partial batch of an epoch is kept */
  uint64_t seed;         /* subset draw and epoch shuffles (SplitMix64 + Fisher-Yates) */
  int precision;         /* ekya_precision of frames and of the compute path */
} ekya_train_opts;

typedef struct {
  int n_train;                          /* frames in the training subset */
  int n_epochs;
  int n_steps;                          /* SGD steps taken */
  float heldout_acc_final;              /* held-out accuracy after the last epoch */
  float heldout_acc[EKYA_MAX_EPOCHS];   /* held-out accuracy after each epoch */
  float epoch_seconds[EKYA_MAX_EPOCHS]; /* GPU time of each epoch's training steps, from the
                                          epoch's first step to the end of its last (both the
                                          data- and the weight-gradient streams) */
  float eval_seconds[EKYA_MAX_EPOCHS];  /* GPU time of the held-out evaluation after each epoch
                                          (it runs on its own stream beside the next epoch's
                                          steps, so the two overlap) */
  float epoch_loss[EKYA_MAX_EPOCHS];    /* mean training loss over the epoch's steps */
  float prefix_seconds;                 /* GPU time of the frozen-prefix cache build */
  float* step_loss;                     /* host, optional: receives per-step losses */
  int step_loss_capacity;               /* entries available behind step_loss */
} ekya_retrain_result;

/* One micro-profiler candidate (section 4.3). */
typedef struct {
  int k_trainable;       /* 1 .. 6 */
  double subsample_frac; /* (0, 1] */
  int epochs;            /* 1 .. EKYA_MAX_EPOCHS */
  float lr;
  float momentum;
  int batch;
  uint64_t shuffle_seed; /* epoch-shuffle seed of this candidate */
} ekya_profile_cfg;

typedef struct {
  int status;                           /* ekya_status of this candidate */
  int n_train;
  float heldout_acc[EKYA_MAX_EPOCHS];   /* accuracy after each epoch */
  float epoch_seconds[EKYA_MAX_EPOCHS]; /* GPU time of each epoch's training steps (as in
                                          ekya_retrain_result) */
  float eval_seconds[EKYA_MAX_EPOCHS];  /* GPU time of the held-out evaluation after each epoch
                                          (on the candidate's own stream, after the steps) */
  float epoch_loss[EKYA_MAX_EPOCHS];    /* mean training loss over the epoch's steps */
  float heldout_acc_final;
} ekya_profile_result;

/* ------------------------------------------------------------ context */

/* Create a context on HIP device `hip_device` for a ResNet18 with
 * `n_classes` (1 .. 1024) outputs.  *out is set on success.
 *  workspace_bytes > 0: the context allocates one device arena of exactly
 *    that size here and never allocates device memory afterwards; a call
 *    whose buffers do not fit returns EKYA_ERR_NOMEM before queueing any GPU
 *    work (size it with ekya_*_workspace below).
 *  workspace_bytes == 0: the arena is sized by the calls themselves; a call
 *    that needs more than the arena holds waits (on the host) for the
 *    context's previous call to finish and replaces the arena before it
 *    queues any work -- releasing device memory may wait for the whole
 *    device, so concurrent work elsewhere on the GPU is delayed once.
 * EKYA_ERR_NOMEM if the arena cannot be allocated. */
ekya_status ekya_create(ekya_ctx** out, int hip_device, int n_classes, size_t workspace_bytes);
/* A context whose network has a hidden fully connected ReLU layer of
 * `hidden` neurons (0 .. EKYA_MAX_HIDDEN; 0 is ekya_create) between the pooled
 * features and the classifier: the number of neurons in the last layer, one
 * of the knobs of a retraining configuration (sections 3.2 and 6.1).  The
 * layer belongs to the classifier stage (trained whenever k_trainable >= 1).
 * Canonical weights then end with fc.0.weight [hidden][512], fc.0.bias
 * [hidden], fc.2.weight [n_classes][hidden], fc.2.bias [n_classes] (torch
 * nn.Sequential names) in place of fc.weight and fc.bias; their length is
 * ekya_weights_count_head(n_classes, hidden). */
ekya_status ekya_create_head(ekya_ctx** out, int hip_device, int n_classes, int hidden,
                             size_t workspace_bytes);
/* Release everything the context owns (synchronises its streams first). */
void ekya_destroy(ekya_ctx* ctx);
/* Length in floats of the canonical weight array for `n_classes`. */
size_t ekya_weights_count(int n_classes);
size_t ekya_weights_count_head(int n_classes, int hidden);
const char* ekya_status_str(ekya_status s);
/* Message of the last failure on this context ("" if none). */
const char* ekya_last_error(const ekya_ctx* ctx);

/* Workspace bytes (for ekya_create) that one call with these arguments
 * plans; host-only computations that need no GPU.  0 if an argument is
 * invalid (the matching call would return EKYA_ERR_INVALID_ARG).  The
 * arena is reused call after call, so a context serving several kinds of
 * call needs the largest of their sizes.  Inference needs the same
 * workspace for any number of frames. */
size_t ekya_retrain_workspace(int n_classes, int k_trainable, int n_frames, int H, int W,
                              int n_heldout, const ekya_train_opts* opts);
size_t ekya_profile_workspace(int n_classes, const ekya_profile_cfg* cfgs, int n_cfgs,
                              int n_frames, int H, int W, int n_heldout, int precision);
size_t ekya_infer_workspace(int n_classes, int resolution, int precision);
/* The same for a context made by ekya_create_head with `hidden` neurons. */
size_t ekya_retrain_workspace_head(int n_classes, int hidden, int k_trainable, int n_frames, int H,
                                   int W, int n_heldout, const ekya_train_opts* opts);
size_t ekya_profile_workspace_head(int n_classes, int hidden, const ekya_profile_cfg* cfgs,
                                   int n_cfgs, int n_frames, int H, int W, int n_heldout,
                                   int precision);
size_t ekya_infer_workspace_head(int n_classes, int hidden, int resolution, int precision);

/* ------------------------------------------------------------ retrain
 * Retrain the last k_trainable stages (sections 3.1 and 4.3).
 *  weights        device fp32, canonical layout, read and updated in place:
 *                 parameters and running statistics of trainable stages
 *                 change; frozen stages stay bitwise unchanged.
 *  frames, labels device, [n_frames, H, W, 3] and [n_frames] (the window).
 *  heldout_*      device, [n_heldout, H, W, 3] and [n_heldout]; accuracy on
 *                 them is measured after every epoch in eval mode.
 *  H, W           >= 32, same for both frame sets.
 *  opts           host; result host (step_loss optional).
 *  stream         caller's HIP stream; all work is ordered after prior work
 *                 on it.  The call returns after the results are on the host.
 * Momentum starts at zero on every call (each window's retraining is a new
 * job).  Returns EKYA_ERR_NONFINITE (with the epochs completed so far filled
 * in) if a training loss is not finite. */
ekya_status ekya_retrain(ekya_ctx* ctx, float* weights, int k_trainable, const void* frames,
                         const int32_t* labels, int n_frames, int H, int W,
                         const void* heldout_frames, const int32_t* heldout_labels, int n_heldout,
                         const ekya_train_opts* opts, ekya_retrain_result* result,
                         void* stream);

/* ------------------------------------------------------------ profile
 * Micro-profile n_cfgs candidates (section 4.3): each one retrains its last
 * k stages from the same `weights` (device fp32 canonical, read only) on the
 * first round-half-up(frac * n_frames) frames of one shared uniform draw
 * (seed `subsample_seed`; a smaller fraction's subset is a prefix of a larger
 * one's), for its epochs, and reports held-out accuracy and GPU time per
 * epoch.  Frozen-prefix caches are built once per distinct depth.  With
 * `concurrent` != 0 every candidate runs on its own HIP stream at the same
 * time (per-epoch times then include sharing the GPU); with 0 they run one
 * after another (per-epoch times are at 100% of the GPU, as the paper's
 * profiler measures them).  Results are bitwise identical in both modes.
 * Synchronous; results[i] (host) receives candidate i. */
ekya_status ekya_profile(ekya_ctx* ctx, const float* weights, const ekya_profile_cfg* cfgs,
                         int n_cfgs, const void* frames, const int32_t* labels, int n_frames,
                         int H, int W, const void* heldout_frames, const int32_t* heldout_labels,
                         int n_heldout, uint64_t subsample_seed, int precision, int concurrent,
                         ekya_profile_result* results);

/* ------------------------------------------------------------ infer
 * Classify n frames (device, [n, H, W, 3]) after resizing them bilinearly
 * (half-pixel centres, no antialiasing) to resolution x resolution (the
 * inference configuration's resolution, section 3.1); eval-mode BatchNorm.
 * labels_out: device int32 [n] (lowest class index wins ties).  weights:
 * device fp32 canonical, read only.  Asynchronous on `stream`: the caller
 * synchronises before reading labels_out.  Frame sampling (every k-th frame)
 * is the caller's choice of which frames to pass. */
ekya_status ekya_infer(ekya_ctx* ctx, const float* weights, const void* frames, int n, int H,
                       int W, int resolution, int precision, int32_t* labels_out, void* stream);

/* ------------------------------------------------------------ kernel timing
 * Per-kernel GPU time, the measurement the micro-profiler rests on (the
 * resource demand of a configuration is measured as GPU time, section 4.3),
 * broken down by GEMM kernel.  ekya_set_kernel_timing(ctx, 1) clears the
 * statistics and makes later ekya_retrain / ekya_infer calls on this context
 * bracket every convolution GEMM launch with two HIP events on the launch's
 * stream (0 turns it off; statistics are kept).  While timing is on, work
 * the library would otherwise overlap on a second stream (weight gradients)
 * runs on the job's stream, so each kernel is timed alone.  ekya_kernel_timing reads
 * entry `index` (0-based; waits for the recorded launches to finish): kernel
 * name into name (NUL-terminated, truncated to name_cap), launch count, summed
 * event time in ms, summed algorithmic flops (2*N*P*Q*K*R*S*C) and bytes
 * (input + weights + output).  Returns 0, or -1 past the last entry or on
 * invalid arguments. */
ekya_status ekya_set_kernel_timing(ekya_ctx* ctx, int enable);
int ekya_kernel_timing(ekya_ctx* ctx, int index, char* name, int name_cap, long long* launches,
                       double* total_ms, double* flops, double* bytes);

/* ------------------------------------------------------------ host helpers
 * The uniform training subset ekya_retrain draws (section 4.3, "Training data
 * sampling"): writes round-half-up(frac * n_frames) (>= 1) distinct frame
 * indices to idx_out (host) and returns that count, or -1 on invalid
 * arguments or if capacity is too small.  Pure host code; no GPU needed. */
int ekya_training_subset(int n_frames, double subsample_frac, uint64_t seed, int32_t* idx_out,
                         int capacity);
/* The order in which epoch `epoch` (0-based) visits the n training frames
 * (positions 0..n-1 of the subset).  Host code; returns 0 or -1. */
int ekya_epoch_order(int n, uint64_t seed, int epoch, int32_t* order_out);

#ifdef __cplusplus
}
#endif
#endif /* EKYA_H_ */
