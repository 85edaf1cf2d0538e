/*
 * ekya_joint.h - running inference and retraining side by side on one GPU.
 *
 * Two mechanisms of the paper's system, built for one MI355X:
 *
 *  1. GPU shares (section 4.1: every inference and retraining job of a window
 *     gets a share of a GPU, in multiples of the quantum Delta, 0.1 in the
 *     evaluation; section 5, "Dynamic reallocation of resources": the shares
 *     are enforced by a GPU partitioning layer).  Here a share is a set of
 *     compute units (CUs): a HIP stream whose kernels run only on those CUs,
 *     and a context whose own streams do the same.
 *
 *  2. Model checkpointing and reloading (section 5): a model checkpointed
 *     during retraining is loaded into the running inference job, which keeps
 *     serving while the new weights are loaded.  Here an ekya_model holds
 *     prepared inference weights in two slots; a load fills the slot no new
 *     inference call will take and then publishes it.
 *
 * Conventions are those of ekya.h (device / host pointers, validation before
 * any GPU work, ekya_status results).
 */
#ifndef EKYA_JOINT_H_
#define EKYA_JOINT_H_

#include "ekya.h"

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ CU shares
 * A CU range [cu_begin, cu_begin + cu_share) is given in fractions of the
 * device (0 <= cu_begin < 1, 0 < cu_share, cu_begin + cu_share <= 1).  It is
 * counted in groups of one CU on every XCD (accelerator complex die; MI355X:
 * 8 XCDs of 4 shader engines of 8 CUs, so 32 groups): groups
 * round(cu_begin * R) .. round((cu_begin + cu_share) * R) - 1 of the
 * R = CUs / XCDs groups, at least one.  The workgroups of a kernel, which
 * the device hands to its XCDs in turn, so find the same number of CUs on
 * every XCD, and a run of groups spreads over the shader engines of each XCD
 * as evenly as whole groups allow.  Disjoint ranges select disjoint CUs.
 *
 * Mask layout: the amdgpu driver deals mask bits to the XCDs first, then to
 * the shader engines of an XCD, then to the CUs of an engine (bit b: CU
 * b / (X S) of engine (b / X) mod S on XCD b mod X, for X XCDs of S
 * engines).  Group g = k S + s takes CU k of engine s on every XCD; when the
 * CUs per engine equal the XCDs (MI355X), XCD j gets CU (j + s + k) mod X of
 * engine s instead, which places the group's bits in X different blocks of
 * R bits, so that a driver numbering the bits XCD by XCD would also give
 * every XCD one CU per group.  Otherwise group g puts XCD j on bit
 * j R + (g + j) mod R, which is one CU per XCD under either numbering.
 *
 * ekya_partition_mask writes that mask (host only, no GPU needed) for a
 * device with n_cu CUs on n_xcd XCDs of n_se shader engines into
 * mask_out[words] (bit i of word i / 32 = mask bit i) and returns the number
 * of CUs selected, or -1 on invalid arguments (n_cu not a multiple of n_xcd,
 * words < ceil(n_cu / 32), an empty or out-of-range selection). */
int ekya_partition_mask(int n_cu, int n_xcd, int n_se, double cu_begin, double cu_share,
                        uint32_t* mask_out, int words);

/* A new HIP stream on hip_device whose kernels run only on the CUs of the
 * range (hipExtStreamCreateWithCUMask; such a stream synchronises with the
 * legacy default stream like a stream created without flags).  *stream_out
 * receives the hipStream_t; release it with ekya_stream_destroy. */
ekya_status ekya_stream_create(int hip_device, double cu_begin, double cu_share,
                               void** stream_out);
ekya_status ekya_stream_destroy(void* stream);
/* The number of CUs a stream's kernels may use (as the runtime reports the
 * stream's CU mask); -1 on error. */
int ekya_stream_cu_count(void* stream);

/* Restrict the streams the context creates for itself (the retraining job's
 * weight-gradient and held-out evaluation streams, the profiler's
 * per-candidate streams) to a CU range; (0, 1) lifts the restriction.  Waits
 * for the context's queued work, then replaces its streams.  The caller's
 * `stream` arguments are the caller's: give them the same range with
 * ekya_stream_create. */
ekya_status ekya_set_cu_partition(ekya_ctx* ctx, double cu_begin, double cu_share);

/* Diagnostic: n_workgroups workgroups of one wavefront each, on `stream`,
 * each write to ids_out[i] (device uint32) the compute unit it ran on:
 * (xcd << 10) | (shader array << 8) | (shader engine << 4) | cu, read from
 * the hardware id registers.  Asynchronous.  n_workgroups in [1, 2^20]. */
ekya_status ekya_cu_ids(int n_workgroups, uint32_t* ids_out, void* stream);

/* ------------------------------------------------------------ hot reload */
typedef struct ekya_model ekya_model;

/* A prepared inference model for one device, class count and precision
 * (EKYA_FP32 / EKYA_BF16): two slots of internal-layout fp32 weights,
 * eval-mode BatchNorm folded to a per-channel scale and shift, and the
 * low-precision convolution weights the inference kernels read.  Allocates
 * its device memory (two slots, about 12 * 11.2 M bytes in bf16) here, none
 * later.  Empty until the first load. */
ekya_status ekya_model_create(ekya_model** out, int hip_device, int n_classes, int precision);
/* The same for a network with a hidden classifier layer (ekya_create_head). */
ekya_status ekya_model_create_head(ekya_model** out, int hip_device, int n_classes, int hidden,
                                   int precision);
/* Waits for the model's queued work, then releases it.  A context that
 * checkpoints into it must stop first (ekya_set_checkpoint(ctx, NULL, 0)). */
void ekya_model_destroy(ekya_model* m);

/* Load canonical fp32 weights (device, ekya_weights_count floats, read only)
 * into the slot that is not published, on `stream`, and publish it.  The
 * load first waits, on `stream`, for every inference call still reading that
 * slot (calls that took it before the previous load).  Inference calls that
 * start after this returns use the new weights once the load has run on the
 * GPU: their stream waits for it, the host never blocks.  Calls already
 * started keep their slot.  version_out (host, optional) receives the
 * version number of the published weights (1, 2, ... per model).  Safe to
 * call from one thread while another calls ekya_infer_model. */
ekya_status ekya_model_load(ekya_model* m, const float* weights, void* stream,
                            uint64_t* version_out);

/* Write the published weights back in canonical layout (device fp32,
 * ekya_weights_count floats) on `stream`; bitwise equal to the weights the
 * publishing load or checkpoint read.  EKYA_ERR_INVALID_ARG if nothing has
 * been published. */
ekya_status ekya_model_export(ekya_model* m, float* weights_out, void* stream,
                              uint64_t* version_out);

/* Version of the published weights (0: none). */
uint64_t ekya_model_version(ekya_model* m);

/* ekya_infer with the model's published weights: the call takes the
 * published slot when it starts and reports its version in version_out
 * (host, optional).  Labels equal bitwise those of ekya_infer with the
 * canonical weights that were published.  Asynchronous on `stream`.  The
 * model's device, class count and hidden layer must be the context's, its
 * precision the frames'. */
ekya_status ekya_infer_model(ekya_ctx* ctx, ekya_model* m, const void* frames, int n, int H, int W,
                             int resolution, int32_t* labels_out, void* stream,
                             uint64_t* version_out);

/* Batched inference over several video streams, each with its own model
 * (every stream's model is retrained on its own window, sections 3.1 and
 * 4.1): frames (device, [sum counts, H, W, 3]) hold counts[i] (host, >= 0)
 * consecutive frames of stream i, classified with models[i]'s published
 * weights into labels_out (device int32, same order).  The streams' groups
 * run on up to 4 streams of the context at once (forked from `stream` and
 * joined back into it), each with its own buffers; each group takes its
 * model's slot when the call starts and versions_out[i] (host, optional)
 * receives its version.  Every model must have published weights and match
 * the context (device, classes, hidden layer); all share one precision,
 * the frames'.  Labels equal bitwise those of ekya_infer_model per stream.
 * Asynchronous on `stream`. */
ekya_status ekya_infer_models(ekya_ctx* ctx, ekya_model* const* models, int n_models,
                              const void* frames, const int* counts, int H, int W, int resolution,
                              int32_t* labels_out, uint64_t* versions_out, void* stream);
/* Workspace bytes of ekya_infer_models with n_models models (host only). */
size_t ekya_infer_models_workspace(int n_classes, int hidden, int resolution, int precision,
                                   int n_models);

/* Checkpointing during retraining: later ekya_retrain calls on ctx publish
 * the weights being trained into m, as ekya_model_load would, on the
 * retraining stream after every `every_epochs` epochs (and after the last
 * epoch), while the job continues.  The retraining precision must be the
 * model's.  m = NULL stops it. */
ekya_status ekya_set_checkpoint(ekya_ctx* ctx, ekya_model* m, int every_epochs);

#ifdef __cplusplus
}
#endif
#endif /* EKYA_JOINT_H_ */
