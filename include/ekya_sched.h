/*
 * ekya_sched.h - host-side calls of the scheduling layer that consumes the
 * micro-profiler's output: accuracy-curve extrapolation (section 4.3,
 * micro-profiling: per-epoch accuracies of short low-fraction runs fitted to
 * a training-progress curve by non-negative least squares, then evaluated at
 * a full retraining) and the thief scheduler (section 4.2, Algorithms 1 and
 * 2: GPU shares and configurations of every stream's inference and
 * retraining jobs for a retraining window).  These run on the CPU, need no
 * GPU and no context, and are deterministic.  Pointers are host pointers
 * owned by the caller; invalid arguments return EKYA_ERR_INVALID_ARG.
 */
#ifndef EKYA_SCHED_H_
#define EKYA_SCHED_H_

#include "ekya.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Non-negative least squares, min ||A x - b||_2 subject to x >= 0, by
 * Lawson and Hanson's active-set method.  A: row-major m x n (1 <= m, n <=
 * 4096, m * n <= 2^22); b: m; x: n (out); rnorm: ||A x - b|| (out, may be
 * null).  EKYA_ERR_UNSUPPORTED if a least-squares subproblem is singular. */
ekya_status ekya_nnls(const double* A, int m, int n, const double* b, double* x, double* rnorm);

/* Training-progress curve of held-out error after x passes over the window's
 * data (x = epochs x fraction of the window trained on):
 * error(x) = 1 / (b0 x + b1) + b2 with b0, b1, b2 >= 0, accuracy = 1 - error
 * (clamped to [0, 1]).  rss: squared error of the fit at its points. */
typedef struct {
  double b0, b1, b2, rss;
} ekya_curve;

/* Fit the curve to n >= 1 points (x[i] > 0, acc[i] in [0, 1]): for each b2
 * below every measured error, 1 / (error - b2) = b0 x + b1 is solved for
 * (b0, b1) >= 0 by NNLS; b2 is chosen on a 64-point grid over [0, min error)
 * refined by golden-section search, minimising the squared error in
 * accuracy.  A point of accuracy 1 forces b2 = 0. */
ekya_status ekya_fit_accuracy_curve(const double* x, const double* acc, int n, ekya_curve* out);
/* Accuracy the curve predicts after x passes (x >= 0). */
double ekya_curve_accuracy(const ekya_curve* c, double x);

/* From one micro-profiler candidate (its configuration and result from
 * ekya_profile over a window of n_frames frames): fit its per-epoch held-out
 * accuracies at x = (e + 1) * n_train / n_frames, and extrapolate to a
 * retraining of epochs_target epochs over the whole window -- accuracy
 * curve(epochs_target) and GPU seconds at the full GPU = the candidate's mean
 * epoch time x (SGD steps of a full epoch / of the candidate's epoch) x
 * epochs_target (per-epoch cost is deterministic).  Outputs may be null. */
ekya_status ekya_extrapolate(const ekya_profile_cfg* cfg, const ekya_profile_result* res,
                             int n_frames, int epochs_target, ekya_curve* curve, double* acc_out,
                             double* gpu_seconds_out);

/* Thief scheduler inputs.  An inference configuration needs a GPU share
 * `cost` (> 0) to keep up with its live stream and reaches accuracy
 * model_accuracy x factor; on a share below its cost it analyses only
 * share / cost of the frames.  A retraining configuration produces a model
 * of accuracy acc_after and takes gpu_seconds on a whole GPU (from
 * ekya_extrapolate). */
typedef struct {
  double cost, factor;
} ekya_infer_cfg;
typedef struct {
  double acc_after, gpu_seconds;
} ekya_train_cfg;
typedef struct {
  double acc_now;                /* accuracy of the stream's current model */
  const ekya_infer_cfg* infer;   /* n_infer >= 1 configurations */
  int n_infer;
  const ekya_train_cfg* train;   /* n_train >= 0 configurations */
  int n_train;
} ekya_video;

/* Outputs, arrays owned by the caller: alloc[2 n_videos] (GPU share of
 * stream v's inference job at 2v, retraining job at 2v + 1, multiples of
 * delta summing to n_gpus), infer_choice[n_videos], train_choice[n_videos]
 * (-1: no retraining), video_accuracy[n_videos] (each stream's estimated
 * mean inference accuracy over the window); accuracy: their mean. */
typedef struct {
  double* alloc;
  int* infer_choice;
  int* train_choice;
  double* video_accuracy;
  double accuracy;
} ekya_schedule;

/* Algorithm 1 over n_videos streams on n_gpus GPUs in quanta of delta
 * (n_gpus / delta a whole number of quanta, at most 4096): start from the
 * fair split of the quanta over the 2 n_videos jobs; every job in turn
 * steals one quantum at a time from every other job while the mean window
 * accuracy (PickConfigs, Algorithm 2, with EstimateAccuracy: the old model
 * serves until the retraining -- gpu_seconds / share, configurations longer
 * than window_s skipped -- finishes, the new one for the rest of the window;
 * inference configurations below accuracy a_min are not picked while
 * another keeps up) strictly improves. */
ekya_status ekya_thief_schedule(const ekya_video* videos, int n_videos, double n_gpus, double delta,
                                double window_s, double a_min, ekya_schedule* out);

#ifdef __cplusplus
}
#endif
#endif /* EKYA_SCHED_H_ */
