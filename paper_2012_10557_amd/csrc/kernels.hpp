// Host-side launchers of every kernel of the library.  All pointers are device
// pointers; every call is asynchronous on `stream` and returns the launch status.
#pragma once

#include <string>
#include <vector>

#include "common.hpp"

namespace ekya {

// Opt-in timing of the GEMM launches: when a thread has a timer installed,
// every conv GEMM launch is bracketed by two events on its stream and logged
// with its algorithmic flops and bytes (read once the stream has finished).
struct LaunchRecord {
  std::string name;
  double flops, bytes;
  hipEvent_t e0, e1;
};
struct KernelTimer {
  std::vector<LaunchRecord> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t take();
};
void set_thread_timer(KernelTimer* t);
KernelTimer* thread_timer();

// The same for the memory-bound kernels: brackets the launches queued between
// construction and done() with two events on `stream` when the calling thread
// has a timer installed, logged with the launch's algorithmic HBM bytes.
class TimedLaunch {
 public:
  explicit TimedLaunch(hipStream_t s) : t_(thread_timer()), s_(s) {
    if (t_) {
      e0_ = t_->take();
      e1_ = t_->take();
      if (hipEventRecord(e0_, s_) != hipSuccess) t_ = nullptr;
    }
  }
  hipError_t done(hipError_t e, const char* name, double bytes) {
    if (t_ && e == hipSuccess) {
      e = hipEventRecord(e1_, s_);
      if (e == hipSuccess) t_->recs.push_back({name, 0.0, bytes, e0_, e1_});
    }
    return e;
  }

 private:
  KernelTimer* t_;
  hipStream_t s_;
  hipEvent_t e0_ = nullptr, e1_ = nullptr;
};

enum DType { DT_F32 = 0, DT_BF16 = 1 };
inline size_t dtype_size(int dt) { return dt == DT_F32 ? 4 : 2; }
inline int dtype_vec(int dt) { return dt == DT_F32 ? 4 : 8; }

// ------------------------------------------------------------- convolution
struct ConvGeom {
  int N, H, W, C;     // input NHWC; C is the stored (padded) channel count
  int K, R, S;        // output channels, kernel rows/cols
  int stride, pad;
  int P, Q;           // output spatial size
  int C0 = 0;         // real input channels (0: same as C); only used for cost accounting
};

// Epilogue of the forward conv: y = acc * scale[k] + shift[k] (+ res) (ReLU),
// any of scale/shift/res may be null (scale null = 1, shift null = 0).
struct ConvEpilogue {
  const float* scale = nullptr;
  const float* shift = nullptr;
  const void* res = nullptr;
  int relu = 0;
};

// BatchNorm chunk partials for the two-launch BatchNorm path, produced by a
// convolution on the bf16 direct-to-LDS path (empty forward epilogue, M
// within bn_fold_path): in the epilogue of an unsplit GEMM whose waves each
// cover 64 output pixels (chunks of 64 rows), or while a split GEMM's
// partials are reduced (chunks of 128 rows).  `done` reports whether they
// were; otherwise the caller computes them.  Forward: statistics of the output.
// Backward (bwd): of g = out * [ymask > 0] (no mask when null) against z and
// mean, as bn_backward's first pass.
struct BnStatsSink {
  float* part = nullptr;  // bn_partials_floats(M, C)
  bool bwd = false;
  const void* ymask = nullptr;
  const void* z = nullptr;
  const float* mean = nullptr;
  bool done = false;
  int rows = 0;  // rows per chunk of the partials when done (64 or 128)
};

// y[N,P,Q,K] = conv(x[N,H,W,C], w[K,R,S,C]) with the epilogue.  `ws` (fp32,
// ws_floats) holds split-reduction partials when the output has too few tiles
// (conv_split_workspace_floats tells how much; null or too small: no split).
hipError_t conv_fwd(int dt, const ConvGeom& g, const void* x, const void* w_krsc, void* y,
                    const ConvEpilogue& epi, float* ws, size_t ws_floats, hipStream_t stream,
                    BnStatsSink* sink = nullptr);
// The 7x7/2 stem reading [.][H][W][3] frames directly (image n at idx[n] when
// idx != null) in place of the padded input; g is the padded-input geometry
// (C = 8).  bf16 with Q <= 112 only (stem_frames_ok).
bool stem_frames_ok(int dt, const ConvGeom& g);
// The stem (epilogue as given, e.g. folded BatchNorm + ReLU) followed by the
// 3x3 / stride 2 / pad 1 max pool, in one kernel: y is [N][(P-1)/2+1][(Q-1)/2+1][64].
// x is the padded input, or with `raw` the 3-channel frames as in
// stem_fwd_frames.  bf16 with Q <= 112 only (stem_pool_ok).
bool stem_pool_ok(int dt, const ConvGeom& g);
hipError_t stem_pool_fwd(int dt, const ConvGeom& g, const void* x, bool raw, const int32_t* idx,
                         const void* w_krsc, void* y, const ConvEpilogue& epi,
                         hipStream_t stream);
hipError_t stem_fwd_frames(int dt, const ConvGeom& g, const void* frames, const int32_t* idx,
                           const void* w_krsc, void* y, const ConvEpilogue& epi,
                           hipStream_t stream);
// dx[N,H,W,C] = conv-transpose of dy[N,P,Q,K] with wT[C,R,S,K] (+ res[N,H,W,C]).
// Needs K a multiple of 64 (bf16) / 32 (fp32) and stride 1 or 2.
hipError_t conv_dgrad(int dt, const ConvGeom& g, const void* dy, const void* w_crsk, void* dx,
                      const void* res, float* ws, size_t ws_floats, hipStream_t stream,
                      BnStatsSink* sink = nullptr);
size_t conv_split_workspace_floats(int dt, const ConvGeom& g, bool dgrad);
// The bf16 data gradient of a 3x3 / stride-2 / pad-1 convolution g plus that
// of a 1x1 / stride-2 / pad-0 convolution gs on the same input (a projection
// shortcut; dy_sc its output gradient, wt_sc its weights [C][1][1][K2]) in
// one launch: dx = dgrad(g) + dgrad(gs), the shortcut's part folded into the
// reduction of the pixels (2 i, 2 j) it reaches.  No residual.
bool conv_dgrad_s2_shortcut_ok(int dt, const ConvGeom& g, const ConvGeom& gs);
hipError_t conv_dgrad_s2_shortcut(const ConvGeom& g, const void* dy, const void* wt,
                                  const ConvGeom& gs, const void* dy_sc, const void* wt_sc,
                                  void* dx, float* ws, size_t ws_floats, hipStream_t stream);
// Split count and partial-buffer size (floats) the weight gradient will use;
// g.C0 must be the real channel count later passed to conv_wgrad as C0 (the
// bf16 stem, 3 channels stored as 8, has its own kernel and scratch).
int conv_wgrad_splits(int dt, const ConvGeom& g);
size_t conv_wgrad_workspace_floats(int dt, const ConvGeom& g);
// dw[K,R,S,C0] (fp32, unpadded channel count C0 <= C) = sum over pixels of
// dy x im2col(x); deterministic split-K through `partials`.
hipError_t conv_wgrad(int dt, const ConvGeom& g, const void* x, const void* dy, float* partials,
                      float* dw, int C0, hipStream_t stream);
// The bf16 stem's weight gradient (as conv_wgrad with C0 = 3) whose output
// gradient is the stem's BatchNorm + ReLU + 3x3/2 max-pool backward, formed
// while it is staged: z the BatchNorm input [N][P][Q][64], dy_pool / arg the
// pooled gradient and window indices, mean and coef (bn_backward_pool_stats)
// its coefficients, gamma, invstd and beta the ReLU mask's.  The same values
// as bn_backward_pool followed by conv_wgrad, without dz in memory.
bool stem_wgrad_pool_ok(int dt, const ConvGeom& g);
hipError_t conv_wgrad_stem_pool(const ConvGeom& g, const void* x, const void* z,
                                const void* dy_pool, const uint8_t* arg, const float* mean,
                                const float* coef, const float* gamma, const float* invstd,
                                const float* beta, float* partials, float* dw, hipStream_t stream);
// The weight gradient left as fp32 split partials [splits][K][R][S][C] (one
// split included) for conv_weight_update: bf16 with C and K multiples of 64.
// conv_wgrad_partials_floats includes the scratch conv_weight_update needs
// after the partials.
bool conv_wgrad_partials_ok(int dt, const ConvGeom& g);
size_t conv_wgrad_partials_floats(int dt, const ConvGeom& g);
// shared: the launch runs beside other work on another stream (the
// all-taps kernel then takes about 96 blocks, under half the CUs).
hipError_t conv_wgrad_partials(int dt, const ConvGeom& g, const void* x, const void* dy,
                               float* partials, int* splits, hipStream_t stream,
                               bool shared = false);

// ---------------------------------------------------------------- BatchNorm
// Per-channel statistics of z[M, C] (NHWC rows).  Writes mean and 1/sqrt(var+eps)
// (biased variance) and, when rm/rv are non-null, updates running statistics
// with momentum 0.1 and the unbiased variance.  Also writes scale = gamma*invstd,
// shift = beta - mean*scale.  `partials` needs bn_partials_floats(M, C).
size_t bn_partials_floats(long long M, int C);
// True when BatchNorm over [M, C] takes the two-launch path (partials per
// 128-row chunk and 64 channels, reduced inside the apply kernels).
bool bn_fold_path(long long M, int C);
// Sum of split partials [splits][M][C] in split order (+ res) into out (dt),
// with the chunk partials the sink asks for (bn_fold_path(M, C) must hold).
hipError_t split_reduce_bn(int dt, const float* part, int splits, long long M, int C,
                           const void* res, void* out, const BnStatsSink& sink,
                           hipStream_t stream);
hipError_t bn_train_stats(int dt, const void* z, long long M, int C, const float* gamma,
                          const float* beta, float* rm, float* rv, float* mean, float* invstd,
                          float* scale, float* shift, float* partials, hipStream_t stream);
// bn_train_stats followed by bn_apply: y = relu?((z - mean)*scale + beta + res).
// Two launches when M is at most 64 chunks of 128 rows and C a multiple of 64.
// ready_rows > 0: `partials` already holds the chunk partials of z in chunks
// of that many rows (64 or 128, from a BnStatsSink).
hipError_t bn_train_forward(int dt, const void* z, long long M, int C, const float* gamma,
                            const float* beta, float* rm, float* rv, float* mean, float* invstd,
                            float* scale, float* shift, const void* res, int relu, void* y,
                            float* partials, hipStream_t stream, int ready_rows = 0);
// y = (z - mean)*scale + beta (+ res) (ReLU), elementwise over [M, C].
hipError_t bn_apply(int dt, const void* z, long long M, int C, const float* mean,
                    const float* scale, const float* beta, const void* res, int relu, void* y,
                    hipStream_t stream);
// Eval-mode fold for `n` BatchNorm layers given by tables of parameter offsets
// into `params`: scale = gamma / sqrt(rv + eps), shift = beta - rm * scale,
// written at out_off[i] (scale) and out_off[i] + C[i] (shift) of `out`.
hipError_t bn_fold(const float* params, const long long* tab, int n, float* out,
                   hipStream_t stream);
// Backward of train-mode BN (with the ReLU mask y > 0 when y != null):
// g = dy * [y > 0]; dgamma = sum g*xhat; dbeta = sum g;
// dz = gamma*invstd*(g - dbeta/M - xhat*dgamma/M).  Writes dgamma/dbeta and
// dz; when g_out != null also writes g.
// ready_rows: as for bn_train_forward.  relu_beta (with y null): the output
// was y = relu(BN(z)) with no residual and this beta; the mask is recomputed
// from z, mean, gamma * invstd and beta exactly as the forward pass rounded
// y, so y need not be read.
hipError_t bn_backward(int dt, const void* dy, const void* y, const void* z, long long M, int C,
                       const float* gamma, const float* mean, const float* invstd, float* dgamma,
                       float* dbeta, void* dz, void* g_out, float* partials, hipStream_t stream,
                       int ready_rows = 0, const float* relu_beta = nullptr);

// Backward of a train-mode BatchNorm + ReLU (no residual) whose output went
// only into the 3x3 / stride 2 / pad 1 max pool: dz [N, H, W, C] from the
// pooled gradient dy_pool and window indices arg ([N, P, Q, C]), equal to
// maxpool_bwd followed by bn_backward with the mask recomputed from z (beta:
// the BatchNorm's shift), without the full-size gradient in memory;
// `partials`: bn_partials_floats(N * H * W, C).
// bn_backward_pool_ok: the shapes it takes (64 channels, width W <= 128).
bool bn_backward_pool_ok(int C, int H, int W);
hipError_t bn_backward_pool(int dt, const void* dy_pool, const uint8_t* arg, const void* z, int N,
                            int H, int W, int C, const float* gamma, const float* beta,
                            const float* mean, const float* invstd, float* dgamma, float* dbeta,
                            void* dz, float* partials, hipStream_t stream);
// Its statistics pass alone: dgamma, dbeta and the input-gradient
// coefficients dz = coef[c] * g + coef[C + c] + coef[2 C + c] * (z - mean),
// *coef pointing into `partials`, for a consumer that forms dz itself
// (conv_wgrad_stem_pool).
hipError_t bn_backward_pool_stats(int dt, const void* dy_pool, const uint8_t* arg, const void* z,
                                  int N, int H, int W, int C, const float* gamma, const float* beta,
                                  const float* mean, const float* invstd, float* dgamma,
                                  float* dbeta, float* partials, const float** coef,
                                  hipStream_t stream);

// ------------------------------------------------------------------ pooling
// Train-mode BatchNorm statistics of z [N, H, W, C] (as bn_train_stats),
// then the 3x3 / stride 2 / pad 1 max pool of relu(BN(z)) computed on load:
// y and arg as maxpool_fwd would give for the stored BatchNorm + ReLU output,
// which is never written.  `partials`: bn_partials_floats(N * H * W, C).
hipError_t bn_relu_maxpool_train(int dt, const void* z, int N, int H, int W, int C,
                                 const float* gamma, const float* beta, float* rm, float* rv,
                                 float* mean, float* invstd, float* scale, float* shift,
                                 float* partials, void* y, uint8_t* arg, hipStream_t stream);
hipError_t maxpool_fwd(int dt, const void* x, int N, int H, int W, int C, void* y, uint8_t* arg,
                       hipStream_t stream);
hipError_t maxpool_bwd(int dt, const void* dy, const uint8_t* arg, int N, int H, int W, int C,
                       void* dx, hipStream_t stream);
// f[N, C] (fp32) = mean over H*W of x.
hipError_t avgpool_fwd(int dt, const void* x, int N, int HW, int C, float* f, hipStream_t stream);
hipError_t avgpool_bwd(int dt, const float* df, int N, int HW, int C, void* dx,
                       hipStream_t stream);

// --------------------------------------------------------------- classifier
// z[N, J] = f[N, I] W[J, I]^T + b
hipError_t fc_fwd(const float* f, const float* Wt, const float* b, int N, int I, int J, float* z,
                  hipStream_t stream);
// Softmax cross-entropy over rows of z[N, J] with labels (selected through
// `idx` when non-null): dz = (softmax - onehot)/N, out[0] = mean loss,
// out[1] = correct count (as float), out[2] = non-finite flag.
hipError_t softmax_ce(const float* z, const int32_t* labels, const int32_t* idx, int N, int J,
                      float* dz, float* out, hipStream_t stream);
// dW[J, I] = dz^T f, db = column sums of dz, df = dz W (df may be null).
hipError_t fc_bwd(const float* dz, const float* f, const float* Wt, int N, int I, int J, float* dW,
                  float* db, float* df, hipStream_t stream);
// Fused classifier head.  Forward: pooled[N, I] (fp32) = mean over HW pixels
// of x[N, HW, I] (x null: features f are used and pooled is not written),
// z = pooled W^T + b.  Backward (J <= 16, I <= 512; head_backward_fused):
// softmax cross-entropy of z with labels (through idx when non-null) as in
// softmax_ce (out[0..2]), dW = dz^T f, db = column sums of dz and, when dout
// is non-null, dout[N, HW, I] = (dz W) / HW.
hipError_t head_forward(int dt, const void* x, int HW, const float* f, const float* W,
                        const float* b, int N, int I, int J, float* pooled, float* z,
                        hipStream_t stream);
// bn (with dout): the BatchNorm whose output (ReLU mask ymask, input z,
// batch mean) dout is the gradient of; when the fused path can, the launch
// also leaves that BatchNorm's backward chunk partials in bn->part and sets
// bn->rows (64: pass it to bn_backward as ready_rows), else rows = 0.
struct HeadBnSink {
  const void* ymask = nullptr;
  const void* z = nullptr;
  const float* mean = nullptr;
  float* part = nullptr;
  int rows = 0;
};
bool head_backward_fused(int J, int I);
hipError_t head_backward(int dt, const float* z, const int32_t* labels, const int32_t* idx, int N,
                         int J, const float* f, const float* W, int I, float* dW, float* db,
                         void* dout, int HW, float* out, hipStream_t stream,
                         HeadBnSink* bn = nullptr);
// Count of rows whose argmax matches the label, accumulated into *count.
hipError_t count_correct(const float* z, const int32_t* labels, int N, int J, int32_t* count,
                         hipStream_t stream);
hipError_t argmax_rows(const float* z, int N, int J, int32_t* out, hipStream_t stream);
// y = max(x, 0) (mask null) or y = x where mask > 0, else 0 (the ReLU
// backward through the ReLU's output), over n fp32 values; y may be x.
hipError_t relu_f32(float* y, const float* x, const float* mask, long long n, hipStream_t stream);

// -------------------------------------------------------------- optimiser
// v = mu v + g; w = w - lr v over n floats.
hipError_t sgd_momentum(float* w, float* v, const float* g, long long n, float lr, float mu,
                        hipStream_t stream);
// The same over n (offset, length) rows of tab; max_len bounds the lengths.
hipError_t sgd_momentum_ranges(float* w, float* v, const float* g, const long long* tab, int n,
                               long long max_len, float lr, float mu, hipStream_t stream);
// One convolution's momentum step from its weight-gradient split partials
// (summed in split order; more than 16 splits are first added in groups of
// 16, in order, into conv_update_groups(splits) scratch slices right after
// the partials, which the buffer must hold): v = mu v + g, w = w - lr v on
// the fp32 [K][RS][C] master, then its [K][RS][C] and [C][RS][K]
// low-precision copies.
int conv_update_groups(int splits);
// out[g][i] = sum of part[s][i] over the splits of group g (16 consecutive
// splits, in order), g < conv_update_groups(splits); n a multiple of 4.
hipError_t split_group_sum(const float* part, int splits, long long n, float* out,
                           hipStream_t stream);
hipError_t conv_weight_update(int dt, const float* part, int splits, int K, int RS, int C,
                              float* w, float* v, float lr, float mu, void* krsc, void* crsk,
                              hipStream_t stream);

// ---------------------------------------------------------- data movement
// dst row i = src row idx[i] (idx null: row i), rows of `row_bytes` (multiple of 16).
hipError_t gather_rows(const void* src, const int32_t* idx, int n, long long row_bytes, void* dst,
                       hipStream_t stream);
// Frames [n, H, W, 3] (row idx[i] when idx != null) -> [n, H, W, Cp] with
// zero channels 3..Cp-1.
hipError_t frames_to_padded(int dt, const void* frames, const int32_t* idx, int n, int H, int W,
                            int Cp, void* dst, hipStream_t stream);
// Bilinear resize (half-pixel centres, clamped) of frames [n, H, W, 3] to
// [n, r, r, Cp] with zero padding channels.
hipError_t resize_to_padded(int dt, const void* frames, int n, int H, int W, int r, int Cp,
                            void* dst, hipStream_t stream);
// Element-wise fp32 -> dt copy.
hipError_t cast_from_f32(int dt, const float* src, long long n, void* dst, hipStream_t stream);

// ------------------------------------------------------ weight (re)packing
// Table row per conv (all entries long long): src_off (fp32, [K][R][S][C0]),
// K, R, S, C0, Cp, krsc_off (elements of dt), crsk_off (elements, -1 = skip).
hipError_t pack_conv_weights(int dt, const float* master, const long long* tab, int n,
                             void* shadow, hipStream_t stream);
// Table row per tensor: off, K, C, R, S (conv) or off, n, 0, 0, 0 (other):
// to_internal = 1 permutes [K][C][R][S] -> [K][R][S][C], 0 the inverse.
hipError_t permute_weights(const float* src, float* dst, const long long* tab, int n,
                           long long total, int to_internal, hipStream_t stream);

// ------------------------------------------------------------- diagnostics
// n one-wavefront workgroups; workgroup i writes the compute unit it ran on,
// (xcd << 10) | (shader array << 8) | (shader engine << 4) | cu, to out[i].
hipError_t cu_ids(int n, uint32_t* out, hipStream_t stream);

}  // namespace ekya
