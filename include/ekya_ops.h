/*
 * ekya_ops.h - op-level entry points of the library's kernels.
 *
 * These expose, one at a time, the layer operations the retraining step is
 * built from (the layers of the ResNet18 edge classifier of section 6.1 and
 * the PyTorch training the paper runs, section 5), so that each kernel can be
 * compared with an independent implementation.  They are synchronous: each
 * call enqueues on `stream`, waits for it, and frees its temporaries.
 *
 * Common rules: every tensor pointer is a device pointer owned by the caller;
 * activations are NHWC with element type per `precision` (EKYA_FP32 float,
 * EKYA_BF16 bfloat16); weights and per-channel vectors are fp32.  Channel
 * counts must be multiples of 8 (bf16) or 4 (fp32), except an input channel
 * count of 3 (an image), which is zero-padded internally.  Invalid sizes
 * return EKYA_ERR_INVALID_ARG before any GPU work; HIP failures return
 * EKYA_ERR_HIP.
 */
#ifndef EKYA_OPS_H_
#define EKYA_OPS_H_

#include "ekya.h"

#ifdef __cplusplus
extern "C" {
#endif

/* y[N,P,Q,K] = sum_{c,r,s} x[N, stride*p + r - pad, stride*q + s - pad, c] * w[K][C][R][S]
 * (cross-correlation with zero padding), P = (H + 2 pad - R)/stride + 1. */
ekya_status ekya_op_conv2d(int precision, const void* x, int N, int H, int W, int C,
                           const float* w, int K, int R, int S, int stride, int pad, void* y,
                           void* stream);
/* dx[N,H,W,C]: gradient of ekya_op_conv2d with respect to x for dy[N,P,Q,K]. */
ekya_status ekya_op_conv2d_dgrad(int precision, const void* dy, const float* w, int N, int H,
                                 int W, int C, int K, int R, int S, int stride, int pad, void* dx,
                                 void* stream);
/* dw[K][C][R][S] (fp32): gradient of ekya_op_conv2d with respect to w. */
ekya_status ekya_op_conv2d_wgrad(int precision, const void* x, const void* dy, int N, int H,
                                 int W, int C, int K, int R, int S, int stride, int pad,
                                 float* dw, void* stream);
/* Train-mode BatchNorm over z[M, C] (M = N*H*W rows): y = gamma*(z-mean)*invstd
 * + beta (then ReLU if relu), biased batch variance, eps 1e-5; running
 * statistics (optional, may be null) updated with momentum 0.1 and the
 * unbiased variance.  mean_out/invstd_out: [C] fp32. */
ekya_status ekya_op_batchnorm_train(int precision, const void* z, long long M, int C,
                                    const float* gamma, const float* beta, float* running_mean,
                                    float* running_var, int relu, void* y, float* mean_out,
                                    float* invstd_out, void* stream);
/* ekya_op_batchnorm_train for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): same arguments, kernels and results (bitwise), but it calls no
 * hipMalloc / hipFree and does not synchronise -- the work is queued on
 * `stream` and the caller synchronises.  Its scratch (partial sums, scale and
 * shift) is one static device array per GPU of 512*2*2048 + 5*2048 floats
 * (about 8.4 MB), enough for every M and C <= 2048; a request that would
 * need more returns EKYA_ERR_INVALID_ARG.  The first call on a device looks
 * up the array's address (make it outside graph capture).  Every call on one
 * GPU shares that array, so calls that overlap on one GPU (different
 * streams without ordering between them) race; nothing in it needs to start
 * at zero. */
ekya_status ekya_op_batchnorm_train_noalloc(int precision, const void* z, long long M, int C,
                                            const float* gamma, const float* beta,
                                            float* running_mean, float* running_var, int relu,
                                            void* y, float* mean_out, float* invstd_out,
                                            void* stream);
/* Backward of ekya_op_batchnorm_train: g = dy * [y_relu > 0] (no mask when
 * y_relu is null); dbeta = sum g, dgamma = sum g*xhat,
 * dz = gamma*invstd/M*(M*g - dbeta - xhat*dgamma). */
ekya_status ekya_op_batchnorm_backward(int precision, const void* dy, const void* y_relu,
                                       const void* z, long long M, int C, const float* gamma,
                                       const float* mean, const float* invstd, void* dz,
                                       float* dgamma, float* dbeta, void* stream);
/* 3x3 stride-2 pad-1 max pooling (padding never wins); arg[N,P,Q,C] (uint8)
 * is the row-major window index of the first maximal element. */
ekya_status ekya_op_maxpool(int precision, const void* x, int N, int H, int W, int C, void* y,
                            uint8_t* arg, void* stream);
ekya_status ekya_op_maxpool_backward(int precision, const void* dy, const uint8_t* arg, int N,
                                     int H, int W, int C, void* dx, void* stream);
/* f[N, C] (fp32) = mean of x over H*W; and its backward dx = df / (H*W). */
ekya_status ekya_op_avgpool(int precision, const void* x, int N, int H, int W, int C, float* f,
                            void* stream);
ekya_status ekya_op_avgpool_backward(int precision, const float* df, int N, int H, int W, int C,
                                     void* dx, void* stream);
/* Classifier: z[N,J] = f[N,I] W[J,I]^T + b, and its backward (fp32). */
ekya_status ekya_op_linear(const float* f, const float* Wt, const float* b, int N, int I, int J,
                           float* z, void* stream);
ekya_status ekya_op_linear_backward(const float* dz, const float* f, const float* Wt, int N,
                                    int I, int J, float* dW, float* db, float* df, void* stream);
/* Mean softmax cross-entropy of z[N,J] against labels[N]: dz = (softmax -
 * onehot)/N; out[0] = mean loss, out[1] = correct count, out[2] = non-finite
 * flag (device fp32 [3]). */
ekya_status ekya_op_softmax_ce(const float* z, const int32_t* labels, int N, int J, float* dz,
                               float* out, void* stream);
/* SGD with momentum over n floats: v = mu v + g; w = w - lr v. */
ekya_status ekya_op_sgd(float* w, float* v, const float* g, long long n, float lr, float mu,
                        void* stream);
/* Bilinear resize (half-pixel centres, clamped at 0, no antialiasing) of
 * frames [n,H,W,3] to [n,r,r,3]. */
ekya_status ekya_op_resize(int precision, const void* frames, int n, int H, int W, int r,
                           void* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* EKYA_OPS_H_ */
