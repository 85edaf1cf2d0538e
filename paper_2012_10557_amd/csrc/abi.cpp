// extern "C" entry points: argument validation (before any GPU work), status
// codes, and the op-level entry points used for kernel-by-kernel parity.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <iterator>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/ekya.h"
#include "../../include/ekya_joint.h"
#include "../../include/ekya_ops.h"
#include "../../include/ekya_sched.h"
#include "curve.hpp"
#include "rng.hpp"
#include "runtime.hpp"

struct ekya_ctx {
  ekya::Ctx c;
};

struct ekya_model {
  ekya::Model m;
};

namespace {

thread_local std::string g_noctx_err;

ekya_status fail(ekya_ctx* ctx, ekya_status s, const std::string& msg) {
  if (ctx) ctx->c.err = msg; else g_noctx_err = msg;
  return s;
}

bool valid_precision(int p) { return p == EKYA_FP32 || p == EKYA_BF16; }

ekya_status check_frames(ekya_ctx* ctx, int H, int W) {
  if (H < 32 || W < 32 || H > 4096 || W > 4096)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "frame height and width must be in [32, 4096]");
  return EKYA_OK;
}

ekya_status hip_status(hipError_t e) {
  if (e == hipSuccess) return EKYA_OK;
  g_noctx_err = std::string("HIP error: ") + hipGetErrorString(e);
  return e == hipErrorOutOfMemory ? EKYA_ERR_NOMEM : EKYA_ERR_HIP;
}

}  // namespace

extern "C" {

size_t ekya_weights_count_head(int n_classes, int hidden) {
  if (n_classes < 1 || n_classes > 1024 || hidden < 0 || hidden > EKYA_MAX_HIDDEN) return 0;
  return (size_t)ekya::Net::build(n_classes, 0, hidden).total;
}

size_t ekya_weights_count(int n_classes) { return ekya_weights_count_head(n_classes, 0); }

const char* ekya_status_str(ekya_status s) {
  switch (s) {
    case EKYA_OK: return "ok";
    case EKYA_ERR_INVALID_ARG: return "invalid argument";
    case EKYA_ERR_NOMEM: return "out of device memory";
    case EKYA_ERR_HIP: return "HIP runtime error";
    case EKYA_ERR_NONFINITE: return "non-finite training loss";
    case EKYA_ERR_UNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}

const char* ekya_last_error(const ekya_ctx* ctx) {
  return ctx ? ctx->c.err.c_str() : g_noctx_err.c_str();
}

ekya_status ekya_create(ekya_ctx** out, int hip_device, int n_classes, size_t workspace_bytes) {
  return ekya_create_head(out, hip_device, n_classes, 0, workspace_bytes);
}

ekya_status ekya_create_head(ekya_ctx** out, int hip_device, int n_classes, int hidden,
                             size_t workspace_bytes) {
  if (!out) return fail(nullptr, EKYA_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  if (n_classes < 1 || n_classes > 1024)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "n_classes must be in [1, 1024]");
  if (hidden < 0 || hidden > EKYA_MAX_HIDDEN)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "hidden must be in [0, EKYA_MAX_HIDDEN]");
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n == 0)
    return fail(nullptr, EKYA_ERR_HIP, "no HIP device available");
  if (hip_device < 0 || hip_device >= n)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "hip_device out of range");
  ekya_ctx* c = new (std::nothrow) ekya_ctx();
  if (!c) return fail(nullptr, EKYA_ERR_NOMEM, "host allocation failed");
  hipError_t e = ekya::ctx_init(c->c, hip_device, n_classes, hidden, workspace_bytes);
  if (e != hipSuccess) {
    ekya::ctx_free(c->c);
    delete c;
    return fail(nullptr, e == hipErrorOutOfMemory ? EKYA_ERR_NOMEM : EKYA_ERR_HIP,
                std::string("HIP error: ") + hipGetErrorString(e));
  }
  *out = c;
  return EKYA_OK;
}

void ekya_destroy(ekya_ctx* ctx) {
  if (!ctx) return;
  ekya::ctx_free(ctx->c);
  delete ctx;
}

static ekya_status check_train(ekya_ctx* ctx, int k, double frac, int epochs, float lr, float mu,
                               int batch) {
  if (k < 1 || k > 6) return fail(ctx, EKYA_ERR_INVALID_ARG, "k_trainable must be in [1, 6]");
  if (!(frac > 0.0 && frac <= 1.0))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "subsample_frac must be in (0, 1]");
  if (epochs < 1 || epochs > EKYA_MAX_EPOCHS)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "epochs must be in [1, EKYA_MAX_EPOCHS]");
  if (!(lr > 0.f) || !std::isfinite(lr)) return fail(ctx, EKYA_ERR_INVALID_ARG, "lr must be > 0");
  if (!(mu >= 0.f && mu < 1.f)) return fail(ctx, EKYA_ERR_INVALID_ARG, "momentum must be in [0, 1)");
  if (batch < 1 || batch > 4096) return fail(ctx, EKYA_ERR_INVALID_ARG, "batch must be in [1, 4096]");
  return EKYA_OK;
}

// Sizes and options of a retraining call (pointers checked by the caller).
static ekya_status check_retrain_args(ekya_ctx* ctx, int k, int n_frames, int H, int W,
                                      int n_heldout, const ekya_train_opts* opts) {
  if (!opts) return fail(ctx, EKYA_ERR_INVALID_ARG, "opts is null");
  if (n_frames < 1 || n_frames > (1 << 24))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "n_frames must be in [1, 2^24]");
  if (n_heldout < 1 || n_heldout > (1 << 24))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "n_heldout must be in [1, 2^24]");
  if (ekya_status s = check_frames(ctx, H, W)) return s;
  if (!valid_precision(opts->precision))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "precision must be EKYA_FP32 or EKYA_BF16");
  return check_train(ctx, k, opts->subsample_frac, opts->epochs, opts->lr, opts->momentum,
                     opts->batch);
}

ekya_status ekya_retrain(ekya_ctx* ctx, float* weights, int k_trainable, const void* frames,
                         const int32_t* labels, int n_frames, int H, int W,
                         const void* heldout_frames, const int32_t* heldout_labels, int n_heldout,
                         const ekya_train_opts* opts, ekya_retrain_result* result, void* stream) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (!weights || !frames || !labels || !heldout_frames || !heldout_labels || !opts || !result)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "null pointer argument");
  if (ekya_status s = check_retrain_args(ctx, k_trainable, n_frames, H, W, n_heldout, opts))
    return s;
  if (result->step_loss_capacity < 0 || (result->step_loss_capacity > 0 && !result->step_loss))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "step_loss capacity without a buffer");
  if (ctx->c.ckpt && ctx->c.ckpt->dt != opts->precision)
    return fail(ctx, EKYA_ERR_INVALID_ARG,
                "the checkpoint model's precision differs from the retraining precision");
  ctx->c.err.clear();
  return ekya::run_retrain(ctx->c, weights, k_trainable, frames, labels, n_frames, H, W,
                           heldout_frames, heldout_labels, n_heldout, *opts, result,
                           (hipStream_t)stream);
}

size_t ekya_retrain_workspace_head(int n_classes, int hidden, int k_trainable, int n_frames, int H,
                                   int W, int n_heldout, const ekya_train_opts* opts) {
  if (n_classes < 1 || n_classes > 1024 || hidden < 0 || hidden > EKYA_MAX_HIDDEN ||
      check_retrain_args(nullptr, k_trainable, n_frames, H, W, n_heldout, opts) != EKYA_OK)
    return 0;
  const ekya::Net net = ekya::Net::build(n_classes, opts->precision, hidden);
  return ekya::retrain_workspace_bytes(net, k_trainable, n_frames, H, W, n_heldout, *opts);
}

size_t ekya_retrain_workspace(int n_classes, int k_trainable, int n_frames, int H, int W,
                              int n_heldout, const ekya_train_opts* opts) {
  return ekya_retrain_workspace_head(n_classes, 0, k_trainable, n_frames, H, W, n_heldout, opts);
}

// Sizes and candidates of a profiling call (pointers checked by the caller).
static ekya_status check_profile_args(ekya_ctx* ctx, const ekya_profile_cfg* cfgs, int n_cfgs,
                                      int n_frames, int H, int W, int n_heldout, int precision) {
  if (!cfgs) return fail(ctx, EKYA_ERR_INVALID_ARG, "cfgs is null");
  if (n_cfgs < 1 || n_cfgs > 256) return fail(ctx, EKYA_ERR_INVALID_ARG, "n_cfgs must be in [1, 256]");
  if (n_frames < 1 || n_frames > (1 << 24))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "n_frames must be in [1, 2^24]");
  if (n_heldout < 1 || n_heldout > (1 << 24))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "n_heldout must be in [1, 2^24]");
  if (ekya_status s = check_frames(ctx, H, W)) return s;
  if (!valid_precision(precision))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "precision must be EKYA_FP32 or EKYA_BF16");
  for (int i = 0; i < n_cfgs; ++i) {
    const ekya_profile_cfg& c = cfgs[i];
    if (ekya_status s = check_train(ctx, c.k_trainable, c.subsample_frac, c.epochs, c.lr, c.momentum,
                                    c.batch))
      return s;
  }
  return EKYA_OK;
}

ekya_status ekya_profile(ekya_ctx* ctx, const float* weights, const ekya_profile_cfg* cfgs,
                         int n_cfgs, const void* frames, const int32_t* labels, int n_frames,
                         int H, int W, const void* heldout_frames, const int32_t* heldout_labels,
                         int n_heldout, uint64_t subsample_seed, int precision, int concurrent,
                         ekya_profile_result* results) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (!weights || !cfgs || !frames || !labels || !heldout_frames || !heldout_labels || !results)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "null pointer argument");
  if (ekya_status s = check_profile_args(ctx, cfgs, n_cfgs, n_frames, H, W, n_heldout, precision))
    return s;
  ctx->c.err.clear();
  return ekya::run_profile(ctx->c, weights, cfgs, n_cfgs, frames, labels, n_frames, H, W,
                           heldout_frames, heldout_labels, n_heldout, subsample_seed, precision,
                           concurrent, results);
}

size_t ekya_profile_workspace_head(int n_classes, int hidden, const ekya_profile_cfg* cfgs,
                                   int n_cfgs, int n_frames, int H, int W, int n_heldout,
                                   int precision) {
  if (n_classes < 1 || n_classes > 1024 || hidden < 0 || hidden > EKYA_MAX_HIDDEN ||
      check_profile_args(nullptr, cfgs, n_cfgs, n_frames, H, W, n_heldout, precision) != EKYA_OK)
    return 0;
  const ekya::Net net = ekya::Net::build(n_classes, precision, hidden);
  return ekya::profile_workspace_bytes(net, cfgs, n_cfgs, n_frames, H, W, n_heldout);
}

size_t ekya_profile_workspace(int n_classes, const ekya_profile_cfg* cfgs, int n_cfgs,
                              int n_frames, int H, int W, int n_heldout, int precision) {
  return ekya_profile_workspace_head(n_classes, 0, cfgs, n_cfgs, n_frames, H, W, n_heldout,
                                     precision);
}

ekya_status ekya_infer(ekya_ctx* ctx, const float* weights, const void* frames, int n, int H,
                       int W, int resolution, int precision, int32_t* labels_out, void* stream) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (n < 0 || n > (1 << 26)) return fail(ctx, EKYA_ERR_INVALID_ARG, "n must be in [0, 2^26]");
  if (n == 0) return EKYA_OK;
  if (!weights || !frames || !labels_out) return fail(ctx, EKYA_ERR_INVALID_ARG, "null pointer argument");
  if (ekya_status s = check_frames(ctx, H, W)) return s;
  if (resolution < 32 || resolution > 4096)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "resolution must be in [32, 4096]");
  if (!valid_precision(precision))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "precision must be EKYA_FP32 or EKYA_BF16");
  ctx->c.err.clear();
  return ekya::run_infer(ctx->c, weights, frames, n, H, W, resolution, precision, labels_out,
                         (hipStream_t)stream);
}

size_t ekya_infer_workspace_head(int n_classes, int hidden, int resolution, int precision) {
  if (n_classes < 1 || n_classes > 1024 || hidden < 0 || hidden > EKYA_MAX_HIDDEN ||
      resolution < 32 || resolution > 4096 || !valid_precision(precision))
    return 0;
  const ekya::Net net = ekya::Net::build(n_classes, precision, hidden);
  return ekya::infer_workspace_bytes(net, resolution);
}

size_t ekya_infer_workspace(int n_classes, int resolution, int precision) {
  return ekya_infer_workspace_head(n_classes, 0, resolution, precision);
}

ekya_status ekya_set_kernel_timing(ekya_ctx* ctx, int enable) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (enable) {
    hipError_t e = ekya::ctx_collect_timing(ctx->c);
    if (e != hipSuccess) return fail(ctx, EKYA_ERR_HIP, std::string("HIP error: ") + hipGetErrorString(e));
    ctx->c.stats.clear();
  }
  ctx->c.timing = enable != 0;
  return EKYA_OK;
}

int ekya_kernel_timing(ekya_ctx* ctx, int index, char* name, int name_cap, long long* launches,
                       double* total_ms, double* flops, double* bytes) {
  if (!ctx || index < 0 || !name || name_cap < 1) return -1;
  if (ekya::ctx_collect_timing(ctx->c) != hipSuccess) return -1;
  if (index >= (int)ctx->c.stats.size()) return -1;
  auto it = ctx->c.stats.begin();
  std::advance(it, index);
  std::snprintf(name, name_cap, "%s", it->first.c_str());
  if (launches) *launches = it->second.launches;
  if (total_ms) *total_ms = it->second.ms;
  if (flops) *flops = it->second.flops;
  if (bytes) *bytes = it->second.bytes;
  return 0;
}

int ekya_training_subset(int n_frames, double subsample_frac, uint64_t seed, int32_t* idx_out,
                         int capacity) {
  if (n_frames < 1 || !(subsample_frac > 0.0 && subsample_frac <= 1.0) || !idx_out) return -1;
  const int n = ekya::subset_count(n_frames, subsample_frac);
  if (n > capacity) return -1;
  std::vector<int32_t> s = ekya::training_subset(n_frames, subsample_frac, seed);
  std::memcpy(idx_out, s.data(), n * sizeof(int32_t));
  return n;
}

int ekya_epoch_order(int n, uint64_t seed, int epoch, int32_t* order_out) {
  if (n < 1 || epoch < 0 || !order_out) return -1;
  std::vector<int32_t> o = ekya::epoch_order(n, seed, epoch);
  std::memcpy(order_out, o.data(), n * sizeof(int32_t));
  return 0;
}

}  // extern "C"

// ------------------------------------------------------------------ ops
namespace {

struct Tmp {
  std::vector<void*> ptrs;
  ~Tmp() {
    for (void* p : ptrs) (void)hipFree(p);
  }
  template <typename T> T* get(size_t n) {
    void* p = nullptr;
    if (hipMalloc(&p, std::max<size_t>(n, 1) * sizeof(T) + 64) != hipSuccess) return nullptr;
    ptrs.push_back(p);
    return reinterpret_cast<T*>(p);
  }
};

bool chan_ok(int dt, int C, bool allow3) {
  if (allow3 && C == 3) return true;
  return C > 0 && C % ekya::dtype_vec(dt) == 0;
}

// Repack fp32 [K][C][R][S] weights into the kernels' low-precision layouts.
hipError_t pack_one(int dt, const float* w, int K, int C, int R, int S, int Cp, Tmp& tmp,
                    void** krsc, void** crsk, hipStream_t st) {
  const long long n = (long long)K * C * R * S;
  float* m = tmp.get<float>(n);
  long long* tab = tmp.get<long long>(16);
  const size_t es = ekya::dtype_size(dt);
  char* sh = tmp.get<char>((size_t)(K * R * S * Cp + n) * es);
  if (!m || !tab || !sh) return hipErrorOutOfMemory;
  long long h[13] = {0, K, C, R, S, 0, K, R, S, C, Cp, 0, (long long)K * R * S * Cp};
  EKYA_HIP(hipMemcpy(tab, h, sizeof(h), hipMemcpyHostToDevice));
  EKYA_HIP(ekya::permute_weights(w, m, tab, 1, n, 1, st));
  EKYA_HIP(ekya::pack_conv_weights(dt, m, tab + 5, 1, sh, st));
  *krsc = sh;
  *crsk = sh + (size_t)K * R * S * Cp * es;
  return hipSuccess;
}

hipError_t pad_input(int dt, const void* x, int N, int H, int W, int C, int& Cp, Tmp& tmp,
                     const void** xp, hipStream_t st) {
  Cp = C;
  *xp = x;
  if (C != 3) return hipSuccess;
  Cp = ekya::dtype_vec(dt);
  void* p = tmp.get<char>((size_t)N * H * W * Cp * ekya::dtype_size(dt));
  if (!p) return hipErrorOutOfMemory;
  EKYA_HIP(ekya::frames_to_padded(dt, x, nullptr, N, H, W, Cp, p, st));
  *xp = p;
  return hipSuccess;
}

ekya::ConvGeom make_geom(int N, int H, int W, int Cp, int K, int R, int S, int stride, int pad) {
  ekya::ConvGeom g;
  g.N = N; g.H = H; g.W = W; g.C = Cp; g.K = K; g.R = R; g.S = S;
  g.stride = stride; g.pad = pad;
  g.P = (H + 2 * pad - R) / stride + 1;
  g.Q = (W + 2 * pad - S) / stride + 1;
  return g;
}

bool conv_args_ok(int dt, int N, int H, int W, int C, int K, int R, int S, int stride, int pad,
                  bool allow3) {
  if (!valid_precision(dt) || N < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || stride < 1 ||
      pad < 0)
    return false;
  if (!chan_ok(dt, C, allow3) || K % ekya::dtype_vec(dt) != 0) return false;
  if (H + 2 * pad < R || W + 2 * pad < S) return false;
  return true;
}

ekya_status sync_status(hipStream_t st, hipError_t e) {
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  return hip_status(e);
}

}  // namespace

extern "C" {

ekya_status ekya_op_conv2d(int precision, const void* x, int N, int H, int W, int C,
                           const float* w, int K, int R, int S, int stride, int pad, void* y,
                           void* stream) {
  if (!x || !w || !y || !conv_args_ok(precision, N, H, W, C, K, R, S, stride, pad, true))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid conv2d arguments");
  hipStream_t st = (hipStream_t)stream;
  Tmp tmp;
  int Cp;
  const void* xp;
  void *krsc, *crsk;
  hipError_t e = pad_input(precision, x, N, H, W, C, Cp, tmp, &xp, st);
  if (e == hipSuccess) e = pack_one(precision, w, K, C, R, S, Cp, tmp, &krsc, &crsk, st);
  const ekya::ConvGeom g = make_geom(N, H, W, Cp, K, R, S, stride, pad);
  const size_t wsf = ekya::conv_split_workspace_floats(precision, g, false);
  float* ws = wsf ? tmp.get<float>(wsf) : nullptr;
  if (wsf && !ws) e = hipErrorOutOfMemory;
  if (e == hipSuccess) e = ekya::conv_fwd(precision, g, xp, krsc, y, ekya::ConvEpilogue(), ws, wsf, st);
  return sync_status(st, e);
}

ekya_status ekya_op_conv2d_dgrad(int precision, const void* dy, const float* w, int N, int H,
                                 int W, int C, int K, int R, int S, int stride, int pad, void* dx,
                                 void* stream) {
  if (!dy || !w || !dx || !conv_args_ok(precision, N, H, W, C, K, R, S, stride, pad, false) ||
      K % (8 * ekya::dtype_vec(precision)) != 0 || stride > 2)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid conv2d_dgrad arguments");
  hipStream_t st = (hipStream_t)stream;
  Tmp tmp;
  void *krsc, *crsk;
  hipError_t e = pack_one(precision, w, K, C, R, S, C, tmp, &krsc, &crsk, st);
  const ekya::ConvGeom g = make_geom(N, H, W, C, K, R, S, stride, pad);
  const size_t wsf = ekya::conv_split_workspace_floats(precision, g, true);
  float* ws = wsf ? tmp.get<float>(wsf) : nullptr;
  if (wsf && !ws) e = hipErrorOutOfMemory;
  if (e == hipSuccess) e = ekya::conv_dgrad(precision, g, dy, crsk, dx, nullptr, ws, wsf, st);
  return sync_status(st, e);
}

ekya_status ekya_op_conv2d_wgrad(int precision, const void* x, const void* dy, int N, int H,
                                 int W, int C, int K, int R, int S, int stride, int pad,
                                 float* dw, void* stream) {
  if (!x || !dy || !dw || !conv_args_ok(precision, N, H, W, C, K, R, S, stride, pad, true))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid conv2d_wgrad arguments");
  hipStream_t st = (hipStream_t)stream;
  Tmp tmp;
  int Cp;
  const void* xp;
  hipError_t e = pad_input(precision, x, N, H, W, C, Cp, tmp, &xp, st);
  ekya::ConvGeom g = make_geom(N, H, W, Cp, K, R, S, stride, pad);
  g.C0 = C;  // the plan (and so its scratch) depends on the real channel count
  float* part = tmp.get<float>(ekya::conv_wgrad_workspace_floats(precision, g));
  float* krsc = tmp.get<float>((size_t)K * R * S * C);
  long long* tab = tmp.get<long long>(8);
  if (!part || !krsc || !tab) e = hipErrorOutOfMemory;
  if (e == hipSuccess) e = ekya::conv_wgrad(precision, g, xp, dy, part, krsc, C, st);
  if (e == hipSuccess) {
    long long h[5] = {0, K, C, R, S};
    e = hipMemcpy(tab, h, sizeof(h), hipMemcpyHostToDevice);
  }
  if (e == hipSuccess) e = ekya::permute_weights(krsc, dw, tab, 1, (long long)K * C * R * S, 0, st);
  return sync_status(st, e);
}

ekya_status ekya_op_batchnorm_train(int precision, const void* z, long long M, int C,
                                    const float* gamma, const float* beta, float* running_mean,
                                    float* running_var, int relu, void* y, float* mean_out,
                                    float* invstd_out, void* stream) {
  if (!valid_precision(precision) || !z || !gamma || !beta || !y || !mean_out || !invstd_out ||
      M < 1 || !chan_ok(precision, C, false) || C > 2048 ||
      (running_mean == nullptr) != (running_var == nullptr))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid batchnorm_train arguments");
  hipStream_t st = (hipStream_t)stream;
  Tmp tmp;
  float* part = tmp.get<float>(ekya::bn_partials_floats(M, C));
  float* ss = tmp.get<float>(2 * (size_t)C);
  hipError_t e = (part && ss) ? hipSuccess : hipErrorOutOfMemory;
  if (e == hipSuccess)
    e = ekya::bn_train_forward(precision, z, M, C, gamma, beta, running_mean, running_var,
                               mean_out, invstd_out, ss, ss + C, nullptr, relu, y, part, st);
  return sync_status(st, e);
}

// ---------------------------------------------- BatchNorm without allocation
// Device scratch of ekya_op_batchnorm_train_noalloc: the BatchNorm partial
// sums (bn_partials_floats(M, C), largest at 512 chunks of 2 x 2048
// channels plus 3 x 2048) followed by the per-channel scale and shift
// (2 x 2048).  Each GPU the library runs on holds its own copy until the
// process ends.  In host code only the address from hipGetSymbolAddress is
// used (the array's name is a host-side stand-in).
constexpr size_t kBnScratchFloats = 512 * 2 * 2048 + 3 * 2048 + 2 * 2048;
static __device__ __align__(256) float scratch[kBnScratchFloats];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per device.
hipError_t scratch_on_current_device(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = reinterpret_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

ekya_status ekya_op_batchnorm_train_noalloc(int precision, const void* z, long long M, int C,
                                            const float* gamma, const float* beta,
                                            float* running_mean, float* running_var, int relu,
                                            void* y, float* mean_out, float* invstd_out,
                                            void* stream) {
  if (!valid_precision(precision) || !z || !gamma || !beta || !y || !mean_out || !invstd_out ||
      M < 1 || !chan_ok(precision, C, false) || C > 2048 ||
      (running_mean == nullptr) != (running_var == nullptr))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid batchnorm_train_noalloc arguments");
  const size_t part = ekya::bn_partials_floats(M, C);
  if (part + 2 * (size_t)C > kBnScratchFloats)
    return fail(nullptr, EKYA_ERR_INVALID_ARG,
                "batchnorm_train_noalloc: M and C need more scratch than the static " +
                    std::to_string(kBnScratchFloats) + " floats");
  float* sp = nullptr;
  hipError_t e = scratch_on_current_device(&sp);
  if (e != hipSuccess) return hip_status(e);
  hipStream_t st = (hipStream_t)stream;
  // every partial is written before it is read, so nothing needs clearing
  float* ss = sp + part;
  e = ekya::bn_train_forward(precision, z, M, C, gamma, beta, running_mean, running_var, mean_out,
                             invstd_out, ss, ss + C, nullptr, relu, y, sp, st);
  if (e == hipSuccess) e = hipGetLastError();
  return hip_status(e);
}

ekya_status ekya_op_batchnorm_backward(int precision, const void* dy, const void* y_relu,
                                       const void* z, long long M, int C, const float* gamma,
                                       const float* mean, const float* invstd, void* dz,
                                       float* dgamma, float* dbeta, void* stream) {
  if (!valid_precision(precision) || !dy || !z || !gamma || !mean || !invstd || !dz || !dgamma ||
      !dbeta || M < 1 || !chan_ok(precision, C, false) || C > 2048)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid batchnorm_backward arguments");
  hipStream_t st = (hipStream_t)stream;
  Tmp tmp;
  float* part = tmp.get<float>(ekya::bn_partials_floats(M, C));
  hipError_t e = part ? hipSuccess : hipErrorOutOfMemory;
  if (e == hipSuccess)
    e = ekya::bn_backward(precision, dy, y_relu, z, M, C, gamma, mean, invstd, dgamma, dbeta, dz,
                          nullptr, part, st);
  return sync_status(st, e);
}

ekya_status ekya_op_maxpool(int precision, const void* x, int N, int H, int W, int C, void* y,
                            uint8_t* arg, void* stream) {
  if (!valid_precision(precision) || !x || !y || N < 1 || H < 1 || W < 1 ||
      !chan_ok(precision, C, false))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid maxpool arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::maxpool_fwd(precision, x, N, H, W, C, y, arg, st));
}

ekya_status ekya_op_maxpool_backward(int precision, const void* dy, const uint8_t* arg, int N,
                                     int H, int W, int C, void* dx, void* stream) {
  if (!valid_precision(precision) || !dy || !arg || !dx || N < 1 || H < 1 || W < 1 ||
      !chan_ok(precision, C, false))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid maxpool_backward arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::maxpool_bwd(precision, dy, arg, N, H, W, C, dx, st));
}

ekya_status ekya_op_avgpool(int precision, const void* x, int N, int H, int W, int C, float* f,
                            void* stream) {
  if (!valid_precision(precision) || !x || !f || N < 1 || H < 1 || W < 1 || C < 1)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid avgpool arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::avgpool_fwd(precision, x, N, H * W, C, f, st));
}

ekya_status ekya_op_avgpool_backward(int precision, const float* df, int N, int H, int W, int C,
                                     void* dx, void* stream) {
  if (!valid_precision(precision) || !df || !dx || N < 1 || H < 1 || W < 1 || C < 1)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid avgpool_backward arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::avgpool_bwd(precision, df, N, H * W, C, dx, st));
}

ekya_status ekya_op_linear(const float* f, const float* Wt, const float* b, int N, int I, int J,
                           float* z, void* stream) {
  if (!f || !Wt || !b || !z || N < 1 || I < 1 || J < 1)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid linear arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::fc_fwd(f, Wt, b, N, I, J, z, st));
}

ekya_status ekya_op_linear_backward(const float* dz, const float* f, const float* Wt, int N,
                                    int I, int J, float* dW, float* db, float* df, void* stream) {
  if (!dz || !f || !Wt || !dW || !db || N < 1 || I < 1 || J < 1)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid linear_backward arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::fc_bwd(dz, f, Wt, N, I, J, dW, db, df, st));
}

ekya_status ekya_op_softmax_ce(const float* z, const int32_t* labels, int N, int J, float* dz,
                               float* out, void* stream) {
  if (!z || !labels || !dz || !out || N < 1 || J < 1)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid softmax_ce arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::softmax_ce(z, labels, nullptr, N, J, dz, out, st));
}

ekya_status ekya_op_sgd(float* w, float* v, const float* g, long long n, float lr, float mu,
                        void* stream) {
  if (!w || !v || !g || n < 0) return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid sgd arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::sgd_momentum(w, v, g, n, lr, mu, st));
}

ekya_status ekya_op_resize(int precision, const void* frames, int n, int H, int W, int r,
                           void* out, void* stream) {
  if (!valid_precision(precision) || !frames || !out || n < 1 || H < 1 || W < 1 || r < 1)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid resize arguments");
  hipStream_t st = (hipStream_t)stream;
  return sync_status(st, ekya::resize_to_padded(precision, frames, n, H, W, r, 3, out, st));
}

}  // extern "C"

// ------------------------------------------------------ scheduling layer
extern "C" {

ekya_status ekya_nnls(const double* A, int m, int n, const double* b, double* x, double* rnorm) {
  if (!A || !b || !x || m < 1 || n < 1 || m > 4096 || n > 4096 || (long long)m * n > (1LL << 22))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid nnls arguments");
  for (long long i = 0; i < (long long)m * n; ++i)
    if (!std::isfinite(A[i])) return fail(nullptr, EKYA_ERR_INVALID_ARG, "nnls: A is not finite");
  for (int i = 0; i < m; ++i)
    if (!std::isfinite(b[i])) return fail(nullptr, EKYA_ERR_INVALID_ARG, "nnls: b is not finite");
  if (!ekya::nnls(A, m, n, b, x, rnorm))
    return fail(nullptr, EKYA_ERR_UNSUPPORTED, "nnls: singular least-squares subproblem");
  return EKYA_OK;
}

ekya_status ekya_fit_accuracy_curve(const double* x, const double* acc, int n, ekya_curve* out) {
  if (!x || !acc || !out || n < 1 || n > 4096)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid curve-fit arguments");
  for (int i = 0; i < n; ++i)
    if (!(x[i] > 0.0) || !std::isfinite(x[i]) || !(acc[i] >= 0.0 && acc[i] <= 1.0))
      return fail(nullptr, EKYA_ERR_INVALID_ARG, "curve fit: need x > 0 and accuracy in [0, 1]");
  ekya::Curve c;
  if (!ekya::fit_accuracy_curve(x, acc, n, &c))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "curve fit failed");
  *out = ekya_curve{c.b0, c.b1, c.b2, c.rss};
  return EKYA_OK;
}

double ekya_curve_accuracy(const ekya_curve* c, double x) {
  if (!c) return 0.0;
  ekya::Curve k;
  k.b0 = c->b0;
  k.b1 = c->b1;
  k.b2 = c->b2;
  return ekya::curve_accuracy(k, x);
}

ekya_status ekya_extrapolate(const ekya_profile_cfg* cfg, const ekya_profile_result* res,
                             int n_frames, int epochs_target, ekya_curve* curve, double* acc_out,
                             double* gpu_seconds_out) {
  if (!cfg || !res || n_frames < 1 || epochs_target < 1 || cfg->epochs < 1 ||
      cfg->epochs > EKYA_MAX_EPOCHS || cfg->batch < 1 || res->n_train < 1 ||
      res->n_train > n_frames || res->status != EKYA_OK)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid extrapolation arguments");
  const double f = (double)res->n_train / n_frames;
  double xs[EKYA_MAX_EPOCHS], acc[EKYA_MAX_EPOCHS], sec = 0.0;
  for (int e = 0; e < cfg->epochs; ++e) {
    xs[e] = (e + 1) * f;
    acc[e] = res->heldout_acc[e];
    sec += res->epoch_seconds[e];
  }
  ekya_curve c;
  if (ekya_status s = ekya_fit_accuracy_curve(xs, acc, cfg->epochs, &c)) return s;
  const long long steps_sub = (res->n_train + cfg->batch - 1) / cfg->batch;
  const long long steps_full = ((long long)n_frames + cfg->batch - 1) / cfg->batch;
  if (curve) *curve = c;
  if (acc_out) *acc_out = ekya_curve_accuracy(&c, (double)epochs_target);
  if (gpu_seconds_out)
    *gpu_seconds_out = sec / cfg->epochs * (double)steps_full / (double)steps_sub * epochs_target;
  return EKYA_OK;
}

ekya_status ekya_thief_schedule(const ekya_video* videos, int n_videos, double n_gpus, double delta,
                                double window_s, double a_min, ekya_schedule* out) {
  if (!videos || !out || !out->alloc || !out->infer_choice || !out->train_choice ||
      !out->video_accuracy || n_videos < 1 || n_videos > 1024 || !(delta > 0.0) ||
      !(n_gpus > 0.0) || !(window_s > 0.0) || !std::isfinite(a_min))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "invalid scheduler arguments");
  const double qd = n_gpus / delta;
  const long long quanta = std::llround(qd);
  if (std::fabs(qd - (double)quanta) > 1e-9 * std::max(1.0, qd) || quanta < 1 || quanta > 4096)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "n_gpus must be a whole number (1..4096) of quanta");
  std::vector<ekya::SchedVideo> vs(n_videos);
  for (int v = 0; v < n_videos; ++v) {
    const ekya_video& in = videos[v];
    if (in.n_infer < 1 || !in.infer || in.n_train < 0 || (in.n_train > 0 && !in.train) ||
        !std::isfinite(in.acc_now))
      return fail(nullptr, EKYA_ERR_INVALID_ARG, "scheduler: a stream needs inference configurations");
    vs[v].acc_now = in.acc_now;
    for (int i = 0; i < in.n_infer; ++i) {
      if (!(in.infer[i].cost > 0.0) || !std::isfinite(in.infer[i].factor))
        return fail(nullptr, EKYA_ERR_INVALID_ARG, "scheduler: inference cost must be > 0");
      vs[v].infer.push_back({in.infer[i].cost, in.infer[i].factor});
    }
    for (int i = 0; i < in.n_train; ++i) {
      if (!(in.train[i].gpu_seconds >= 0.0) || !std::isfinite(in.train[i].acc_after))
        return fail(nullptr, EKYA_ERR_INVALID_ARG, "scheduler: retraining cost must be >= 0");
      vs[v].train.push_back({in.train[i].acc_after, in.train[i].gpu_seconds});
    }
  }
  const ekya::SchedResult r = ekya::thief_schedule(vs, (int)quanta, delta, window_s, a_min);
  for (int j = 0; j < 2 * n_videos; ++j) out->alloc[j] = r.quanta[j] * delta;
  for (int v = 0; v < n_videos; ++v) {
    out->infer_choice[v] = r.infer_choice[v];
    out->train_choice[v] = r.train_choice[v];
    out->video_accuracy[v] = r.video_accuracy[v];
  }
  out->accuracy = r.accuracy;
  return EKYA_OK;
}

}  // extern "C"

// ------------------------------------------------------- joint inference and retraining
namespace {

bool valid_range(double begin, double share) {
  return begin >= 0.0 && begin < 1.0 && share > 0.0 && begin + share <= 1.0 + 1e-9;
}

}  // namespace

extern "C" {

int ekya_partition_mask(int n_cu, int n_xcd, int n_se, double cu_begin, double cu_share,
                        uint32_t* mask_out, int words) {
  if (n_cu > (1 << 16) || n_xcd > (1 << 10) || n_se > (1 << 10)) return -1;
  return ekya::partition_mask(n_cu, n_xcd, n_se, cu_begin, cu_share, mask_out, words);
}

ekya_status ekya_stream_create(int hip_device, double cu_begin, double cu_share,
                               void** stream_out) {
  if (!stream_out) return fail(nullptr, EKYA_ERR_INVALID_ARG, "stream_out is null");
  *stream_out = nullptr;
  if (!valid_range(cu_begin, cu_share))
    return fail(nullptr, EKYA_ERR_INVALID_ARG,
                "CU range must satisfy 0 <= cu_begin < 1, cu_share > 0, cu_begin + cu_share <= 1");
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n == 0)
    return fail(nullptr, EKYA_ERR_HIP, "no HIP device available");
  if (hip_device < 0 || hip_device >= n)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "hip_device out of range");
  std::vector<uint32_t> mask;
  int count = 0;
  hipError_t e = ekya::device_partition_mask(hip_device, cu_begin, cu_share, mask, &count);
  if (e != hipSuccess)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "the CU range selects no row of CUs");
  int prev = 0;
  if (hipGetDevice(&prev) != hipSuccess) prev = hip_device;
  hipStream_t st = nullptr;
  e = hipSetDevice(hip_device);
  if (e == hipSuccess) e = ekya::create_masked_stream(mask, &st);
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_status(e);
  *stream_out = st;
  return EKYA_OK;
}

ekya_status ekya_stream_destroy(void* stream) {
  if (!stream) return fail(nullptr, EKYA_ERR_INVALID_ARG, "stream is null");
  return hip_status(hipStreamDestroy((hipStream_t)stream));
}

int ekya_stream_cu_count(void* stream) {
  hipDevice_t dev = 0;
  if (hipStreamGetDevice((hipStream_t)stream, &dev) != hipSuccess) return -1;
  int n_cu = 0;
  if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return -1;
  // sized for either reading of the size argument (words or bits)
  std::vector<uint32_t> mask((size_t)32 * ((n_cu + 31) / 32), 0u);
  if (hipExtStreamGetCUMask((hipStream_t)stream, (uint32_t)mask.size(), mask.data()) != hipSuccess)
    return -1;
  int c = 0;
  for (int i = 0; i < n_cu; ++i) c += (mask[i / 32] >> (i % 32)) & 1u;
  return c;
}

ekya_status ekya_set_cu_partition(ekya_ctx* ctx, double cu_begin, double cu_share) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (!valid_range(cu_begin, cu_share))
    return fail(ctx, EKYA_ERR_INVALID_ARG,
                "CU range must satisfy 0 <= cu_begin < 1, cu_share > 0, cu_begin + cu_share <= 1");
  std::vector<uint32_t> mask;
  const bool whole = cu_begin == 0.0 && cu_share >= 1.0;
  if (!whole) {
    int count = 0;
    if (ekya::device_partition_mask(ctx->c.device, cu_begin, cu_share, mask, &count) != hipSuccess)
      return fail(ctx, EKYA_ERR_INVALID_ARG, "the CU range selects no row of CUs");
  }
  hipError_t e = ekya::ctx_reset_streams(ctx->c);
  if (e != hipSuccess) return fail(ctx, EKYA_ERR_HIP, std::string("HIP error: ") + hipGetErrorString(e));
  ctx->c.cu_mask = mask;
  return EKYA_OK;
}

ekya_status ekya_cu_ids(int n_workgroups, uint32_t* ids_out, void* stream) {
  if (n_workgroups < 1 || n_workgroups > (1 << 20))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "n_workgroups must be in [1, 2^20]");
  if (!ids_out) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ids_out is null");
  return hip_status(ekya::cu_ids(n_workgroups, ids_out, (hipStream_t)stream));
}

ekya_status ekya_model_create(ekya_model** out, int hip_device, int n_classes, int precision) {
  return ekya_model_create_head(out, hip_device, n_classes, 0, precision);
}

ekya_status ekya_model_create_head(ekya_model** out, int hip_device, int n_classes, int hidden,
                                   int precision) {
  if (!out) return fail(nullptr, EKYA_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  if (n_classes < 1 || n_classes > 1024)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "n_classes must be in [1, 1024]");
  if (hidden < 0 || hidden > EKYA_MAX_HIDDEN)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "hidden must be in [0, EKYA_MAX_HIDDEN]");
  if (!valid_precision(precision))
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "precision must be EKYA_FP32 or EKYA_BF16");
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n == 0)
    return fail(nullptr, EKYA_ERR_HIP, "no HIP device available");
  if (hip_device < 0 || hip_device >= n)
    return fail(nullptr, EKYA_ERR_INVALID_ARG, "hip_device out of range");
  ekya_model* m = new (std::nothrow) ekya_model();
  if (!m) return fail(nullptr, EKYA_ERR_NOMEM, "host allocation failed");
  hipError_t e = ekya::model_init(m->m, hip_device, n_classes, hidden, precision);
  if (e != hipSuccess) {
    ekya::model_free(m->m);
    delete m;
    return hip_status(e);
  }
  *out = m;
  return EKYA_OK;
}

void ekya_model_destroy(ekya_model* m) {
  if (!m) return;
  ekya::model_free(m->m);
  delete m;
}

ekya_status ekya_model_load(ekya_model* m, const float* weights, void* stream,
                            uint64_t* version_out) {
  if (!m || !weights) return fail(nullptr, EKYA_ERR_INVALID_ARG, "null pointer argument");
  return hip_status(ekya::model_load(m->m, weights, nullptr, (hipStream_t)stream, version_out));
}

ekya_status ekya_model_export(ekya_model* m, float* weights_out, void* stream,
                              uint64_t* version_out) {
  if (!m || !weights_out) return fail(nullptr, EKYA_ERR_INVALID_ARG, "null pointer argument");
  bool empty = false;
  hipError_t e = ekya::model_export(m->m, weights_out, (hipStream_t)stream, version_out, &empty);
  if (empty) return fail(nullptr, EKYA_ERR_INVALID_ARG, "the model has no published weights");
  return hip_status(e);
}

uint64_t ekya_model_version(ekya_model* m) {
  if (!m) return 0;
  std::lock_guard<std::mutex> lk(m->m.mu);
  return m->m.current < 0 ? 0 : m->m.slot[m->m.current].version;
}

ekya_status ekya_infer_model(ekya_ctx* ctx, ekya_model* m, const void* frames, int n, int H, int W,
                             int resolution, int32_t* labels_out, void* stream,
                             uint64_t* version_out) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (!m) return fail(ctx, EKYA_ERR_INVALID_ARG, "model is null");
  if (n < 0 || n > (1 << 26)) return fail(ctx, EKYA_ERR_INVALID_ARG, "n must be in [0, 2^26]");
  if (m->m.device != ctx->c.device || m->m.n_classes != ctx->c.n_classes ||
      m->m.hidden != ctx->c.hidden)
    return fail(ctx, EKYA_ERR_INVALID_ARG,
                "the model's device, class count or hidden layer differs from the context's");
  if (ekya_model_version(m) == 0)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "the model has no published weights (call ekya_model_load first)");
  if (n == 0) return EKYA_OK;
  if (!frames || !labels_out) return fail(ctx, EKYA_ERR_INVALID_ARG, "null pointer argument");
  if (ekya_status s = check_frames(ctx, H, W)) return s;
  if (resolution < 32 || resolution > 4096)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "resolution must be in [32, 4096]");
  ctx->c.err.clear();
  return ekya::run_infer_model(ctx->c, m->m, frames, n, H, W, resolution, labels_out,
                               (hipStream_t)stream, version_out);
}

ekya_status ekya_infer_models(ekya_ctx* ctx, ekya_model* const* models, int n_models,
                              const void* frames, const int* counts, int H, int W, int resolution,
                              int32_t* labels_out, uint64_t* versions_out, void* stream) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (!models || !counts) return fail(ctx, EKYA_ERR_INVALID_ARG, "null pointer argument");
  if (n_models < 1 || n_models > 4096)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "n_models must be in [1, 4096]");
  long long total = 0;
  std::vector<ekya::Model*> ms(n_models);
  for (int i = 0; i < n_models; ++i) {
    if (!models[i]) return fail(ctx, EKYA_ERR_INVALID_ARG, "a model is null");
    const ekya::Model& m = models[i]->m;
    if (m.device != ctx->c.device || m.n_classes != ctx->c.n_classes || m.hidden != ctx->c.hidden)
      return fail(ctx, EKYA_ERR_INVALID_ARG,
                  "a model's device, class count or hidden layer differs from the context's");
    if (m.dt != models[0]->m.dt)
      return fail(ctx, EKYA_ERR_INVALID_ARG, "the models' precisions differ");
    if (ekya_model_version(models[i]) == 0)
      return fail(ctx, EKYA_ERR_INVALID_ARG, "a model has no published weights");
    if (counts[i] < 0) return fail(ctx, EKYA_ERR_INVALID_ARG, "counts must be >= 0");
    total += counts[i];
    ms[i] = &models[i]->m;
  }
  if (total > (1 << 26)) return fail(ctx, EKYA_ERR_INVALID_ARG, "more than 2^26 frames");
  if (total > 0 && (!frames || !labels_out))
    return fail(ctx, EKYA_ERR_INVALID_ARG, "null pointer argument");
  if (ekya_status s = check_frames(ctx, H, W)) return s;
  if (resolution < 32 || resolution > 4096)
    return fail(ctx, EKYA_ERR_INVALID_ARG, "resolution must be in [32, 4096]");
  ctx->c.err.clear();
  return ekya::run_infer_models(ctx->c, ms.data(), n_models, frames, counts, H, W, resolution,
                                labels_out, versions_out, (hipStream_t)stream);
}

size_t ekya_infer_models_workspace(int n_classes, int hidden, int resolution, int precision,
                                   int n_models) {
  if (n_classes < 1 || n_classes > 1024 || hidden < 0 || hidden > EKYA_MAX_HIDDEN ||
      resolution < 32 || resolution > 4096 || !valid_precision(precision) || n_models < 1 ||
      n_models > 4096)
    return 0;
  const ekya::Net net = ekya::Net::build(n_classes, precision, hidden);
  return ekya::infer_models_workspace_bytes(net, resolution, n_models);
}

ekya_status ekya_set_checkpoint(ekya_ctx* ctx, ekya_model* m, int every_epochs) {
  if (!ctx) return fail(nullptr, EKYA_ERR_INVALID_ARG, "ctx is null");
  if (m) {
    if (every_epochs < 1) return fail(ctx, EKYA_ERR_INVALID_ARG, "every_epochs must be >= 1");
    if (m->m.device != ctx->c.device || m->m.n_classes != ctx->c.n_classes ||
        m->m.hidden != ctx->c.hidden)
      return fail(ctx, EKYA_ERR_INVALID_ARG,
                  "the model's device, class count or hidden layer differs from the context's");
  }
  ctx->c.ckpt = m ? &m->m : nullptr;
  ctx->c.ckpt_every = m ? every_epochs : 0;
  return EKYA_OK;
}

}  // extern "C"
