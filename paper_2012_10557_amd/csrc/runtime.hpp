// Host runtime behind the C ABI: context, workspace arenas, and the
// retraining / profiling / inference jobs.
#pragma once

#include <map>
#include <string>
#include <vector>

#include "../../include/ekya.h"
#include "kernels.hpp"
#include "net.hpp"

namespace ekya {

// Device buffer owned by the context.
struct DeviceBuf {
  void* p = nullptr;
  size_t cap = 0;
  hipError_t alloc(size_t bytes);  // exactly `bytes` (releases what it held)
  void release();
};

// Bump allocator over a DeviceBuf; a measuring pass (base == nullptr) sizes it.
struct Arena {
  char* base = nullptr;
  size_t used = 0;
  template <typename T> T* take(size_t count) {
    size_t a = (used + 255) & ~(size_t)255;
    used = a + count * sizeof(T);
    return base ? reinterpret_cast<T*>(base + a) : nullptr;
  }
  void* take_bytes(size_t bytes) { return take<char>(bytes); }
};

// Device copies of the per-network tables the kernels read.
struct Tables {
  DeviceBuf buf;
  const long long* permute = nullptr;
  int n_permute = 0;
  const long long* fold_all = nullptr;
  int n_fold_all = 0;
  const long long* pack_all = nullptr;  // every conv, [K][R][S][C] shadow only
  int n_pack_all = 0;
  // per lowest trainable stage (0..5)
  const long long* fold_train[6] = {nullptr};
  int n_fold_train[6] = {0};
  const long long* pack_frozen[6] = {nullptr};
  int n_pack_frozen[6] = {0};
  const long long* pack_train[6] = {nullptr};
  int n_pack_train[6] = {0};
  // step-end SGD ranges (offset, length) and repacking of the parameters
  // without a fused per-convolution update
  const long long* sgd_rest[6] = {nullptr};
  int n_sgd_rest[6] = {0};
  long long sgd_rest_max[6] = {0};
  const long long* pack_rest[6] = {nullptr};
  int n_pack_rest[6] = {0};
};

struct KernelStat {
  long long launches = 0;
  double ms = 0.0, flops = 0.0, bytes = 0.0;
};

struct Ctx {
  int device = 0;
  int n_classes = 0;
  std::string err;
  Net net[2];
  Tables tabs[2];
  // The workspace arena every call plans its device buffers in.  With
  // fixed_ws it was allocated once at creation and is never replaced; a call
  // that needs more fails before queueing any work.  Otherwise a call that
  // needs more replaces it before queueing any work, after the context's
  // previous call has finished.
  DeviceBuf ws;
  bool fixed_ws = false;
  // Recorded after the last work of every call that used the arena; the next
  // call's stream waits for it (calls on one context run in turn on the GPU).
  hipEvent_t last_done = nullptr;
  std::vector<hipStream_t> streams;  // profiler streams (default priority)
  hipStream_t eval_stream = nullptr;  // retraining's held-out evaluation (default priority)
  bool timing = false;
  KernelTimer timer;
  std::map<std::string, KernelStat> stats;
};

// Read the events of finished timed launches into `stats`.
hipError_t ctx_collect_timing(Ctx& c);

hipError_t ctx_init(Ctx& c, int device, int n_classes, size_t workspace_bytes);

// Bytes of workspace arena a call with these arguments plans (host only;
// arguments already validated).
size_t retrain_workspace_bytes(const Net& net, int k, int n_frames, int H, int W, int n_heldout,
                               const ekya_train_opts& o);
size_t profile_workspace_bytes(const Net& net, const ekya_profile_cfg* cfgs, int n_cfgs,
                               int n_frames, int H, int W, int n_heldout);
size_t infer_workspace_bytes(const Net& net, int resolution);
void ctx_free(Ctx& c);

ekya_status run_retrain(Ctx& c, float* weights, int k, const void* frames, const int32_t* labels,
                        int n_frames, int H, int W, const void* hframes, const int32_t* hlabels,
                        int n_heldout, const ekya_train_opts& o, ekya_retrain_result* res,
                        hipStream_t stream);
ekya_status run_profile(Ctx& c, const float* weights, const ekya_profile_cfg* cfgs, int n_cfgs,
                        const void* frames, const int32_t* labels, int n_frames, int H, int W,
                        const void* hframes, const int32_t* hlabels, int n_heldout,
                        uint64_t subsample_seed, int precision, int concurrent,
                        ekya_profile_result* out);
ekya_status run_infer(Ctx& c, const float* weights, const void* frames, int n, int H, int W,
                      int resolution, int precision, int32_t* labels_out, hipStream_t stream);

}  // namespace ekya
