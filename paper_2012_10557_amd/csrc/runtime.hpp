// Host runtime behind the C ABI: context, workspace arenas, and the
// retraining / profiling / inference jobs.
#pragma once

#include <map>
#include <mutex>
#include <string>
#include <utility>
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

// One slot of a prepared inference model: internal-layout fp32 weights,
// folded eval-mode BatchNorm and the low-precision convolution weights.
struct ModelSlot {
  float* master = nullptr;
  float* fold = nullptr;
  void* shadow = nullptr;
  hipEvent_t ready = nullptr;  // recorded after the load that filled the slot
  // per stream, an event recorded after the latest inference call (or
  // export) on that stream that read the slot; a load into the slot waits
  // for all of them
  std::vector<std::pair<hipStream_t, hipEvent_t>> uses;
  uint64_t version = 0;
};

// Double-buffered inference model (hot reload of retrained weights).
struct Model {
  int device = 0;
  int n_classes = 0;
  int hidden = 0;
  int dt = 0;
  Net net;
  Tables tabs;
  DeviceBuf mem;
  ModelSlot slot[2];
  int current = -1;  // published slot, -1 before the first load
  uint64_t next_version = 1;
  std::vector<hipEvent_t> pool;  // spare use events
  std::mutex mu;                 // guards everything above after init
};

hipError_t model_init(Model& m, int device, int n_classes, int hidden, int dt);
void model_free(Model& m);
// Fill the unpublished slot on `stream` from canonical weights (canonical !=
// null) or from internal-layout fp32 weights (internal), then publish it.
hipError_t model_load(Model& m, const float* canonical, const float* internal, hipStream_t stream,
                      uint64_t* version);
hipError_t model_export(Model& m, float* canonical_out, hipStream_t stream, uint64_t* version,
                        bool* empty);

// CU mask of a range [begin, begin + share) of a device with n_cu CUs on
// n_xcd dies of n_se shader engines; returns the CU count or -1.
int partition_mask(int n_cu, int n_xcd, int n_se, double begin, double share, uint32_t* mask,
                   int words);
hipError_t device_partition_mask(int device, double begin, double share,
                                 std::vector<uint32_t>& mask, int* count);
hipError_t create_masked_stream(const std::vector<uint32_t>& mask, hipStream_t* s);

struct KernelStat {
  long long launches = 0;
  double ms = 0.0, flops = 0.0, bytes = 0.0;
};

struct Ctx {
  int device = 0;
  int n_classes = 0;
  int hidden = 0;  // neurons of the hidden classifier layer (0: none)
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
  // inference lanes of ekya_infer_models, and their fork / join events
  std::vector<hipStream_t> lanes;
  hipEvent_t lane_fork = nullptr;
  hipEvent_t lane_join[4] = {nullptr, nullptr, nullptr, nullptr};
  // CU mask of the context's own streams (empty: every CU)
  std::vector<uint32_t> cu_mask;
  // checkpointing during retraining: publish into ckpt every ckpt_every epochs
  Model* ckpt = nullptr;
  int ckpt_every = 0;
  bool timing = false;
  KernelTimer timer;
  std::map<std::string, KernelStat> stats;
};

// Read the events of finished timed launches into `stats`.
hipError_t ctx_collect_timing(Ctx& c);

hipError_t ctx_init(Ctx& c, int device, int n_classes, int hidden, size_t workspace_bytes);
// Wait for the context's queued work and release its own streams (they are
// created again, with the current cu_mask, when next needed).
hipError_t ctx_reset_streams(Ctx& c);

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
size_t infer_models_workspace_bytes(const Net& net, int resolution, int n_models);
ekya_status run_infer_models(Ctx& c, Model* const* models, int n_models, const void* frames,
                             const int* counts, int H, int W, int resolution, int32_t* labels_out,
                             uint64_t* versions, hipStream_t stream);
ekya_status run_infer_model(Ctx& c, Model& m, const void* frames, int n, int H, int W,
                            int resolution, int32_t* labels_out, hipStream_t stream,
                            uint64_t* version);

}  // namespace ekya
