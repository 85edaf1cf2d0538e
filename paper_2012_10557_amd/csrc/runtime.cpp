// Retraining, micro-profiling and inference jobs.
//
// Retraining of the last k stages (sections 3.1 and 4.3):
//   1. draw the uniform training subset S of the window (host, seeded);
//   2. run the frozen stages once per frame of S and of the held-out set, in
//      eval mode, into the feature cache (stages below the lowest trainable
//      stage never change during the job, so this is an exact reuse);
//   3. for every epoch: visit S in a seeded random order in batches (last
//      partial batch kept); per batch gather cached features, run the
//      trainable stages in train mode, mean softmax cross-entropy, backward
//      through the trainable stages only, SGD with momentum, repack the
//      low-precision weight copies;
//   4. after every epoch measure held-out accuracy in eval mode (the
//      micro-profiler's per-epoch accuracy, section 4.3) and the epoch's GPU
//      time (resource demand per epoch at the full GPU, section 4.3).
// All device work of a job is ordered on one stream; the host reads results
// once at the end.
#include "runtime.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <thread>

#include "rng.hpp"

namespace ekya {

hipError_t DeviceBuf::alloc(size_t bytes) {
  release();
  hipError_t e = hipMalloc(&p, std::max<size_t>(bytes, 256));
  if (e != hipSuccess) {
    p = nullptr;
    return e;
  }
  cap = std::max<size_t>(bytes, 256);
  return hipSuccess;
}

void DeviceBuf::release() {
  if (p) (void)hipFree(p);
  p = nullptr;
  cap = 0;
}

// Convolutions whose momentum step runs right after their weight gradient
// (conv_weight_update from the split partials); the others' gradients go
// through the gradient buffer and the step-end SGD.
static bool fused_update(const Net& net, const ConvL& c) {
  ConvGeom g;
  g.C = c.cin_pad;
  g.K = c.cout;
  return c.cin == c.cin_pad && conv_wgrad_partials_ok(net.dt, g);
}

// (offset, length) ranges of the trainable parameters from stage lo on that
// the step-end SGD updates: everything but the fused convolutions' weights.
static std::vector<long long> sgd_rest_table(const Net& net, int lo, long long* max_len) {
  std::vector<std::pair<long long, long long>> skip;
  for (const ConvL& c : net.conv)
    if (c.stage >= lo && c.stage <= 4 && fused_update(net, c))
      skip.push_back({c.off, c.off + (long long)c.cout * c.R * c.S * c.cin});
  std::sort(skip.begin(), skip.end());
  std::vector<long long> t;
  long long pos = net.stage_begin[lo];
  *max_len = 0;
  auto emit = [&](long long a, long long b) {
    if (b <= a) return;
    t.insert(t.end(), {a, b - a});
    *max_len = std::max(*max_len, b - a);
  };
  for (auto& r : skip) {
    emit(pos, r.first);
    pos = std::max(pos, r.second);
  }
  emit(pos, net.total);
  return t;
}

// ----------------------------------------------------------------- tables
static hipError_t upload_tables(const Net& net, Tables& t) {
  std::vector<long long> all;
  std::vector<std::pair<const long long**, size_t>> fix;
  auto put = [&](const std::vector<long long>& v, const long long** dst, int* n, int row) {
    fix.push_back({dst, all.size()});
    *n = (int)(v.size() / row);
    all.insert(all.end(), v.begin(), v.end());
  };
  put(net.permute_table(), &t.permute, &t.n_permute, 5);
  put(net.fold_table(0, 5), &t.fold_all, &t.n_fold_all, 6);
  put(net.pack_table(0, 4, false), &t.pack_all, &t.n_pack_all, 8);
  for (int lo = 0; lo <= 5; ++lo) {
    put(net.fold_table(lo, 5), &t.fold_train[lo], &t.n_fold_train[lo], 6);
    put(net.pack_table(0, lo - 1, false), &t.pack_frozen[lo], &t.n_pack_frozen[lo], 8);
    put(net.pack_table(lo, 4, true), &t.pack_train[lo], &t.n_pack_train[lo], 8);
    put(sgd_rest_table(net, lo, &t.sgd_rest_max[lo]), &t.sgd_rest[lo], &t.n_sgd_rest[lo], 2);
    std::vector<long long> pr;
    for (const ConvL& c : net.conv)
      if (c.stage >= lo && c.stage <= 4 && !fused_update(net, c))
        pr.insert(pr.end(), {c.off, c.cout, c.R, c.S, c.cin, c.cin_pad, c.sh_krsc, c.sh_crsk});
    put(pr, &t.pack_rest[lo], &t.n_pack_rest[lo], 8);
  }
  EKYA_HIP(t.buf.alloc(all.size() * sizeof(long long) + 16));
  EKYA_HIP(hipMemcpy(t.buf.p, all.data(), all.size() * sizeof(long long), hipMemcpyHostToDevice));
  for (auto& f : fix) *f.first = reinterpret_cast<const long long*>(t.buf.p) + f.second;
  return hipSuccess;
}

hipError_t ctx_init(Ctx& c, int device, int n_classes, int hidden, size_t workspace_bytes) {
  c.device = device;
  c.n_classes = n_classes;
  c.hidden = hidden;
  EKYA_HIP(hipSetDevice(device));
  for (int dt = 0; dt < 2; ++dt) {
    c.net[dt] = Net::build(n_classes, dt, hidden);
    EKYA_HIP(upload_tables(c.net[dt], c.tabs[dt]));
  }
  EKYA_HIP(hipEventCreateWithFlags(&c.last_done, hipEventDisableTiming));
  if (workspace_bytes > 0) {
    EKYA_HIP(c.ws.alloc(workspace_bytes));
    c.fixed_ws = true;
  }
  return hipSuccess;
}

// Give the call `need` bytes of arena and order `stream` after the
// context's previous call.  On failure nothing has been queued.
static ekya_status acquire_workspace(Ctx& c, size_t need, hipStream_t stream) {
  if (need > c.ws.cap) {
    if (c.fixed_ws) {
      c.err = "workspace of " + std::to_string(c.ws.cap) + " bytes is too small: the call needs " +
              std::to_string(need) + " bytes";
      return EKYA_ERR_NOMEM;
    }
    // grow mode: the previous call must be done with the old arena
    hipError_t e = hipEventSynchronize(c.last_done);
    if (e == hipSuccess) e = c.ws.alloc(need + need / 8 + (1 << 20));
    if (e != hipSuccess) {
      c.err = std::string("workspace of ") + std::to_string(need) + " bytes: " + hipGetErrorString(e);
      return e == hipErrorOutOfMemory ? EKYA_ERR_NOMEM : EKYA_ERR_HIP;
    }
  }
  hipError_t e = hipStreamWaitEvent(stream, c.last_done, 0);
  if (e != hipSuccess) {
    c.err = std::string("HIP error: ") + hipGetErrorString(e);
    return EKYA_ERR_HIP;
  }
  return EKYA_OK;
}

hipError_t ctx_collect_timing(Ctx& c) {
  for (LaunchRecord& r : c.timer.recs) {
    EKYA_HIP(hipEventSynchronize(r.e1));
    float ms = 0.f;
    EKYA_HIP(hipEventElapsedTime(&ms, r.e0, r.e1));
    KernelStat& st = c.stats[r.name];
    st.launches += 1;
    st.ms += ms;
    st.flops += r.flops;
    st.bytes += r.bytes;
    c.timer.pool.push_back(r.e0);
    c.timer.pool.push_back(r.e1);
  }
  c.timer.recs.clear();
  return hipSuccess;
}

void ctx_free(Ctx& c) {
  (void)hipSetDevice(c.device);
  (void)hipDeviceSynchronize();
  (void)ctx_collect_timing(c);
  for (hipEvent_t e : c.timer.pool) (void)hipEventDestroy(e);
  c.timer.pool.clear();
  for (hipStream_t s : c.streams) (void)hipStreamDestroy(s);
  c.streams.clear();
  for (hipStream_t s : c.lanes) (void)hipStreamDestroy(s);
  c.lanes.clear();
  if (c.eval_stream) (void)hipStreamDestroy(c.eval_stream);
  c.eval_stream = nullptr;
  if (c.lane_fork) (void)hipEventDestroy(c.lane_fork);
  c.lane_fork = nullptr;
  for (hipEvent_t& e : c.lane_join) {
    if (e) (void)hipEventDestroy(e);
    e = nullptr;
  }
  if (c.last_done) (void)hipEventDestroy(c.last_done);
  c.last_done = nullptr;
  c.ws.release();
  for (auto& t : c.tabs) t.buf.release();
}

// A stream of the context's own (default priority), restricted to the
// context's CU partition when it has one.
static hipError_t ctx_stream(const Ctx& c, hipStream_t* s) {
  if (c.cu_mask.empty()) return hipStreamCreateWithFlags(s, hipStreamNonBlocking);
  return create_masked_stream(c.cu_mask, s);
}

hipError_t ctx_reset_streams(Ctx& c) {
  EKYA_HIP(hipSetDevice(c.device));
  EKYA_HIP(hipEventSynchronize(c.last_done));
  for (hipStream_t s : c.streams) EKYA_HIP(hipStreamSynchronize(s));
  for (hipStream_t s : c.lanes) EKYA_HIP(hipStreamSynchronize(s));
  if (c.eval_stream) EKYA_HIP(hipStreamSynchronize(c.eval_stream));
  for (hipStream_t s : c.streams) (void)hipStreamDestroy(s);
  c.streams.clear();
  for (hipStream_t s : c.lanes) (void)hipStreamDestroy(s);
  c.lanes.clear();
  if (c.eval_stream) (void)hipStreamDestroy(c.eval_stream);
  c.eval_stream = nullptr;
  return hipSuccess;
}

// ------------------------------------------------------------ CU shares
// The amdgpu driver deals CU-mask bits to the dies first, then to the
// shader engines of a die, then to the CUs of an engine: bit b is CU
// b / (X S) of engine (b / X) mod S on die b mod X (X dies, S engines, R CUs
// per die).  A share is counted in groups of one CU per die; group
// g = k S + s takes CU k of engine s on every die, so a run of groups spreads
// over the engines of every die as evenly as whole groups allow.  Where
// R = X S (the CUs per engine equal the dies, as on MI355X: 8 dies of 4
// engines of 8 CUs) the CU index k is rotated to (j + s + k) mod X for die j:
// the bits of a group then also fall in X different blocks of R bits, so a
// die-by-die numbering (bit b on die b / R) would still give every die one
// CU per group.  Otherwise the group of row r puts die j on bit
// j R + (r + j) mod R, one CU per die under either numbering.  Disjoint group
// ranges give disjoint bits.
int partition_mask(int n_cu, int n_xcd, int n_se, double begin, double share, uint32_t* mask,
                   int words) {
  if (n_cu < 1 || n_xcd < 1 || n_se < 1 || n_cu % n_xcd != 0 || !mask ||
      words < (n_cu + 31) / 32)
    return -1;
  if (!(begin >= 0.0 && begin < 1.0) || !(share > 0.0) || begin + share > 1.0 + 1e-9) return -1;
  const int X = n_xcd, R = n_cu / n_xcd;
  const int g0 = (int)std::lround(begin * R);
  const int g1 = std::min(R, (int)std::lround((begin + share) * R));
  if (g1 <= g0) return -1;
  std::fill(mask, mask + words, 0u);
  const bool engines = R % n_se == 0 && R / n_se == X;
  for (int g = g0; g < g1; ++g)
    for (int j = 0; j < X; ++j) {
      int b;
      if (engines) {
        const int S = n_se, k = g / S, s = g % S;
        b = X * S * ((j + s + k) % X) + X * s + j;
      } else {
        b = j * R + (g + j) % R;
      }
      mask[b / 32] |= 1u << (b % 32);
    }
  return (g1 - g0) * X;
}

// Shader engines per die: 4 on the CDNA3 and CDNA4 dies.
static constexpr int kEnginesPerXcd = 4;

hipError_t device_partition_mask(int device, double begin, double share,
                                 std::vector<uint32_t>& mask, int* count) {
  int n_cu = 0, n_xcd = 1;
  EKYA_HIP(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device));
  if (hipDeviceGetAttribute(&n_xcd, hipDeviceAttributeNumberOfXccs, device) != hipSuccess ||
      n_xcd < 1 || n_cu % n_xcd != 0)
    n_xcd = 1;
  mask.assign((n_cu + 31) / 32, 0u);
  *count = partition_mask(n_cu, n_xcd, kEnginesPerXcd, begin, share, mask.data(),
                          (int)mask.size());
  return *count > 0 ? hipSuccess : hipErrorInvalidValue;
}

// hipExtStreamCreateWithCUMask's size argument counts mask words in the
// runtime (its documentation calls it the size of the bit array): the mask
// is passed zero-padded to 32 times its words, which reads the same mask
// under either reading and ignores bits past the device's CUs.
hipError_t create_masked_stream(const std::vector<uint32_t>& mask, hipStream_t* s) {
  std::vector<uint32_t> padded(mask.size() * 32, 0u);
  std::copy(mask.begin(), mask.end(), padded.begin());
  return hipExtStreamCreateWithCUMask(s, (uint32_t)padded.size(), padded.data());
}


// --------------------------------------------------------- eval forward
// Buffers for running stages in eval mode on up to `cap` frames.
struct EvalBufs {
  void *p0 = nullptr, *p1 = nullptr, *t1 = nullptr, *sc = nullptr;
  float* pooled = nullptr;
  float* hid = nullptr;  // hidden classifier layer's activations
  float* logits = nullptr;
  float* ws = nullptr;  // split-reduction partials of the forward convs
  size_t ws_floats = 0;
};

static ConvGeom conv_geom(const Net& net, const Geo& g, int ci, int n);

static long long max_act_elems(const Net& net, const Geo& g, int lo, int hi) {
  long long m = 0;
  if (lo <= 0 && hi >= 0) m = std::max(m, (long long)g.sh * g.sw * 64);
  for (size_t i = 1; i < net.conv.size(); ++i) {
    const ConvL& c = net.conv[i];
    if (c.stage < lo || c.stage > hi) continue;
    m = std::max(m, (long long)g.ih[i] * g.iw[i] * c.cin);
    m = std::max(m, (long long)g.oh[i] * g.ow[i] * c.cout);
  }
  return std::max(m, 512LL);
}

static void plan_eval(Arena& a, const Net& net, const Geo& g, int lo, int hi, int cap, EvalBufs& b) {
  const size_t es = dtype_size(net.dt);
  const long long m = max_act_elems(net, g, lo, hi) * cap;
  b.p0 = a.take_bytes(m * es);
  b.p1 = a.take_bytes(m * es);
  b.t1 = a.take_bytes(m * es);
  b.sc = a.take_bytes(m * es);
  b.pooled = a.take<float>((size_t)cap * 512);
  if (net.hidden > 0) b.hid = a.take<float>((size_t)cap * net.hidden);
  b.logits = a.take<float>((size_t)cap * net.n_classes);
  // split-reduction scratch for every frame count a call may use, so that a
  // convolution's plan never depends on how large this scratch happens to be
  size_t ws = 16;
  for (size_t i = 0; i < net.conv.size(); ++i)
    if (net.conv[i].stage >= lo && net.conv[i].stage <= hi)
      for (int n = 1; n <= cap; ++n)
        ws = std::max(ws, conv_split_workspace_floats(net.dt, conv_geom(net, g, (int)i, n), false));
  b.ws_floats = ws;
  b.ws = a.take<float>(ws);
}

static ConvGeom conv_geom(const Net& net, const Geo& g, int ci, int n) {
  const ConvL& c = net.conv[ci];
  ConvGeom cg;
  cg.N = n;
  cg.H = g.ih[ci];
  cg.W = g.iw[ci];
  cg.C = c.cin_pad;
  cg.K = c.cout;
  cg.R = c.R;
  cg.S = c.S;
  cg.stride = c.stride;
  cg.pad = c.pad;
  cg.P = g.oh[ci];
  cg.Q = g.ow[ci];
  cg.C0 = c.cin;
  return cg;
}

static inline const char* shadow_at(const Net& net, const void* shadow, long long off) {
  return reinterpret_cast<const char*>(shadow) + off * (long long)dtype_size(net.dt);
}
static inline void* shadow_at(const Net& net, void* shadow, long long off) {
  return reinterpret_cast<char*>(shadow) + off * (long long)dtype_size(net.dt);
}

// Run stages lo..hi in eval mode (BatchNorm folded into the conv epilogue) on
// n frames.  Output: hi <= 3: the stage's output tensor; hi == 4: the pooled
// fp32 features [n, 512]; hi == 5: fp32 logits [n, classes].
// raw: x (stage 0 only) is [.][H][W][3] frames, image i at raw_idx[i] when
// raw_idx != null, read directly by the stem (stem_frames_ok).
static hipError_t eval_forward(const Net& net, const Geo& g, const void* shadow, const float* fold,
                               const float* master, int lo, int hi, const void* x, int n,
                               EvalBufs& b, void* out, hipStream_t st, bool raw = false,
                               const int32_t* raw_idx = nullptr) {
  const int dt = net.dt;
  const void* cur = x;
  auto fold_scale = [&](int bi) { return fold + 2 * net.bn[bi].st; };
  auto fold_shift = [&](int bi) { return fold + 2 * net.bn[bi].st + net.bn[bi].C; };
  for (int s = lo; s <= hi; ++s) {
    if (s == 0) {
      ConvEpilogue e;
      e.scale = fold_scale(net.conv[0].bn);
      e.shift = fold_shift(net.conv[0].bn);
      e.relu = 1;
      void* dst = (hi == 0) ? out : b.p0;
      const ConvGeom cg = conv_geom(net, g, 0, n);
      if (stem_pool_ok(dt, cg)) {  // stem and max pool in one kernel
        EKYA_HIP(stem_pool_fwd(dt, cg, cur, raw, raw_idx,
                               shadow_at(net, shadow, net.conv[0].sh_krsc), dst, e, st));
        cur = dst;
        continue;
      }
      if (raw)
        EKYA_HIP(stem_fwd_frames(dt, cg, cur, raw_idx, shadow_at(net, shadow, net.conv[0].sh_krsc),
                                 b.t1, e, st));
      else
        EKYA_HIP(conv_fwd(dt, cg, cur, shadow_at(net, shadow, net.conv[0].sh_krsc), b.t1, e, b.ws,
                          b.ws_floats, st));
      EKYA_HIP(maxpool_fwd(dt, b.t1, n, g.sh, g.sw, 64, dst, nullptr, st));
      cur = dst;
    } else if (s <= 4) {
      int nb_in_stage = 0;
      for (const BlockL& bl : net.blk) nb_in_stage += (bl.stage == s);
      int bidx = 0;
      for (const BlockL& bl : net.blk) {
        if (bl.stage != s) continue;
        const bool last = (++bidx == nb_in_stage);
        void* dst = (last && hi == s && s <= 3) ? out : (cur == b.p0 ? b.p1 : b.p0);
        ConvEpilogue e1;
        e1.scale = fold_scale(net.conv[bl.c1].bn);
        e1.shift = fold_shift(net.conv[bl.c1].bn);
        e1.relu = 1;
        EKYA_HIP(conv_fwd(dt, conv_geom(net, g, bl.c1, n), cur,
                          shadow_at(net, shadow, net.conv[bl.c1].sh_krsc), b.t1, e1, b.ws,
                          b.ws_floats, st));
        const void* res = cur;
        if (bl.cd >= 0) {
          ConvEpilogue ed;
          ed.scale = fold_scale(net.conv[bl.cd].bn);
          ed.shift = fold_shift(net.conv[bl.cd].bn);
          EKYA_HIP(conv_fwd(dt, conv_geom(net, g, bl.cd, n), cur,
                            shadow_at(net, shadow, net.conv[bl.cd].sh_krsc), b.sc, ed, b.ws,
                            b.ws_floats, st));
          res = b.sc;
        }
        ConvEpilogue e2;
        e2.scale = fold_scale(net.conv[bl.c2].bn);
        e2.shift = fold_shift(net.conv[bl.c2].bn);
        e2.res = res;
        e2.relu = 1;
        EKYA_HIP(conv_fwd(dt, conv_geom(net, g, bl.c2, n), b.t1,
                          shadow_at(net, shadow, net.conv[bl.c2].sh_krsc), dst, e2, b.ws,
                          b.ws_floats, st));
        cur = dst;
      }
      if (s == 4) {
        float* pd = (hi == 4) ? reinterpret_cast<float*>(out) : b.pooled;
        EKYA_HIP(avgpool_fwd(dt, cur, n, g.lh[4] * g.lw[4], 512, pd, st));
        cur = pd;
      }
    } else {  // s == 5
      const float* f = reinterpret_cast<const float*>(cur);
      if (net.hidden > 0) {
        EKYA_HIP(fc_fwd(f, master + net.fc1_w, master + net.fc1_b, n, 512, net.hidden, b.hid, st));
        EKYA_HIP(relu_f32(b.hid, b.hid, nullptr, (long long)n * net.hidden, st));
        f = b.hid;
      }
      EKYA_HIP(fc_fwd(f, master + net.fc_w, master + net.fc_b, n, net.head_in(), net.n_classes,
                      reinterpret_cast<float*>(out), st));
    }
  }
  return hipSuccess;
}

// ----------------------------------------------------------- train job
struct BlockAct {
  void *X = nullptr, *Z1 = nullptr, *A1 = nullptr, *Z2 = nullptr, *Zd = nullptr, *OUT = nullptr;
};

struct TrainJob {
  // configuration
  const Net* net = nullptr;
  const Tables* tabs = nullptr;
  Geo geo;
  int dt = 0, k = 1, lowest = 5;
  int B = 64, n_s = 0, n_h = 0, epochs = 1, n_steps = 0;
  float lr = 0.01f, mu = 0.9f;
  hipStream_t st = nullptr;
  // inputs
  const float* weights = nullptr;  // canonical
  const void* frames = nullptr;
  const int32_t* labels = nullptr;
  const void* hframes = nullptr;
  const int32_t* hlabels = nullptr;
  const void* cache = nullptr;     // training rows (positions in S), lowest >= 1
  const void* hcache = nullptr;    // held-out rows
  long long row_bytes = 0;
  std::vector<int32_t> h_order, h_fidx;  // host copies (epochs x n_s)
  // device buffers
  float *master = nullptr, *grad = nullptr, *mom = nullptr;
  void* shadow = nullptr;
  float *bn_mean = nullptr, *bn_invstd = nullptr, *bn_scale = nullptr, *bn_shift = nullptr;
  float* fold = nullptr;
  int32_t *d_order = nullptr, *d_fidx = nullptr;
  void* x0 = nullptr;
  void* stem_Z = nullptr;
  void* stem_A = nullptr;
  uint8_t* stem_arg = nullptr;
  std::vector<BlockAct> acts;  // per block of the network (only trainable ones set)
  void* g[6] = {nullptr};      // gradient scratch
  // weight gradients run on st2 while st continues down the data-gradient
  // chain; dz of conv2 / conv1 / downsample per block parity (double
  // buffered so st2 may lag one block), st2's own split scratch, and events
  hipStream_t st2 = nullptr;
  // retraining only: each epoch's held-out evaluation runs on st3 beside the
  // next epoch, from snapshots of the weights it reads; fork / done events
  hipStream_t st3 = nullptr;
  bool eval_overlap = false;  // planned with the snapshot buffers st3 reads
  void* shadow_snap = nullptr;
  float* master_snap = nullptr;
  hipEvent_t ev_eval_fork = nullptr, ev_eval_done = nullptr;
  bool eval_pending = false;
  void* gz2[2] = {nullptr}, *gz1[2] = {nullptr}, *gzd[2] = {nullptr};
  float* ws2 = nullptr;
  size_t ws2_floats = 0;
  // The backward pass records at most three forks per residual block (eight
  // blocks at full depth) plus the end join, the forward pass one per
  // projection shortcut; each half of the arrays holds more than that.
  static constexpr int kForks = 64;
  hipEvent_t fork[kForks] = {nullptr};
  hipEvent_t joined[kForks] = {nullptr};
  // joined[] index of the end-of-backward join that st has not waited for
  // yet (-1: none); see settle()
  int pending_join = -1;
  float *pooled = nullptr, *logits = nullptr, *dz = nullptr, *dpooled = nullptr;
  float *hid = nullptr, *dhid = nullptr;  // hidden classifier layer: activations, gradient
  float* ws = nullptr;         // split-K partials
  size_t ws_floats = 0;
  float* bn_ws = nullptr;      // BatchNorm partials
  size_t bn_ws_floats = 0;
  float* bn_ws2 = nullptr;     // BatchNorm partials of work on st2 (projection shortcuts)
  float* ce_out = nullptr;     // n_steps x 3
  int32_t* hcount = nullptr;   // epochs
  EvalBufs eval;
  int eval_cap = 0;
  void* eval_in = nullptr;     // padded frames for held-out eval when lowest == 0
  // ev[e]: start of epoch e on st (ev[epochs]: end of the loop); ev_tr[e]:
  // end of epoch e's training steps (both streams); ev_e0/ev_e1[e]: around
  // epoch e's held-out evaluation on the stream that runs it
  hipEvent_t ev[EKYA_MAX_EPOCHS + 1] = {nullptr};
  hipEvent_t ev_tr[EKYA_MAX_EPOCHS] = {nullptr};
  hipEvent_t ev_e0[EKYA_MAX_EPOCHS] = {nullptr}, ev_e1[EKYA_MAX_EPOCHS] = {nullptr};
  // retraining only: publish the weights into ckpt every ckpt_every epochs
  Model* ckpt = nullptr;
  int ckpt_every = 0;
};

// three forks per residual block, one more per projection shortcut whose
// data gradient is folded into conv1's, the end join
static_assert(3 * 8 + 3 + 1 <= TrainJob::kForks / 2, "fork events for a full-depth backward pass");

static size_t ws_floats(const TrainJob& j) {
  const Net& net = *j.net;
  size_t m = 0;
  for (size_t i = 0; i < net.conv.size(); ++i) {
    const ConvL& c = net.conv[i];
    if (c.stage < j.lowest || c.stage > 4) continue;
    // every batch size up to B (the last batch of an epoch may be partial)
    for (int n = 1; n <= j.B; ++n) {
      ConvGeom cg = conv_geom(net, j.geo, (int)i, n);
      m = std::max(m, conv_wgrad_workspace_floats(j.dt, cg));
      // the last weight gradients of a step run on the main stream in ws
      if (fused_update(net, c)) m = std::max(m, conv_wgrad_partials_floats(j.dt, cg));
      m = std::max(m, bn_partials_floats((long long)n * cg.P * cg.Q, c.cout));
      m = std::max(m, conv_split_workspace_floats(j.dt, cg, false));
      if (c.stage > 0) m = std::max(m, conv_split_workspace_floats(j.dt, cg, true));
    }
  }
  return std::max<size_t>(m, 16);
}

// Split scratch of the weight gradients (their own, used on st2).
static size_t wgrad_ws_floats(const TrainJob& j) {
  const Net& net = *j.net;
  size_t m = 16;
  for (size_t i = 0; i < net.conv.size(); ++i) {
    const ConvL& c = net.conv[i];
    if (c.stage < j.lowest || c.stage > 4) continue;
    for (int n = 1; n <= j.B; ++n) {
      const ConvGeom cg = conv_geom(net, j.geo, (int)i, n);
      m = std::max(m, fused_update(net, c) ? conv_wgrad_partials_floats(j.dt, cg)
                                           : conv_wgrad_workspace_floats(j.dt, cg));
    }
  }
  return m;
}

static long long train_max_elems(const TrainJob& j) {
  return max_act_elems(*j.net, j.geo, j.lowest, 4);
}

// Assign every device buffer of a job (arena sizing pass when a.base == null).
static void plan_job(Arena& a, TrainJob& j) {
  const Net& net = *j.net;
  const size_t es = dtype_size(j.dt);
  const long long tb = net.stage_begin[j.lowest];
  j.master = a.take<float>(net.total);
  j.grad = a.take<float>(net.total);
  j.mom = a.take<float>(net.total);
  (void)tb;
  j.shadow = a.take_bytes(net.shadow_elems * es);
  if (j.eval_overlap) {
    j.shadow_snap = a.take_bytes(net.shadow_elems * es);
    j.master_snap = a.take<float>(net.total);
  }
  j.bn_mean = a.take<float>(net.bn_channels);
  j.bn_invstd = a.take<float>(net.bn_channels);
  j.bn_scale = a.take<float>(net.bn_channels);
  j.bn_shift = a.take<float>(net.bn_channels);
  j.fold = a.take<float>(2 * net.bn_channels);
  j.d_order = a.take<int32_t>((size_t)j.epochs * j.n_s);
  j.d_fidx = a.take<int32_t>((size_t)j.epochs * j.n_s);
  const long long in_elems = j.geo.stage_in_elems(net, j.lowest);
  const size_t in_es = (j.lowest == 5) ? 4 : es;
  j.x0 = a.take_bytes((size_t)j.B * in_elems * in_es);
  j.acts.assign(net.blk.size(), BlockAct());
  if (j.lowest == 0) {
    j.stem_Z = a.take_bytes((size_t)j.B * j.geo.sh * j.geo.sw * 64 * es);
    j.stem_A = a.take_bytes((size_t)j.B * j.geo.sh * j.geo.sw * 64 * es);
    j.stem_arg = a.take<uint8_t>((size_t)j.B * j.geo.mh * j.geo.mw * 64);
  }
  for (size_t bi = 0; bi < net.blk.size(); ++bi) {
    const BlockL& b = net.blk[bi];
    if (b.stage < j.lowest || b.stage > 4) continue;
    BlockAct& t = j.acts[bi];
    const long long o1 = (long long)j.geo.oh[b.c1] * j.geo.ow[b.c1] * net.conv[b.c1].cout * j.B;
    t.Z1 = a.take_bytes(o1 * es);
    t.A1 = a.take_bytes(o1 * es);
    t.Z2 = a.take_bytes(o1 * es);
    t.OUT = a.take_bytes(o1 * es);
    if (b.cd >= 0) t.Zd = a.take_bytes(o1 * es);
    if (j.lowest == 0 && b.stage == 1 && bi == 0) {
      // input of layer1 comes from the stem's max pool
      t.X = a.take_bytes((size_t)j.B * j.geo.mh * j.geo.mw * 64 * es);
    }
  }
  const long long gmax = train_max_elems(j) * j.B;
  if (j.lowest <= 4) {
    for (int i = 0; i < 6; ++i) j.g[i] = a.take_bytes(gmax * es);
    for (int p = 0; p < 2; ++p) {
      j.gz2[p] = a.take_bytes(gmax * es);
      j.gz1[p] = a.take_bytes(gmax * es);
      j.gzd[p] = a.take_bytes(gmax * es);
    }
    // st2 also runs the projection-shortcut convolutions of the forward pass
    j.ws2_floats = std::max(wgrad_ws_floats(j), ws_floats(j));
    j.ws2 = a.take<float>(j.ws2_floats);
  }
  j.pooled = a.take<float>((size_t)j.B * 512);
  j.dpooled = a.take<float>((size_t)j.B * 512);
  if (net.hidden > 0) {
    j.hid = a.take<float>((size_t)j.B * net.hidden);
    j.dhid = a.take<float>((size_t)j.B * net.hidden);
  }
  j.logits = a.take<float>((size_t)j.B * net.n_classes);
  j.dz = a.take<float>((size_t)j.B * net.n_classes);
  j.ws_floats = ws_floats(j);
  j.ws = a.take<float>(j.ws_floats);
  j.bn_ws_floats = 16;
  for (size_t i = 0; i < net.conv.size(); ++i) {
    const ConvL& c = net.conv[i];
    if (c.stage < j.lowest || c.stage > 4) continue;
    for (int n = 1; n <= j.B; ++n) {
      const ConvGeom cg = conv_geom(net, j.geo, (int)i, n);
      j.bn_ws_floats = std::max(j.bn_ws_floats, bn_partials_floats((long long)n * cg.P * cg.Q, c.cout));
    }
  }
  j.bn_ws = a.take<float>(j.bn_ws_floats);
  j.bn_ws2 = a.take<float>(j.bn_ws_floats);
  j.ce_out = a.take<float>((size_t)j.n_steps * 3);
  j.hcount = a.take<int32_t>(j.epochs);
  // Held-out chunks: at most 512 frames; when the lowest trainable stage has
  // >= 256 channels its convolutions take 256 x 128 tiles one per CU, so a
  // chunk is cut to the frames whose tiles fill the 256 CUs once (400 frames
  // at 224 px would take 308 tiles: two rounds, the second one a fifth full).
  int cap = 512;
  if (j.lowest >= 1 && j.lowest <= 4) {
    const long long ch = 64LL << (j.lowest - 1);
    const long long hw = (long long)j.geo.lh[j.lowest] * j.geo.lw[j.lowest];
    if (ch >= 256 && hw > 0) cap = (int)std::max(1LL, std::min(512LL, 256LL * 128 / (hw * (ch / 256))));
  }
  j.eval_cap = std::max(1, std::min(j.n_h, cap));
  plan_eval(a, net, j.geo, j.lowest, 5, j.eval_cap, j.eval);
  if (j.lowest == 0) j.eval_in = a.take_bytes((size_t)j.eval_cap * in_elems * es);
}

static inline float* bnp(float* base, const BnL& b) { return base + b.st; }

// Average pool (x: layer4's output; null: the pooled features in x0) and
// the classifier: pooled and logits, or with a hidden layer the pooled
// features, the hidden layer's ReLU activations and the logits.
static hipError_t train_head_forward(TrainJob& j, int nb, const void* x) {
  const Net& net = *j.net;
  const int hw = j.geo.lh[4] * j.geo.lw[4];
  const float* f = x ? nullptr : reinterpret_cast<const float*>(j.x0);
  float* pooled = x ? j.pooled : nullptr;
  if (net.hidden == 0)
    return head_forward(j.dt, x, hw, f, j.master + net.fc_w, j.master + net.fc_b, nb, 512,
                        net.n_classes, pooled, j.logits, j.st);
  EKYA_HIP(head_forward(j.dt, x, hw, f, j.master + net.fc1_w, j.master + net.fc1_b, nb, 512,
                        net.hidden, pooled, j.hid, j.st));
  EKYA_HIP(relu_f32(j.hid, j.hid, nullptr, (long long)nb * net.hidden, j.st));
  return fc_fwd(j.hid, j.master + net.fc_w, j.master + net.fc_b, nb, net.hidden, net.n_classes,
                j.logits, j.st);
}

// Train-mode forward of stages lowest..5 on the batch in x0 (nb frames).
static hipError_t train_forward(TrainJob& j, int nb) {
  const Net& net = *j.net;
  const int dt = j.dt;
  hipStream_t st = j.st;
  // train-mode BN (statistics, running-statistic update, apply) of layer bi
  // on stream q with partial scratch part (ready > 0: the convolution
  // producing z left its chunk statistics there, in chunks of that many rows)
  auto bn_train_on = [&](int bi, const void* z, long long M, const void* res, int relu, void* y,
                         int ready, float* part, hipStream_t q) {
    const BnL& b = net.bn[bi];
    return bn_train_forward(dt, z, M, b.C, j.master + b.g, j.master + b.b, j.master + b.rm,
                            j.master + b.rv, bnp(j.bn_mean, b), bnp(j.bn_invstd, b),
                            bnp(j.bn_scale, b), bnp(j.bn_shift, b), res, relu, y, part, q, ready);
  };
  auto bn_train = [&](int bi, const void* z, long long M, const void* res, int relu, void* y,
                      int ready) { return bn_train_on(bi, z, M, res, relu, y, ready, j.bn_ws, st); };
  BnStatsSink sk;
  sk.part = j.bn_ws;
  // A projection shortcut (convolution + BatchNorm, BatchNorm partials in
  // bn_ws2) runs on st2 beside the block's main branch, with st2's split
  // scratch; st waits for it before the second BatchNorm, which adds it.
  // Events from the top of the fork arrays (the backward pass uses them from
  // the bottom).  With one stream it runs between the first convolution and
  // its BatchNorm.
  const bool two = j.st2 != st;
  BnStatsSink skd;
  skd.part = j.bn_ws2;
  int fi = TrainJob::kForks - 1;
  const void* cur = j.x0;
  for (int s = j.lowest; s <= 4; ++s) {
    if (s == 0) {
      ConvGeom cg = conv_geom(net, j.geo, 0, nb);
      EKYA_HIP(conv_fwd(dt, cg, cur, shadow_at(net, j.shadow, net.conv[0].sh_krsc), j.stem_Z,
                        ConvEpilogue(), j.ws, j.ws_floats, st, &sk));
      const long long M = (long long)nb * cg.P * cg.Q;
      void* xm = j.acts[0].X;
      if (sk.done || bn_fold_path(M, 64)) {  // the two-launch BatchNorm, then the pool
        EKYA_HIP(bn_train(net.conv[0].bn, j.stem_Z, M, nullptr, 1, j.stem_A, sk.rows));
        EKYA_HIP(maxpool_fwd(dt, j.stem_A, nb, j.geo.sh, j.geo.sw, 64, xm, j.stem_arg, st));
      } else {  // BatchNorm + ReLU applied inside the pool: stem_A is never written
        const BnL& b = net.bn[net.conv[0].bn];
        EKYA_HIP(bn_relu_maxpool_train(dt, j.stem_Z, nb, j.geo.sh, j.geo.sw, 64, j.master + b.g,
                                       j.master + b.b, j.master + b.rm, j.master + b.rv,
                                       bnp(j.bn_mean, b), bnp(j.bn_invstd, b), bnp(j.bn_scale, b),
                                       bnp(j.bn_shift, b), j.bn_ws, xm, j.stem_arg, st));
      }
      cur = xm;
      continue;
    }
    for (size_t bi = 0; bi < net.blk.size(); ++bi) {
      const BlockL& b = net.blk[bi];
      if (b.stage != s) continue;
      BlockAct& t = j.acts[bi];
      t.X = const_cast<void*>(cur);
      ConvGeom g1 = conv_geom(net, j.geo, b.c1, nb);
      const long long M = (long long)nb * g1.P * g1.Q;
      const void* res = t.X;
      int joined = -1;
      const bool side = b.cd >= 0 && two;
      if (side) {  // the block input is ready: fork before queueing the main branch
        if (fi < TrainJob::kForks / 2) return hipErrorInvalidValue;
        EKYA_HIP(hipEventRecord(j.fork[fi], st));
      }
      EKYA_HIP(conv_fwd(dt, g1, t.X, shadow_at(net, j.shadow, net.conv[b.c1].sh_krsc), t.Z1,
                        ConvEpilogue(), j.ws, j.ws_floats, st, &sk));
      const int ready1 = sk.done ? sk.rows : 0;
      if (b.cd >= 0) {  // projection shortcut: its BN output is the residual
        hipStream_t q = side ? j.st2 : st;
        if (side) EKYA_HIP(hipStreamWaitEvent(q, j.fork[fi], 0));
        EKYA_HIP(conv_fwd(dt, conv_geom(net, j.geo, b.cd, nb), t.X,
                          shadow_at(net, j.shadow, net.conv[b.cd].sh_krsc), t.Zd, ConvEpilogue(),
                          side ? j.ws2 : j.ws, side ? j.ws2_floats : j.ws_floats, q, &skd));
        EKYA_HIP(bn_train_on(net.conv[b.cd].bn, t.Zd, M, nullptr, 0, j.g[0],
                             skd.done ? skd.rows : 0, j.bn_ws2, q));
        if (side) {
          EKYA_HIP(hipEventRecord(j.joined[fi], q));
          joined = fi--;
        }
        res = j.g[0];
      }
      EKYA_HIP(bn_train(net.conv[b.c1].bn, t.Z1, M, nullptr, 1, t.A1, ready1));
      EKYA_HIP(conv_fwd(dt, conv_geom(net, j.geo, b.c2, nb), t.A1,
                        shadow_at(net, j.shadow, net.conv[b.c2].sh_krsc), t.Z2, ConvEpilogue(), j.ws,
                        j.ws_floats, st, &sk));
      if (joined >= 0) EKYA_HIP(hipStreamWaitEvent(st, j.joined[joined], 0));
      EKYA_HIP(bn_train(net.conv[b.c2].bn, t.Z2, M, res, 1, t.OUT, sk.done ? sk.rows : 0));
      cur = t.OUT;
    }
    if (s == 4)  // average pool + classifier in one kernel
      return train_head_forward(j, nb, cur);
  }
  return train_head_forward(j, nb, nullptr);
}

// Loss of the batch (labels through fid, loss / correct / flag into ce) and
// backward of stages 5..lowest; gradients land in j.grad.
static hipError_t train_backward(TrainJob& j, int nb, const int32_t* fid, float* ce) {
  const Net& net = *j.net;
  const int dt = j.dt;
  hipStream_t st = j.st;
  const float* f = (j.lowest == 5) ? reinterpret_cast<const float*>(j.x0) : j.pooled;
  void* dout = j.g[1];
  void* dnext = j.g[2];
  void* gG = j.g[3];
  void* gA = j.g[5];
  const int hw = j.geo.lh[4] * j.geo.lw[4];
  int head_ready = 0;  // rows per chunk of the last BatchNorm's backward partials in bn_ws
  if (net.hidden > 0) {
    // softmax cross-entropy, the output layer, the hidden layer's ReLU, the
    // hidden layer, then the average-pool backward
    EKYA_HIP(softmax_ce(j.logits, j.labels, fid, nb, net.n_classes, j.dz, ce, st));
    EKYA_HIP(fc_bwd(j.dz, j.hid, j.master + net.fc_w, nb, net.hidden, net.n_classes,
                    j.grad + net.fc_w, j.grad + net.fc_b, j.dhid, st));
    EKYA_HIP(relu_f32(j.dhid, j.dhid, j.hid, (long long)nb * net.hidden, st));
    EKYA_HIP(fc_bwd(j.dhid, f, j.master + net.fc1_w, nb, 512, net.hidden, j.grad + net.fc1_w,
                    j.grad + net.fc1_b, j.lowest == 5 ? nullptr : j.dpooled, st));
    if (j.lowest < 5) EKYA_HIP(avgpool_bwd(dt, j.dpooled, nb, hw, 512, dout, st));
  } else if (head_backward_fused(net.n_classes, 512)) {
    // softmax cross-entropy, classifier gradients and average-pool backward
    // (with the backward partials of the last block's output BatchNorm)
    HeadBnSink hb;
    if (j.lowest < 5) {
      const size_t lb = net.blk.size() - 1;
      hb.ymask = j.acts[lb].OUT;
      hb.z = j.acts[lb].Z2;
      hb.mean = bnp(j.bn_mean, net.bn[net.conv[net.blk[lb].c2].bn]);
      hb.part = j.bn_ws;
    }
    EKYA_HIP(head_backward(dt, j.logits, j.labels, fid, nb, net.n_classes, f, j.master + net.fc_w,
                           512, j.grad + net.fc_w, j.grad + net.fc_b,
                           j.lowest == 5 ? nullptr : dout, hw, ce, st, &hb));
    head_ready = hb.rows;
  } else {
    EKYA_HIP(softmax_ce(j.logits, j.labels, fid, nb, net.n_classes, j.dz, ce, st));
    EKYA_HIP(fc_bwd(j.dz, f, j.master + net.fc_w, nb, 512, net.n_classes, j.grad + net.fc_w,
                    j.grad + net.fc_b, j.lowest == 5 ? nullptr : j.dpooled, st));
    if (j.lowest < 5) EKYA_HIP(avgpool_bwd(dt, j.dpooled, nb, hw, 512, dout, st));
  }
  if (j.lowest == 5) return hipSuccess;
  // (ready > 0: the data gradient producing dy left the chunk statistics in
  // bn_ws, in chunks of that many rows)
  auto bn_bwd = [&](int bi, const void* dy, const void* ymask, const void* z, long long M, void* dz,
                    void* gout, int ready) {
    const BnL& b = net.bn[bi];
    return bn_backward(dt, dy, ymask, z, M, b.C, j.master + b.g, bnp(j.bn_mean, b),
                       bnp(j.bn_invstd, b), j.grad + b.g, j.grad + b.b, dz, gout, j.bn_ws, st,
                       ready);
  };
  // a BatchNorm + ReLU with no residual: its mask recomputed from z
  auto bn_bwd_relu = [&](int bi, const void* dy, const void* z, long long M, void* dz, int ready) {
    const BnL& b = net.bn[bi];
    return bn_backward(dt, dy, nullptr, z, M, b.C, j.master + b.g, bnp(j.bn_mean, b),
                       bnp(j.bn_invstd, b), j.grad + b.g, j.grad + b.b, dz, nullptr, j.bn_ws, st,
                       ready, j.master + b.b);
  };
  // statistics sink of the BatchNorm whose dy a data gradient produces
  auto sink_for = [&](int bni, const void* ymask, const void* z) {
    BnStatsSink k;
    k.part = j.bn_ws;
    k.bwd = true;
    k.ymask = ymask;
    k.z = z;
    k.mean = bnp(j.bn_mean, net.bn[bni]);
    return k;
  };
  // Weight gradients run on st2.  A fused convolution leaves its gradient as
  // split partials in ws2; its momentum step rewrites the weight copy that
  // the convolution's own data gradient (on st) reads, so when that data
  // gradient comes later the step is deferred to the next fork (or the end
  // of the pass) -- before the next weight gradient overwrites ws2.  A fork
  // is an event recorded on st that st2 waits for; every event recorded on
  // st costs st a bubble, so there is one fork per group of weight gradients
  // whose inputs are ready (a block's conv2 and shortcut, then its conv1).
  // The lowest block (no data gradient of its input) forks once more after
  // its conv2 data gradient, so that conv2's momentum step overlaps the end
  // of the pass.  st waits for st2 only before it reuses a dz buffer parity
  // (two blocks later) and at the end.  A weight gradient with no data gradient after it
  // on st (the last block, the stem) runs on st itself with st's scratch ws
  // (`main`).  With one stream (st2 == st) the same order runs serially.
  int nf = 0, nj = 0;
  int last_join[2] = {-1, -1};  // per buffer parity: join event of its last reader
  int deferred = -1, deferred_splits = 0;
  const bool two = j.st2 != st;
  auto update = [&](int ci, const float* part, int splits, hipStream_t q) {
    const ConvL& c = net.conv[ci];
    return conv_weight_update(dt, part, splits, c.cout, c.R * c.S, c.cin, j.master + c.off,
                              j.mom + c.off, j.lr, j.mu, shadow_at(net, j.shadow, c.sh_krsc),
                              shadow_at(net, j.shadow, c.sh_crsk), q);
  };
  // st2 waits for everything queued on st so far (the forward pass uses the
  // top half of the event arrays); a deferred momentum step follows on st2
  auto fork = [&]() -> hipError_t {
    if (two) {
      if (nf >= TrainJob::kForks / 2) return hipErrorInvalidValue;
      EKYA_HIP(hipEventRecord(j.fork[nf], st));
      EKYA_HIP(hipStreamWaitEvent(j.st2, j.fork[nf], 0));
      ++nf;
    }
    if (deferred >= 0) {
      EKYA_HIP(update(deferred, j.ws2, deferred_splits, j.st2));
      deferred = -1;
    }
    return hipSuccess;
  };
  // weight gradient of conv ci from x and dy (queued on st before the last
  // fork unless main); dgrad_after: its data gradient is queued on st later
  bool st2_grad = false;  // st2 wrote a weight gradient that the optimizer step reads
  auto wgrad = [&](int ci, const void* x, const void* dy, bool main,
                   bool dgrad_after) -> hipError_t {
    const ConvL& c = net.conv[ci];
    const ConvGeom cg = conv_geom(net, j.geo, ci, nb);
    hipStream_t q = main ? st : j.st2;
    float* scratch = main ? j.ws : j.ws2;
    if (!main && deferred >= 0) EKYA_HIP(fork());  // ws2 still holds the deferred partials
    if (fused_update(net, c)) {
      int splits = 0;
      EKYA_HIP(conv_wgrad_partials(dt, cg, x, dy, scratch, &splits, q, two && !main));
      if (!main && dgrad_after) {
        deferred = ci;
        deferred_splits = splits;
      } else {
        EKYA_HIP(update(ci, scratch, splits, q));
      }
    } else {
      EKYA_HIP(conv_wgrad(dt, cg, x, dy, scratch, j.grad + c.off, c.cin, q));
      if (!main && two) st2_grad = true;
    }
    return hipSuccess;
  };
  auto join = [&](int parity) -> hipError_t {  // st2 has queued every reader of this parity
    if (!two) return hipSuccess;
    if (nj >= TrainJob::kForks / 2) return hipErrorInvalidValue;
    EKYA_HIP(hipEventRecord(j.joined[nj], j.st2));
    last_join[parity] = nj++;
    return hipSuccess;
  };
  auto reuse = [&](int parity) -> hipError_t {  // st may overwrite this parity's dz buffers
    if (last_join[parity] >= 0) EKYA_HIP(hipStreamWaitEvent(st, j.joined[last_join[parity]], 0));
    last_join[parity] = -1;
    return hipSuccess;
  };
  auto dgrad = [&](int ci, const void* dy, void* dx, const void* res, int n,
                   BnStatsSink* sink) {
    return conv_dgrad(dt, conv_geom(net, j.geo, ci, n), dy,
                      shadow_at(net, j.shadow, net.conv[ci].sh_crsk), dx, res, j.ws, j.ws_floats, st,
                      sink);
  };
  int dout_ready = head_ready;  // statistics of the next block's conv2 BatchNorm are in bn_ws (chunk rows)
  int blk_count = 0;
  for (int s = 4; s >= j.lowest; --s) {
    if (s == 0) {
      // stem: max-pool backward, BN + ReLU backward, weight gradient
      const int par = blk_count & 1;
      EKYA_HIP(reuse(par));
      const long long M = (long long)nb * j.geo.sh * j.geo.sw;
      if (bn_fold_path(M, 64) || !bn_backward_pool_ok(64, j.geo.sh, j.geo.sw)) {
        EKYA_HIP(maxpool_bwd(dt, dout, j.stem_arg, nb, j.geo.sh, j.geo.sw, 64, gA, st));
        EKYA_HIP(bn_bwd_relu(net.conv[0].bn, gA, j.stem_Z, M, j.gz1[par], 0));
      } else {  // the pool's backward gathered inside the BatchNorm backward
        const BnL& b = net.bn[net.conv[0].bn];
        const ConvGeom cg = conv_geom(net, j.geo, 0, nb);
        if (stem_wgrad_pool_ok(dt, cg)) {
          // the weight gradient forms the stem's output gradient itself
          const float* coef = nullptr;
          EKYA_HIP(bn_backward_pool_stats(dt, dout, j.stem_arg, j.stem_Z, nb, j.geo.sh, j.geo.sw,
                                          64, j.master + b.g, j.master + b.b, bnp(j.bn_mean, b),
                                          bnp(j.bn_invstd, b), j.grad + b.g, j.grad + b.b,
                                          j.bn_ws, &coef, st));
          EKYA_HIP(conv_wgrad_stem_pool(cg, j.x0, j.stem_Z, dout, j.stem_arg, bnp(j.bn_mean, b),
                                        coef, j.master + b.g, bnp(j.bn_invstd, b),
                                        j.master + b.b, j.ws, j.grad + net.conv[0].off, st));
          break;
        }
        EKYA_HIP(bn_backward_pool(dt, dout, j.stem_arg, j.stem_Z, nb, j.geo.sh, j.geo.sw, 64,
                                  j.master + b.g, j.master + b.b, bnp(j.bn_mean, b),
                                  bnp(j.bn_invstd, b), j.grad + b.g, j.grad + b.b, j.gz1[par],
                                  j.bn_ws, st));
      }
      EKYA_HIP(wgrad(0, j.x0, j.gz1[par], true, false));
      break;
    }
    int first_bi = -1;
    for (size_t bi = 0; bi < net.blk.size(); ++bi)
      if (net.blk[bi].stage == s && first_bi < 0) first_bi = (int)bi;
    for (int bi = (int)net.blk.size() - 1; bi >= 0; --bi) {
      const BlockL& b = net.blk[bi];
      if (b.stage != s) continue;
      BlockAct& t = j.acts[bi];
      const int par = blk_count++ & 1;
      EKYA_HIP(reuse(par));
      void* gZ2 = j.gz2[par];
      void* gZ1 = j.gz1[par];
      void* gZd = j.gzd[par];
      const bool need_dx = !(s == j.lowest && bi == first_bi);
      ConvGeom g1 = conv_geom(net, j.geo, b.c1, nb);
      const long long M = (long long)nb * g1.P * g1.Q;
      // g = dOut * [OUT > 0]; BN2 backward (and the shortcut's BN backward)
      EKYA_HIP(bn_bwd(net.conv[b.c2].bn, dout, t.OUT, t.Z2, M, gZ2, gG, dout_ready));
      dout_ready = 0;
      if (b.cd >= 0) EKYA_HIP(bn_bwd(net.conv[b.cd].bn, gG, nullptr, t.Zd, M, gZd, nullptr, 0));
      // After each fork the data-gradient work is queued on st before the
      // weight-gradient work on st2, so the critical chain is dispatched first.
      EKYA_HIP(fork());
      // a projection shortcut beside a stride-2 conv1: its data gradient is
      // folded into conv1's (no full-size partial gradient in between),
      // unless conv1's data gradient has to leave the next block's
      // BatchNorm statistics (the small-batch path)
      const bool next_sink = bi > 0 && net.blk[bi - 1].stage >= j.lowest;
      const ConvGeom gd = b.cd >= 0 ? conv_geom(net, j.geo, b.cd, nb) : g1;
      const bool fold_sc = b.cd >= 0 && need_dx && conv_dgrad_s2_shortcut_ok(dt, g1, gd) &&
                           !(next_sink && bn_fold_path((long long)nb * g1.H * g1.W, g1.C));
      const void* dx_sc = gG;
      if (b.cd >= 0 && need_dx && !fold_sc) EKYA_HIP(dgrad(b.cd, gZd, dnext, nullptr, nb, nullptr));
      if (b.cd >= 0) dx_sc = dnext;
      BnStatsSink sk1 = sink_for(net.conv[b.c1].bn, t.A1, t.Z1);
      EKYA_HIP(dgrad(b.c2, gZ2, gA, nullptr, nb, &sk1));
      if (b.cd >= 0 && !fold_sc) EKYA_HIP(wgrad(b.cd, t.X, gZd, false, need_dx));
      EKYA_HIP(wgrad(b.c2, t.A1, gZ2, false, true));
      // conv1's BatchNorm + ReLU has no residual: its ReLU mask is recomputed
      // from Z1 (exactly the stored A1 > 0) instead of reading A1, unless the
      // statistics were already taken with A1 in conv2's data gradient
      if (sk1.done)
        EKYA_HIP(bn_bwd(net.conv[b.c1].bn, gA, t.A1, t.Z1, M, gZ1, nullptr, sk1.rows));
      else
        EKYA_HIP(bn_bwd_relu(net.conv[b.c1].bn, gA, t.Z1, M, gZ1, 0));
      if (need_dx) {
        EKYA_HIP(fork());
        // dOut of the block processed next (bi - 1): its conv2 BatchNorm's statistics
        BnStatsSink skn;
        BnStatsSink* psk = nullptr;
        if (next_sink) {
          const BlockL& nbk = net.blk[bi - 1];
          skn = sink_for(net.conv[nbk.c2].bn, j.acts[bi - 1].OUT, j.acts[bi - 1].Z2);
          psk = &skn;
        }
        if (fold_sc) {
          EKYA_HIP(conv_dgrad_s2_shortcut(g1, gZ1, shadow_at(net, j.shadow, net.conv[b.c1].sh_crsk),
                                          gd, gZd, shadow_at(net, j.shadow, net.conv[b.cd].sh_crsk),
                                          dnext, j.ws, j.ws_floats, st));
          // the shortcut's weights are read up to here: its weight gradient
          // and momentum step go on st2 only after a fork behind that launch
          EKYA_HIP(fork());
          EKYA_HIP(wgrad(b.cd, t.X, gZd, false, false));
        } else {
          EKYA_HIP(dgrad(b.c1, gZ1, dnext, dx_sc, nb, psk));
        }
        dout_ready = (psk && psk->done) ? psk->rows : 0;
      } else if (deferred >= 0) {
        // no later work on st reads the conv2 weights: the deferred momentum
        // step runs on st2 beside this block's remaining work on st
        EKYA_HIP(fork());
      }
      EKYA_HIP(wgrad(b.c1, t.X, gZ1, !need_dx, need_dx));
      EKYA_HIP(join(par));
      if (need_dx) std::swap(dout, dnext);
    }
  }
  // The end join.  st waits for it here when what follows on st needs st2's
  // results (a still-deferred momentum step, or a weight gradient for the
  // optimizer step); otherwise st runs the optimizer step of the remaining
  // parameters first and waits in settle() before anything that reads the
  // convolution weights or buffers st2 read.
  if (two) {
    if (nj >= TrainJob::kForks / 2) return hipErrorInvalidValue;
    EKYA_HIP(hipEventRecord(j.joined[nj], j.st2));
    if (deferred >= 0 || st2_grad)
      EKYA_HIP(hipStreamWaitEvent(st, j.joined[nj], 0));
    else
      j.pending_join = nj;
    ++nj;
  }
  if (deferred >= 0) EKYA_HIP(update(deferred, j.ws2, deferred_splits, st));
  return hipSuccess;
}

// st waits for the pending end-of-backward join, if any.
static hipError_t settle(TrainJob& j) {
  if (j.pending_join >= 0) EKYA_HIP(hipStreamWaitEvent(j.st, j.joined[j.pending_join], 0));
  j.pending_join = -1;
  return hipSuccess;
}

// Fill the feature cache rows [row0, row0 + n) from frames (optionally
// through idx), chunk by chunk.
static hipError_t build_cache(const Net& net, const Geo& g, const void* shadow, const float* fold,
                              const float* master, int lowest, const void* frames,
                              const int32_t* d_idx, int n, void* cache, long long row_bytes,
                              long long row0, void* padded, int cap, EvalBufs& eb,
                              hipStream_t st) {
  const size_t es = dtype_size(net.dt);
  const long long fbytes = (long long)g.H * g.W * 3 * es;
  // equal chunks of at most cap frames (600 frames: 2 x 300, not 512 + 88,
  // whose short tail costs the big-tile convolutions a nearly empty round)
  const int per = n > 0 ? cdiv(n, cdiv(n, cap)) : cap;
  for (int i0 = 0; i0 < n; i0 += per) {
    const int cnt = std::min(per, n - i0);
    const void* src = d_idx ? frames : reinterpret_cast<const char*>(frames) + i0 * fbytes;
    void* out = reinterpret_cast<char*>(cache) + (row0 + i0) * row_bytes;
    if (stem_frames_ok(net.dt, conv_geom(net, g, 0, cnt))) {  // the stem reads the frames
      EKYA_HIP(eval_forward(net, g, shadow, fold, master, 0, lowest - 1, src, cnt, eb, out, st,
                            true, d_idx ? d_idx + i0 : nullptr));
      continue;
    }
    EKYA_HIP(frames_to_padded(net.dt, src, d_idx ? d_idx + i0 : nullptr, cnt, g.H, g.W,
                              net.conv[0].cin_pad, padded, st));
    EKYA_HIP(eval_forward(net, g, shadow, fold, master, 0, lowest - 1, padded, cnt, eb, out, st));
  }
  return hipSuccess;
}

// Initial device state of a job: internal-layout master weights, zeroed
// gradients/momentum, folded eval BatchNorm, low-precision weight copies.
static hipError_t job_setup(TrainJob& j) {
  const Net& net = *j.net;
  const Tables& t = *j.tabs;
  EKYA_HIP(permute_weights(j.weights, j.master, t.permute, t.n_permute, net.total, 1, j.st));
  EKYA_HIP(hipMemsetAsync(j.grad, 0, net.total * sizeof(float), j.st));
  EKYA_HIP(hipMemsetAsync(j.mom, 0, net.total * sizeof(float), j.st));
  EKYA_HIP(hipMemsetAsync(j.hcount, 0, j.epochs * sizeof(int32_t), j.st));
  EKYA_HIP(bn_fold(j.master, t.fold_all, t.n_fold_all, j.fold, j.st));
  EKYA_HIP(pack_conv_weights(j.dt, j.master, t.pack_frozen[j.lowest], t.n_pack_frozen[j.lowest],
                             j.shadow, j.st));
  EKYA_HIP(pack_conv_weights(j.dt, j.master, t.pack_train[j.lowest], t.n_pack_train[j.lowest],
                             j.shadow, j.st));
  EKYA_HIP(hipMemcpyAsync(j.d_order, j.h_order.data(), j.h_order.size() * sizeof(int32_t),
                          hipMemcpyHostToDevice, j.st));
  EKYA_HIP(hipMemcpyAsync(j.d_fidx, j.h_fidx.data(), j.h_fidx.size() * sizeof(int32_t),
                          hipMemcpyHostToDevice, j.st));
  return hipSuccess;
}

// The epoch loop (after setup and cache build); records an event per epoch.
static hipError_t job_epochs(TrainJob& j) {
  const Net& net = *j.net;
  const Tables& t = *j.tabs;
  const size_t es = dtype_size(j.dt);
  const long long fbytes = (long long)j.geo.H * j.geo.W * 3 * es;
  int step = 0;
  EKYA_HIP(hipEventRecord(j.ev[0], j.st));
  for (int e = 0; e < j.epochs; ++e) {
    for (int b0 = 0; b0 < j.n_s; b0 += j.B) {
      const int nb = std::min(j.B, j.n_s - b0);
      const int32_t* ord = j.d_order + (size_t)e * j.n_s + b0;
      const int32_t* fid = j.d_fidx + (size_t)e * j.n_s + b0;
      EKYA_HIP(settle(j));  // the gather overwrites the input st2 read
      if (j.lowest == 0)
        EKYA_HIP(frames_to_padded(j.dt, j.frames, fid, nb, j.geo.H, j.geo.W, net.conv[0].cin_pad,
                                  j.x0, j.st));
      else
        EKYA_HIP(gather_rows(j.cache, ord, nb, j.row_bytes, j.x0, j.st));
      EKYA_HIP(train_forward(j, nb));
      EKYA_HIP(train_backward(j, nb, fid, j.ce_out + 3 * step));
      // the parameters without a fused update (BatchNorm, classifier, and
      // convolutions outside conv_weight_update's reach)
      EKYA_HIP(sgd_momentum_ranges(j.master, j.mom, j.grad, t.sgd_rest[j.lowest],
                                   t.n_sgd_rest[j.lowest], t.sgd_rest_max[j.lowest], j.lr, j.mu,
                                   j.st));
      EKYA_HIP(pack_conv_weights(j.dt, j.master, t.pack_rest[j.lowest], t.n_pack_rest[j.lowest],
                                 j.shadow, j.st));
      ++step;
    }
    EKYA_HIP(settle(j));
    EKYA_HIP(hipEventRecord(j.ev_tr[e], j.st));
    // the previous evaluation still reads the folded BatchNorm and its buffers
    if (j.eval_pending) EKYA_HIP(hipStreamWaitEvent(j.st, j.ev_eval_done, 0));
    j.eval_pending = false;
    // held-out accuracy in eval mode with the current running statistics
    EKYA_HIP(bn_fold(j.master, t.fold_train[j.lowest], t.n_fold_train[j.lowest], j.fold, j.st));
    if (j.ckpt && ((e + 1) % j.ckpt_every == 0 || e + 1 == j.epochs))
      EKYA_HIP(model_load(*j.ckpt, nullptr, j.master, j.st, nullptr));
    hipStream_t qe = j.st;
    const void* esh = j.shadow;
    const float* ems = j.master;
    if (j.st3 && j.n_h > 0) {  // on st3 from this epoch's weights, beside the next epoch
      EKYA_HIP(hipMemcpyAsync(j.shadow_snap, j.shadow, net.shadow_elems * es,
                              hipMemcpyDeviceToDevice, j.st));
      EKYA_HIP(hipMemcpyAsync(j.master_snap, j.master, net.total * sizeof(float),
                              hipMemcpyDeviceToDevice, j.st));
      EKYA_HIP(hipEventRecord(j.ev_eval_fork, j.st));
      EKYA_HIP(hipStreamWaitEvent(j.st3, j.ev_eval_fork, 0));
      qe = j.st3;
      esh = j.shadow_snap;
      ems = j.master_snap;
    }
    EKYA_HIP(hipEventRecord(j.ev_e0[e], qe));
    for (int h0 = 0; h0 < j.n_h; h0 += j.eval_cap) {
      const int cnt = std::min(j.eval_cap, j.n_h - h0);
      const void* in;
      if (j.lowest == 0) {
        EKYA_HIP(frames_to_padded(j.dt, reinterpret_cast<const char*>(j.hframes) + h0 * fbytes,
                                  nullptr, cnt, j.geo.H, j.geo.W, net.conv[0].cin_pad, j.eval_in,
                                  qe));
        in = j.eval_in;
      } else {
        in = reinterpret_cast<const char*>(j.hcache) + (long long)h0 * j.row_bytes;
      }
      EKYA_HIP(eval_forward(net, j.geo, esh, j.fold, ems, j.lowest, 5, in, cnt, j.eval,
                            j.eval.logits, qe));
      EKYA_HIP(count_correct(j.eval.logits, j.hlabels + h0, cnt, net.n_classes, j.hcount + e,
                             qe));
    }
    EKYA_HIP(hipEventRecord(j.ev_e1[e], qe));
    if (qe != j.st) {
      EKYA_HIP(hipEventRecord(j.ev_eval_done, qe));
      j.eval_pending = true;
    }
    EKYA_HIP(hipEventRecord(j.ev[e + 1], j.st));
  }
  if (j.eval_pending) EKYA_HIP(hipStreamWaitEvent(j.st, j.ev_eval_done, 0));
  j.eval_pending = false;
  return hipSuccess;
}

static void job_prepare_host(TrainJob& j, const std::vector<int32_t>& S, uint64_t shuffle_seed) {
  j.h_order.resize((size_t)j.epochs * j.n_s);
  j.h_fidx.resize((size_t)j.epochs * j.n_s);
  for (int e = 0; e < j.epochs; ++e) {
    std::vector<int32_t> o = epoch_order(j.n_s, shuffle_seed, e);
    for (int i = 0; i < j.n_s; ++i) {
      j.h_order[(size_t)e * j.n_s + i] = o[i];
      j.h_fidx[(size_t)e * j.n_s + i] = S[o[i]];
    }
  }
  j.n_steps = j.epochs * ((j.n_s + j.B - 1) / j.B);
}

struct JobResult {
  std::vector<float> ce;       // n_steps x 3
  std::vector<int32_t> hc;     // epochs
  std::vector<float> secs;     // epochs: training steps
  std::vector<float> esecs;    // epochs: held-out evaluation
  ekya_status status = EKYA_OK;
};

static hipError_t job_collect(TrainJob& j, JobResult& r) {
  r.ce.resize((size_t)j.n_steps * 3);
  r.hc.resize(j.epochs);
  r.secs.resize(j.epochs);
  r.esecs.resize(j.epochs);
  EKYA_HIP(hipMemcpyAsync(r.ce.data(), j.ce_out, r.ce.size() * sizeof(float), hipMemcpyDeviceToHost,
                          j.st));
  EKYA_HIP(hipMemcpyAsync(r.hc.data(), j.hcount, r.hc.size() * sizeof(int32_t),
                          hipMemcpyDeviceToHost, j.st));
  EKYA_HIP(hipStreamSynchronize(j.st));
  for (int e = 0; e < j.epochs; ++e) {
    float ms = 0.f;
    EKYA_HIP(hipEventElapsedTime(&ms, j.ev[e], j.ev_tr[e]));
    r.secs[e] = ms * 1e-3f;
    ms = 0.f;
    if (j.n_h > 0) EKYA_HIP(hipEventElapsedTime(&ms, j.ev_e0[e], j.ev_e1[e]));
    r.esecs[e] = ms * 1e-3f;
  }
  r.status = EKYA_OK;
  for (int s = 0; s < j.n_steps; ++s)
    if (r.ce[3 * s + 2] != 0.f || !std::isfinite(r.ce[3 * s])) {
      r.status = EKYA_ERR_NONFINITE;
      break;
    }
  return hipSuccess;
}

// Every event here orders work between streams of this device (or times it);
// the host reads results only after a stream synchronisation.  Without the
// system-scope fence a recorded event costs its stream a shorter bubble.
static hipError_t create_events(TrainJob& j) {
  for (int e = 0; e <= j.epochs; ++e)
    EKYA_HIP(hipEventCreateWithFlags(&j.ev[e], hipEventDisableSystemFence));
  for (int e = 0; e < j.epochs; ++e) {
    EKYA_HIP(hipEventCreateWithFlags(&j.ev_tr[e], hipEventDisableSystemFence));
    EKYA_HIP(hipEventCreateWithFlags(&j.ev_e0[e], hipEventDisableSystemFence));
    EKYA_HIP(hipEventCreateWithFlags(&j.ev_e1[e], hipEventDisableSystemFence));
  }
  if (j.st3) {
    EKYA_HIP(hipEventCreateWithFlags(&j.ev_eval_fork, hipEventDisableTiming | hipEventDisableSystemFence));
    EKYA_HIP(hipEventCreateWithFlags(&j.ev_eval_done, hipEventDisableTiming | hipEventDisableSystemFence));
  }
  for (int i = 0; i < TrainJob::kForks; ++i) {
    EKYA_HIP(hipEventCreateWithFlags(&j.fork[i], hipEventDisableTiming | hipEventDisableSystemFence));
    EKYA_HIP(
        hipEventCreateWithFlags(&j.joined[i], hipEventDisableTiming | hipEventDisableSystemFence));
  }
  return hipSuccess;
}
static void destroy_events(TrainJob& j) {
  if (j.ev_eval_fork) (void)hipEventDestroy(j.ev_eval_fork);
  if (j.ev_eval_done) (void)hipEventDestroy(j.ev_eval_done);
  j.ev_eval_fork = j.ev_eval_done = nullptr;
  for (int e = 0; e <= EKYA_MAX_EPOCHS; ++e)
    if (j.ev[e]) {
      (void)hipEventDestroy(j.ev[e]);
      j.ev[e] = nullptr;
    }
  for (hipEvent_t* a : {j.ev_tr, j.ev_e0, j.ev_e1})
    for (int e = 0; e < EKYA_MAX_EPOCHS; ++e)
      if (a[e]) {
        (void)hipEventDestroy(a[e]);
        a[e] = nullptr;
      }
  for (int i = 0; i < TrainJob::kForks; ++i) {
    if (j.fork[i]) (void)hipEventDestroy(j.fork[i]);
    if (j.joined[i]) (void)hipEventDestroy(j.joined[i]);
    j.fork[i] = j.joined[i] = nullptr;
  }
}

#define EKYA_CHECK_HIP(expr)                                   \
  do {                                                         \
    hipError_t e_ = (expr);                                    \
    if (e_ != hipSuccess) {                                    \
      c.err = std::string("HIP error: ") + hipGetErrorString(e_); \
      return e_ == hipErrorOutOfMemory ? EKYA_ERR_NOMEM : EKYA_ERR_HIP; \
    }                                                          \
  } while (0)

// --------------------------------------------------------------- retrain
struct TimerGuard {
  explicit TimerGuard(Ctx& c) { set_thread_timer(c.timing ? &c.timer : nullptr); }
  ~TimerGuard() { set_thread_timer(nullptr); }
};

// Retraining job shape from the call's arguments (host only).
static void config_retrain(TrainJob& j, const Net& net, int k, int n_frames, int H, int W,
                           int n_heldout, const ekya_train_opts& o, bool eval_overlap) {
  j.net = &net;
  j.geo = Geo::build(net, H, W);
  j.dt = o.precision;
  j.k = k;
  j.lowest = 6 - k;
  j.B = o.batch;
  j.epochs = o.epochs;
  j.lr = o.lr;
  j.mu = o.momentum;
  j.n_h = n_heldout;
  j.n_s = subset_count(n_frames, o.subsample_frac);
  j.n_steps = j.epochs * cdiv(j.n_s, j.B);
  j.eval_overlap = eval_overlap;
  const long long feat = j.geo.stage_in_elems(net, j.lowest);
  j.row_bytes = feat * ((j.lowest == 5) ? 4 : (long long)dtype_size(j.dt));
}

// Frames per chunk of a frozen-prefix cache build.
static constexpr int kCacheChunk = 512;

struct RetrainBufs {
  void* cache = nullptr;  // training rows, then held-out rows
  int32_t* d_S = nullptr;
  void* padded = nullptr;
  EvalBufs ceb;
};

// Job buffers, the feature cache and its build scratch.
static void plan_retrain(Arena& a, TrainJob& j, RetrainBufs& r) {
  const Net& net = *j.net;
  plan_job(a, j);
  r = RetrainBufs();
  if (j.lowest >= 1) {
    r.cache = a.take_bytes((size_t)(j.n_s + j.n_h) * j.row_bytes);
    r.d_S = a.take<int32_t>(j.n_s);
    r.padded = a.take_bytes((size_t)kCacheChunk * j.geo.H * j.geo.W * net.conv[0].cin_pad *
                            dtype_size(j.dt));
    plan_eval(a, net, j.geo, 0, j.lowest - 1, kCacheChunk, r.ceb);
  }
}

size_t retrain_workspace_bytes(const Net& net, int k, int n_frames, int H, int W, int n_heldout,
                               const ekya_train_opts& o) {
  TrainJob j;
  config_retrain(j, net, k, n_frames, H, W, n_heldout, o, true);
  RetrainBufs r;
  Arena a;
  plan_retrain(a, j, r);
  return a.used;
}

ekya_status run_retrain(Ctx& c, float* weights, int k, const void* frames, const int32_t* labels,
                        int n_frames, int H, int W, const void* hframes, const int32_t* hlabels,
                        int n_heldout, const ekya_train_opts& o, ekya_retrain_result* res,
                        hipStream_t stream) {
  EKYA_CHECK_HIP(hipSetDevice(c.device));
  TimerGuard tg(c);
  const int dt = o.precision;
  const Net& net = c.net[dt];
  TrainJob j;
  // per-kernel timing runs serially, so each timed kernel runs alone; otherwise
  // each epoch's held-out evaluation overlaps the next epoch on st3
  config_retrain(j, net, k, n_frames, H, W, n_heldout, o, !c.timing);
  RetrainBufs rb;
  {
    Arena meas;
    plan_retrain(meas, j, rb);
    if (ekya_status s = acquire_workspace(c, meas.used, stream)) return s;
  }
  j.tabs = &c.tabs[dt];
  j.st = stream;
  // library-owned side streams (default priority): weight gradients, held-out evaluation
  if (c.streams.empty()) {
    hipStream_t s2;
    EKYA_CHECK_HIP(ctx_stream(c, &s2));
    c.streams.push_back(s2);
  }
  j.st2 = c.timing ? stream : c.streams[0];
  if (j.eval_overlap) {
    if (!c.eval_stream) EKYA_CHECK_HIP(ctx_stream(c, &c.eval_stream));
    j.st3 = c.eval_stream;
  }
  j.ckpt = c.ckpt;
  j.ckpt_every = c.ckpt_every;
  j.weights = weights;
  j.frames = frames;
  j.labels = labels;
  j.hframes = hframes;
  j.hlabels = hlabels;
  std::vector<int32_t> S = training_subset(n_frames, o.subsample_frac, o.seed);
  job_prepare_host(j, S, o.seed);
  Arena real;
  real.base = reinterpret_cast<char*>(c.ws.p);
  plan_retrain(real, j, rb);
  void* cache = rb.cache;
  int32_t* d_S = rb.d_S;
  void* padded = rb.padded;
  EvalBufs& ceb = rb.ceb;
  const int ccap = kCacheChunk;
  j.cache = cache;
  j.hcache = cache ? reinterpret_cast<char*>(cache) + (long long)j.n_s * j.row_bytes : nullptr;

  EKYA_CHECK_HIP(create_events(j));
  hipEvent_t p0 = nullptr, p1 = nullptr;
  EKYA_CHECK_HIP(hipEventCreateWithFlags(&p0, hipEventDisableSystemFence));
  EKYA_CHECK_HIP(hipEventCreateWithFlags(&p1, hipEventDisableSystemFence));
  auto run = [&]() -> hipError_t {
    EKYA_HIP(job_setup(j));
    EKYA_HIP(hipEventRecord(p0, stream));
    if (j.lowest >= 1) {
      EKYA_HIP(hipMemcpyAsync(d_S, S.data(), S.size() * sizeof(int32_t), hipMemcpyHostToDevice,
                              stream));
      EKYA_HIP(build_cache(net, j.geo, j.shadow, j.fold, j.master, j.lowest, frames, d_S, j.n_s,
                           cache, j.row_bytes, 0, padded, ccap, ceb, stream));
      EKYA_HIP(build_cache(net, j.geo, j.shadow, j.fold, j.master, j.lowest, hframes, nullptr,
                           j.n_h, cache, j.row_bytes, j.n_s, padded, ccap, ceb, stream));
    }
    EKYA_HIP(hipEventRecord(p1, stream));
    EKYA_HIP(job_epochs(j));
    // write back: internal -> canonical (frozen parts round-trip exactly)
    EKYA_HIP(permute_weights(j.master, weights, c.tabs[dt].permute, c.tabs[dt].n_permute,
                             net.total, 0, stream));
    return hipSuccess;
  };
  hipError_t he = run();
  (void)hipEventRecord(c.last_done, stream);  // after whatever was queued
  JobResult r;
  if (he == hipSuccess) he = job_collect(j, r);
  float pms = 0.f;
  if (he == hipSuccess) he = hipEventElapsedTime(&pms, p0, p1);
  destroy_events(j);
  (void)hipEventDestroy(p0);
  (void)hipEventDestroy(p1);
  EKYA_CHECK_HIP(he);

  res->n_train = j.n_s;
  res->n_epochs = j.epochs;
  res->n_steps = j.n_steps;
  res->prefix_seconds = pms * 1e-3f;
  const int spe = (j.n_s + j.B - 1) / j.B;
  for (int e = 0; e < j.epochs; ++e) {
    res->heldout_acc[e] = j.n_h ? (float)r.hc[e] / (float)j.n_h : 0.f;
    res->epoch_seconds[e] = r.secs[e];
    res->eval_seconds[e] = r.esecs[e];
    double l = 0.0;
    for (int s = 0; s < spe; ++s) l += r.ce[3 * (e * spe + s)];
    res->epoch_loss[e] = (float)(l / spe);
  }
  res->heldout_acc_final = res->heldout_acc[j.epochs - 1];
  if (res->step_loss)
    for (int s = 0; s < std::min(j.n_steps, res->step_loss_capacity); ++s)
      res->step_loss[s] = r.ce[3 * s];
  if (r.status != EKYA_OK) c.err = "training loss is not finite";
  return r.status;
}

// --------------------------------------------------------------- profile
// A frozen-prefix feature cache shared by the candidates of one depth.
struct CacheInfo {
  int lowest;
  int n_rows_s;  // training rows (prefix of the shared draw) held
  long long row_bytes;
  void* p;
};

struct ProfilePlan {
  std::vector<TrainJob> jobs;
  std::vector<CacheInfo> caches;
  int n_max = 0;  // frames of the shared draw
  int32_t* d_S = nullptr;
  void* padded = nullptr;
  EvalBufs ceb;
  float *pmaster = nullptr, *pfold = nullptr;
  void* pshadow = nullptr;
};

// Candidate jobs and per-depth caches from the call's arguments (host only).
static void config_profile(ProfilePlan& pp, const Net& net, const ekya_profile_cfg* cfgs, int n_cfgs,
                           int n_frames, int H, int W, int n_heldout) {
  const Geo geo = Geo::build(net, H, W);
  const size_t es = dtype_size(net.dt);
  pp.n_max = 0;
  for (int i = 0; i < n_cfgs; ++i)
    pp.n_max = std::max(pp.n_max, subset_count(n_frames, cfgs[i].subsample_frac));
  pp.caches.clear();
  for (int i = 0; i < n_cfgs; ++i) {
    const int lo = 6 - cfgs[i].k_trainable;
    if (lo == 0) continue;
    const int ns = subset_count(n_frames, cfgs[i].subsample_frac);
    bool found = false;
    for (auto& ci : pp.caches)
      if (ci.lowest == lo) {
        ci.n_rows_s = std::max(ci.n_rows_s, ns);
        found = true;
      }
    if (!found)
      pp.caches.push_back({lo, ns, geo.stage_in_elems(net, lo) * (long long)((lo == 5) ? 4 : es), nullptr});
  }
  pp.jobs.assign(n_cfgs, TrainJob());
  for (int i = 0; i < n_cfgs; ++i) {
    TrainJob& j = pp.jobs[i];
    const ekya_profile_cfg& cf = cfgs[i];
    j.net = &net;
    j.geo = geo;
    j.dt = net.dt;
    j.k = cf.k_trainable;
    j.lowest = 6 - cf.k_trainable;
    j.B = cf.batch;
    j.epochs = cf.epochs;
    j.lr = cf.lr;
    j.mu = cf.momentum;
    j.n_h = n_heldout;
    j.n_s = subset_count(n_frames, cf.subsample_frac);
    j.n_steps = j.epochs * cdiv(j.n_s, j.B);
  }
}

static void plan_profile(Arena& a, ProfilePlan& pp, int n_heldout, int H, int W) {
  const Net& net = *pp.jobs[0].net;
  const Geo& geo = pp.jobs[0].geo;
  const size_t es = dtype_size(net.dt);
  for (auto& j : pp.jobs) plan_job(a, j);
  for (auto& ci : pp.caches) ci.p = a.take_bytes((size_t)(ci.n_rows_s + n_heldout) * ci.row_bytes);
  pp.d_S = a.take<int32_t>(std::max(1, pp.n_max));
  pp.padded = a.take_bytes((size_t)kCacheChunk * H * W * net.conv[0].cin_pad * es);
  plan_eval(a, net, geo, 0, 4, kCacheChunk, pp.ceb);
  pp.pmaster = a.take<float>(net.total);
  pp.pfold = a.take<float>(2 * net.bn_channels);
  pp.pshadow = a.take_bytes(net.shadow_elems * es);
}

size_t profile_workspace_bytes(const Net& net, const ekya_profile_cfg* cfgs, int n_cfgs,
                               int n_frames, int H, int W, int n_heldout) {
  ProfilePlan pp;
  config_profile(pp, net, cfgs, n_cfgs, n_frames, H, W, n_heldout);
  Arena a;
  plan_profile(a, pp, n_heldout, H, W);
  return a.used;
}

ekya_status run_profile(Ctx& c, const float* weights, const ekya_profile_cfg* cfgs, int n_cfgs,
                        const void* frames, const int32_t* labels, int n_frames, int H, int W,
                        const void* hframes, const int32_t* hlabels, int n_heldout,
                        uint64_t subsample_seed, int precision, int concurrent,
                        ekya_profile_result* out) {
  EKYA_CHECK_HIP(hipSetDevice(c.device));
  const int dt = precision;
  const Net& net = c.net[dt];
  const Geo geo = Geo::build(net, H, W);
  ProfilePlan pp;
  config_profile(pp, net, cfgs, n_cfgs, n_frames, H, W, n_heldout);
  // streams: per candidate a main and a side stream, plus one for the caches
  while ((int)c.streams.size() < 2 * n_cfgs + 1) {
    hipStream_t s;
    EKYA_CHECK_HIP(ctx_stream(c, &s));
    c.streams.push_back(s);
  }
  hipStream_t s0 = c.streams[n_cfgs];
  {
    Arena meas;
    plan_profile(meas, pp, n_heldout, H, W);
    if (ekya_status s = acquire_workspace(c, meas.used, s0)) return s;
  }
  // one shared draw; each candidate uses a prefix of it
  const int n_max = pp.n_max;
  const std::vector<int32_t> S = partial_shuffle(n_frames, n_max, subsample_seed);
  std::vector<TrainJob>& jobs = pp.jobs;
  std::vector<CacheInfo>& caches = pp.caches;
  for (int i = 0; i < n_cfgs; ++i) {
    TrainJob& j = jobs[i];
    j.tabs = &c.tabs[dt];
    j.st = c.streams[i];
    j.st2 = c.timing ? j.st : c.streams[n_cfgs + 1 + i];
    j.weights = weights;
    j.frames = frames;
    j.labels = labels;
    j.hframes = hframes;
    j.hlabels = hlabels;
    std::vector<int32_t> Si(S.begin(), S.begin() + j.n_s);
    job_prepare_host(j, Si, cfgs[i].shuffle_seed);
  }
  const int ccap = kCacheChunk;
  Arena real;
  real.base = reinterpret_cast<char*>(c.ws.p);
  plan_profile(real, pp, n_heldout, H, W);
  int32_t* d_S = pp.d_S;
  void* padded = pp.padded;
  EvalBufs& ceb = pp.ceb;
  float* pmaster = pp.pmaster;
  float* pfold = pp.pfold;
  void* pshadow = pp.pshadow;

  // caches: the frozen prefix of the starting weights, built once per depth on s0
  const Tables& t = c.tabs[dt];
  auto build = [&]() -> hipError_t {
    EKYA_HIP(permute_weights(weights, pmaster, t.permute, t.n_permute, net.total, 1, s0));
    EKYA_HIP(bn_fold(pmaster, t.fold_all, t.n_fold_all, pfold, s0));
    EKYA_HIP(pack_conv_weights(dt, pmaster, t.pack_all, t.n_pack_all, pshadow, s0));
    if (!caches.empty())
      EKYA_HIP(hipMemcpyAsync(d_S, S.data(), S.size() * sizeof(int32_t), hipMemcpyHostToDevice, s0));
    for (auto& ci : caches) {
      EKYA_HIP(build_cache(net, geo, pshadow, pfold, pmaster, ci.lowest, frames, d_S, ci.n_rows_s,
                           ci.p, ci.row_bytes, 0, padded, ccap, ceb, s0));
      EKYA_HIP(build_cache(net, geo, pshadow, pfold, pmaster, ci.lowest, hframes, nullptr,
                           n_heldout, ci.p, ci.row_bytes, ci.n_rows_s, padded, ccap, ceb, s0));
    }
    return hipSuccess;
  };
  hipError_t he = build();
  if (he == hipSuccess) he = hipStreamSynchronize(s0);
  // held-out rows of a depth's cache sit after its n_rows_s training rows
  for (int i = 0; i < n_cfgs && he == hipSuccess; ++i) {
    TrainJob& j = jobs[i];
    for (auto& ci : caches)
      if (ci.lowest == j.lowest) {
        j.cache = ci.p;
        j.row_bytes = ci.row_bytes;
        j.hcache = reinterpret_cast<char*>(ci.p) + (long long)ci.n_rows_s * ci.row_bytes;
      }
  }
  std::vector<hipError_t> errs(n_cfgs, hipSuccess);
  auto run_job = [&](int i) {
    TrainJob& j = jobs[i];
    hipError_t e = create_events(j);
    if (e == hipSuccess) e = job_setup(j);
    if (e == hipSuccess) e = job_epochs(j);
    errs[i] = e;
  };
  if (he == hipSuccess) {
    if (concurrent) {
      std::vector<std::thread> th;
      for (int i = 0; i < n_cfgs; ++i) th.emplace_back([&, i]() {
        (void)hipSetDevice(c.device);
        run_job(i);
      });
      for (auto& x : th) x.join();
    } else {
      for (int i = 0; i < n_cfgs; ++i) {
        run_job(i);
        if (errs[i] == hipSuccess) errs[i] = hipStreamSynchronize(jobs[i].st);
      }
    }
  }
  ekya_status overall = EKYA_OK;
  for (int i = 0; i < n_cfgs; ++i) {
    TrainJob& j = jobs[i];
    ekya_profile_result& o = out[i];
    std::memset(&o, 0, sizeof(o));
    hipError_t e = (he != hipSuccess) ? he : errs[i];
    JobResult r;
    if (e == hipSuccess) e = job_collect(j, r);
    if (e != hipSuccess) {
      o.status = (e == hipErrorOutOfMemory) ? EKYA_ERR_NOMEM : EKYA_ERR_HIP;
      c.err = std::string("HIP error: ") + hipGetErrorString(e);
      overall = (ekya_status)o.status;
    } else {
      o.status = r.status;
      o.n_train = j.n_s;
      const int spe = (j.n_s + j.B - 1) / j.B;
      for (int ep = 0; ep < j.epochs; ++ep) {
        o.heldout_acc[ep] = n_heldout ? (float)r.hc[ep] / (float)n_heldout : 0.f;
        o.epoch_seconds[ep] = r.secs[ep];
        o.eval_seconds[ep] = r.esecs[ep];
        double l = 0.0;
        for (int s = 0; s < spe; ++s) l += r.ce[3 * (ep * spe + s)];
        o.epoch_loss[ep] = (float)(l / spe);
      }
      o.heldout_acc_final = o.heldout_acc[j.epochs - 1];
      if (r.status != EKYA_OK && overall == EKYA_OK) {
        overall = r.status;
        c.err = "training loss is not finite";
      }
    }
    destroy_events(j);
  }
  // every candidate's streams are idle before the next call reuses the arena
  for (const TrainJob& j : jobs) {
    (void)hipStreamSynchronize(j.st);
    (void)hipStreamSynchronize(j.st2);
  }
  (void)hipEventRecord(c.last_done, s0);
  return overall;
}

// ----------------------------------------------------------------- infer
// Frames per chunk of batched inference.
static constexpr int kInferChunk = 512;

struct InferBufs {
  float *master = nullptr, *fold = nullptr;
  void *shadow = nullptr, *padded = nullptr;
  EvalBufs eb;
};

// own_weights: the call prepares the weights in its arena (ekya_infer);
// otherwise they come from a prepared model.
static void plan_infer(Arena& a, const Net& net, const Geo& geo, int resolution, InferBufs& b,
                       bool own_weights = true) {
  const size_t es = dtype_size(net.dt);
  if (own_weights) {
    b.master = a.take<float>(net.total);
    b.fold = a.take<float>(2 * net.bn_channels);
    b.shadow = a.take_bytes(net.shadow_elems * es);
  }
  b.padded = a.take_bytes((size_t)kInferChunk * resolution * resolution * net.conv[0].cin_pad * es);
  plan_eval(a, net, geo, 0, 5, kInferChunk, b.eb);
}

size_t infer_workspace_bytes(const Net& net, int resolution) {
  InferBufs b;
  Arena a;
  plan_infer(a, net, Geo::build(net, resolution, resolution), resolution, b);
  return a.used;
}

// Inference weights from internal-layout fp32 weights: folded eval-mode
// BatchNorm and the low-precision convolution weights.
static hipError_t prepare_inference(const Net& net, const Tables& t, const float* master,
                                    float* fold, void* shadow, hipStream_t stream) {
  EKYA_HIP(bn_fold(master, t.fold_all, t.n_fold_all, fold, stream));
  EKYA_HIP(pack_conv_weights(net.dt, master, t.pack_all, t.n_pack_all, shadow, stream));
  return hipSuccess;
}

// Classify n frames with prepared weights, chunk by chunk.
static hipError_t infer_frames(const Net& net, const Geo& geo, const float* master,
                               const float* fold, const void* shadow, const void* frames, int n,
                               int H, int W, int resolution, int32_t* labels_out, InferBufs& ib,
                               hipStream_t stream) {
  const size_t es = dtype_size(net.dt);
  const int cap = kInferChunk;
  EvalBufs& eb = ib.eb;
  const long long fbytes = (long long)H * W * 3 * es;
  const int per = n > 0 ? cdiv(n, cdiv(n, cap)) : cap;  // equal chunks (2000: 4 x 500)
  for (int i0 = 0; i0 < n; i0 += per) {
    const int cnt = std::min(per, n - i0);
    const void* src = reinterpret_cast<const char*>(frames) + i0 * fbytes;
    const bool raw_ok = stem_frames_ok(net.dt, conv_geom(net, geo, 0, cnt));
    if (resolution == H && resolution == W && raw_ok) {
      EKYA_HIP(eval_forward(net, geo, shadow, fold, master, 0, 5, src, cnt, eb, eb.logits, stream,
                            true));  // the stem reads the frames
    } else if (raw_ok) {
      // resized to 3-channel frames, which the stem reads as it reads the
      // originals (the same staged bytes as an 8-channel padded copy)
      EKYA_HIP(resize_to_padded(net.dt, src, cnt, H, W, resolution, 3, ib.padded, stream));
      EKYA_HIP(eval_forward(net, geo, shadow, fold, master, 0, 5, ib.padded, cnt, eb, eb.logits,
                            stream, true));
    } else {
      if (resolution == H && resolution == W)
        EKYA_HIP(frames_to_padded(net.dt, src, nullptr, cnt, H, W, net.conv[0].cin_pad, ib.padded,
                                  stream));
      else
        EKYA_HIP(resize_to_padded(net.dt, src, cnt, H, W, resolution, net.conv[0].cin_pad,
                                  ib.padded, stream));
      EKYA_HIP(eval_forward(net, geo, shadow, fold, master, 0, 5, ib.padded, cnt, eb, eb.logits,
                            stream));
    }
    EKYA_HIP(argmax_rows(eb.logits, cnt, net.n_classes, labels_out + i0, stream));
  }
  return hipSuccess;
}

ekya_status run_infer(Ctx& c, const float* weights, const void* frames, int n, int H, int W,
                      int resolution, int precision, int32_t* labels_out, hipStream_t stream) {
  EKYA_CHECK_HIP(hipSetDevice(c.device));
  TimerGuard tg(c);
  const int dt = precision;
  const Net& net = c.net[dt];
  const Geo geo = Geo::build(net, resolution, resolution);
  InferBufs ib;
  {
    Arena meas;
    plan_infer(meas, net, geo, resolution, ib);
    if (ekya_status s = acquire_workspace(c, meas.used, stream)) return s;
  }
  Arena real;
  real.base = reinterpret_cast<char*>(c.ws.p);
  plan_infer(real, net, geo, resolution, ib);
  const Tables& t = c.tabs[dt];
  auto run = [&]() -> hipError_t {
    EKYA_HIP(permute_weights(weights, ib.master, t.permute, t.n_permute, net.total, 1, stream));
    EKYA_HIP(prepare_inference(net, t, ib.master, ib.fold, ib.shadow, stream));
    return infer_frames(net, geo, ib.master, ib.fold, ib.shadow, frames, n, H, W, resolution,
                        labels_out, ib, stream);
  };
  hipError_t he = run();
  (void)hipEventRecord(c.last_done, stream);  // after whatever was queued
  EKYA_CHECK_HIP(he);
  return EKYA_OK;
}

// ------------------------------------------------------------ hot reload
hipError_t model_init(Model& m, int device, int n_classes, int hidden, int dt) {
  m.device = device;
  m.n_classes = n_classes;
  m.hidden = hidden;
  m.dt = dt;
  EKYA_HIP(hipSetDevice(device));
  m.net = Net::build(n_classes, dt, hidden);
  EKYA_HIP(upload_tables(m.net, m.tabs));
  Arena a;
  for (int i = 0; i < 2; ++i) {
    a.take<float>(m.net.total);
    a.take<float>(2 * m.net.bn_channels);
    a.take_bytes(m.net.shadow_elems * dtype_size(dt));
  }
  EKYA_HIP(m.mem.alloc(a.used));
  Arena r;
  r.base = reinterpret_cast<char*>(m.mem.p);
  for (ModelSlot& sl : m.slot) {
    sl.master = r.take<float>(m.net.total);
    sl.fold = r.take<float>(2 * m.net.bn_channels);
    sl.shadow = r.take_bytes(m.net.shadow_elems * dtype_size(dt));
    EKYA_HIP(hipEventCreateWithFlags(&sl.ready, hipEventDisableTiming));
  }
  return hipSuccess;
}

void model_free(Model& m) {
  (void)hipSetDevice(m.device);
  for (ModelSlot& sl : m.slot) {
    if (sl.ready) (void)hipEventSynchronize(sl.ready);
    for (auto& u : sl.uses) {
      (void)hipEventSynchronize(u.second);
      (void)hipEventDestroy(u.second);
    }
    sl.uses.clear();
    if (sl.ready) (void)hipEventDestroy(sl.ready);
    sl.ready = nullptr;
  }
  for (hipEvent_t e : m.pool) (void)hipEventDestroy(e);
  m.pool.clear();
  m.mem.release();
  m.tabs.buf.release();
}

// Record that the call just queued on `stream` read slot s (caller holds mu).
static hipError_t model_note_use(Model& m, int s, hipStream_t stream) {
  ModelSlot& sl = m.slot[s];
  for (auto& u : sl.uses)
    if (u.first == stream) return hipEventRecord(u.second, stream);
  hipEvent_t e;
  if (!m.pool.empty()) {
    e = m.pool.back();
    m.pool.pop_back();
  } else {
    EKYA_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  sl.uses.push_back({stream, e});
  return hipEventRecord(e, stream);
}

hipError_t model_load(Model& m, const float* canonical, const float* internal, hipStream_t stream,
                      uint64_t* version) {
  std::lock_guard<std::mutex> lk(m.mu);
  EKYA_HIP(hipSetDevice(m.device));
  const int s = m.current < 0 ? 0 : 1 - m.current;
  ModelSlot& sl = m.slot[s];
  // the calls still reading this slot finish before it is overwritten
  for (auto& u : sl.uses) EKYA_HIP(hipStreamWaitEvent(stream, u.second, 0));
  for (auto& u : sl.uses) m.pool.push_back(u.second);
  sl.uses.clear();
  if (canonical)
    EKYA_HIP(permute_weights(canonical, sl.master, m.tabs.permute, m.tabs.n_permute, m.net.total,
                             1, stream));
  else
    EKYA_HIP(hipMemcpyAsync(sl.master, internal, m.net.total * sizeof(float),
                            hipMemcpyDeviceToDevice, stream));
  EKYA_HIP(prepare_inference(m.net, m.tabs, sl.master, sl.fold, sl.shadow, stream));
  EKYA_HIP(hipEventRecord(sl.ready, stream));
  sl.version = m.next_version++;
  m.current = s;
  if (version) *version = sl.version;
  return hipSuccess;
}

hipError_t model_export(Model& m, float* canonical_out, hipStream_t stream, uint64_t* version,
                        bool* empty) {
  std::lock_guard<std::mutex> lk(m.mu);
  *empty = m.current < 0;
  if (*empty) return hipSuccess;
  EKYA_HIP(hipSetDevice(m.device));
  ModelSlot& sl = m.slot[m.current];
  EKYA_HIP(hipStreamWaitEvent(stream, sl.ready, 0));
  EKYA_HIP(permute_weights(sl.master, canonical_out, m.tabs.permute, m.tabs.n_permute,
                           m.net.total, 0, stream));
  EKYA_HIP(model_note_use(m, m.current, stream));
  if (version) *version = sl.version;
  return hipSuccess;
}

// Inference for several streams' models in one call: the frames of model i
// are counts[i] consecutive frames.  The models' groups run on up to
// kInferLanes streams of the context (forked from `stream`, joined back),
// each lane with its own buffers; lane l takes groups l, l + lanes, ...
static constexpr int kInferLanes = 4;

static_assert(kInferLanes <= (int)(sizeof(Ctx::lane_join) / sizeof(hipEvent_t)),
              "a join event per lane");

static int infer_lanes(int n_models) { return std::max(1, std::min(n_models, kInferLanes)); }

size_t infer_models_workspace_bytes(const Net& net, int resolution, int n_models) {
  InferBufs b;
  Arena a;
  const Geo g = Geo::build(net, resolution, resolution);
  for (int l = 0; l < infer_lanes(n_models); ++l) plan_infer(a, net, g, resolution, b, false);
  return a.used;
}

ekya_status run_infer_models(Ctx& c, Model* const* models, int n_models, const void* frames,
                             const int* counts, int H, int W, int resolution, int32_t* labels_out,
                             uint64_t* versions, hipStream_t stream) {
  EKYA_CHECK_HIP(hipSetDevice(c.device));
  TimerGuard tg(c);
  const int dt = models[0]->dt;
  const Net& net = c.net[dt];
  const Geo geo = Geo::build(net, resolution, resolution);
  const int lanes = infer_lanes(n_models);
  {
    Arena meas;
    InferBufs b;
    for (int l = 0; l < lanes; ++l) plan_infer(meas, net, geo, resolution, b, false);
    if (ekya_status s = acquire_workspace(c, meas.used, stream)) return s;
  }
  while ((int)c.lanes.size() < lanes) {
    hipStream_t s;
    EKYA_CHECK_HIP(ctx_stream(c, &s));
    c.lanes.push_back(s);
  }
  if (!c.lane_fork) {
    EKYA_CHECK_HIP(hipEventCreateWithFlags(&c.lane_fork, hipEventDisableTiming));
    for (int l = 0; l < kInferLanes; ++l)
      EKYA_CHECK_HIP(hipEventCreateWithFlags(&c.lane_join[l], hipEventDisableTiming));
  }
  Arena real;
  real.base = reinterpret_cast<char*>(c.ws.p);
  std::vector<InferBufs> ib(lanes);
  for (int l = 0; l < lanes; ++l) plan_infer(real, net, geo, resolution, ib[l], false);
  const long long fbytes = (long long)H * W * 3 * dtype_size(dt);
  std::vector<long long> first(n_models + 1, 0);
  for (int i = 0; i < n_models; ++i) first[i + 1] = first[i] + counts[i];
  auto run = [&]() -> hipError_t {
    EKYA_HIP(hipEventRecord(c.lane_fork, stream));
    for (int l = 0; l < lanes; ++l) EKYA_HIP(hipStreamWaitEvent(c.lanes[l], c.lane_fork, 0));
    for (int i = 0; i < n_models; ++i) {
      const int l = i % lanes;
      hipStream_t q = c.lanes[l];
      Model& m = *models[i];
      std::lock_guard<std::mutex> lk(m.mu);  // take, read and mark the slot together
      const int s = m.current;
      ModelSlot& sl = m.slot[s];
      EKYA_HIP(hipStreamWaitEvent(q, sl.ready, 0));
      if (counts[i] > 0)
        EKYA_HIP(infer_frames(net, geo, sl.master, sl.fold, sl.shadow,
                              reinterpret_cast<const char*>(frames) + first[i] * fbytes, counts[i],
                              H, W, resolution, labels_out + first[i], ib[l], q));
      EKYA_HIP(model_note_use(m, s, q));
      if (versions) versions[i] = sl.version;
    }
    for (int l = 0; l < lanes; ++l) {
      EKYA_HIP(hipEventRecord(c.lane_join[l], c.lanes[l]));
      EKYA_HIP(hipStreamWaitEvent(stream, c.lane_join[l], 0));
    }
    return hipSuccess;
  };
  hipError_t he = run();
  (void)hipEventRecord(c.last_done, stream);
  EKYA_CHECK_HIP(he);
  return EKYA_OK;
}

ekya_status run_infer_model(Ctx& c, Model& m, const void* frames, int n, int H, int W,
                            int resolution, int32_t* labels_out, hipStream_t stream,
                            uint64_t* version) {
  EKYA_CHECK_HIP(hipSetDevice(c.device));
  TimerGuard tg(c);
  const Net& net = c.net[m.dt];
  const Geo geo = Geo::build(net, resolution, resolution);
  InferBufs ib;
  {
    Arena meas;
    plan_infer(meas, net, geo, resolution, ib, false);
    if (ekya_status s = acquire_workspace(c, meas.used, stream)) return s;
  }
  Arena real;
  real.base = reinterpret_cast<char*>(c.ws.p);
  plan_infer(real, net, geo, resolution, ib, false);
  hipError_t he;
  {
    // the slot is taken, read and marked as read under the lock, so a load
    // that overwrites it later waits for this call
    std::lock_guard<std::mutex> lk(m.mu);
    if (m.current < 0) {
      c.err = "the model has no published weights (call ekya_model_load first)";
      return EKYA_ERR_INVALID_ARG;
    }
    const int s = m.current;
    ModelSlot& sl = m.slot[s];
    he = hipStreamWaitEvent(stream, sl.ready, 0);
    if (he == hipSuccess)
      he = infer_frames(net, geo, sl.master, sl.fold, sl.shadow, frames, n, H, W, resolution,
                        labels_out, ib, stream);
    const hipError_t hu = model_note_use(m, s, stream);
    if (he == hipSuccess) he = hu;
    if (version) *version = sl.version;
  }
  (void)hipEventRecord(c.last_done, stream);
  EKYA_CHECK_HIP(he);
  return EKYA_OK;
}

}  // namespace ekya
