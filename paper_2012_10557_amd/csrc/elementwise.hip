// Memory-bound kernels of the retraining step: BatchNorm statistics, apply and
// backward; pooling; the classifier layer; softmax cross-entropy; SGD with
// momentum; frame gather / padding / resize; weight repacking.  Every
// reduction is two-level with a fixed order, so results do not depend on
// scheduling (concurrent and sequential runs are bitwise equal).
#include <climits>
#include <algorithm>
#include <type_traits>

#include "kernels.hpp"

namespace ekya {
namespace {

constexpr float BN_EPS = 1e-5f;
constexpr float BN_MOMENTUM = 0.1f;

template <typename T> __device__ __forceinline__ void unit_to_f(uint4 u, float* v) {
  Unit<T> x;
  x.u = u;
#pragma unroll
  for (int i = 0; i < Elt<T>::E; ++i) v[i] = to_f(x.e[i]);
}
template <typename T> __device__ __forceinline__ uint4 f_to_unit(const float* v) {
  Unit<T> x;
#pragma unroll
  for (int i = 0; i < Elt<T>::E; ++i) x.e[i] = from_f<T>(v[i]);
  return x.u;
}

// E per-channel floats p[c0 .. c0+E) (c0 a multiple of E) as 16-byte loads.
template <int E> __device__ __forceinline__ void chan_load(const float* p, int c0, float (&v)[E]) {
#pragma unroll
  for (int i = 0; i < E; i += 4) {
    const float4 t = *reinterpret_cast<const float4*>(p + c0 + i);
    v[i] = t.x;
    v[i + 1] = t.y;
    v[i + 2] = t.z;
    v[i + 3] = t.w;
  }
}

inline int grid_for(long long n, int per_block = 256, int cap = 8192) {
  long long b = cdivl(n, per_block);
  if (b < 1) b = 1;
  return (int)std::min<long long>(b, cap);
}

// Chunks of rows for the partial sums of large-M BatchNorm: about
// BN_CHUNK_ELEMS elements each (at least one row) and at most BN_MAX_CHUNKS
// of them -- up to four blocks per CU stream the activations, and the final
// per-channel reduction reads each channel's partials in one round of loads.
constexpr int BN_MAX_CHUNKS = 1024;
constexpr long long BN_CHUNK_ELEMS = 16384;
inline int bn_chunks(long long M, int C) {
  long long c = cdivl(M * C, BN_CHUNK_ELEMS);
  if (c > BN_MAX_CHUNKS) c = BN_MAX_CHUNKS;
  if (c > M) c = M;
  if (c < 1) c = 1;
  return (int)c;
}

// The ReLU mask of a BatchNorm output recomputed from its input: the forward
// pass stored y = relu((z - mean) * (gamma * invstd) + beta) as T (one fused
// multiply-add, as below), so y > 0 exactly when that value rounded to T is.
// mb (beta) null: no recomputed mask.
template <int E>
__device__ __forceinline__ void mask_coef(const float* gamma, const float* invstd, const float* mb,
                                          int c0, float (&sc)[E], float (&be)[E]) {
  float ga[E], is[E];
  chan_load<E>(gamma, c0, ga);
  chan_load<E>(invstd, c0, is);
  chan_load<E>(mb, c0, be);
#pragma unroll
  for (int i = 0; i < E; ++i) sc[i] = ga[i] * is[i];
}
template <typename T, int E>
__device__ __forceinline__ void apply_mask(const float (&sc)[E], const float (&be)[E],
                                           const float (&mu)[E], const float (&zz)[E],
                                           float (&g)[E]) {
#pragma unroll
  for (int i = 0; i < E; ++i) {
    const float t = __builtin_fmaf(zz[i] - mu[i], sc[i], be[i]);
    g[i] = to_f((T)t) > 0.f ? g[i] : 0.f;
  }
}

// --------------------------------------------------------- BN statistics
// Per chunk of rows: shifted sums S1 = sum(z - K), S2 = sum((z - K)^2) with the
// shift K[c] = z[0][c]; all chunks share K, so the final sums are plain adds.
template <typename T>
__global__ __launch_bounds__(256) void bn_stats_partial(const T* z, long long M, int C,
                                                        long long rows_per_chunk, float* part) {
  constexpr int E = Elt<T>::E;
  const int tpr = C / E;              // threads per row
  const int rpi = 256 / tpr;          // rows in flight
  const int t = threadIdx.x;
  const int cu = t % tpr, rsub = t / tpr;
  const long long r0 = blockIdx.x * rows_per_chunk;
  const long long r1 = std::min<long long>(M, r0 + rows_per_chunk);
  float s1[E], s2[E], K[E];
#pragma unroll
  for (int i = 0; i < E; ++i) s1[i] = s2[i] = 0.f;
  if (rsub < rpi) {
    unit_to_f<T>(*reinterpret_cast<const uint4*>(z + cu * E), K);
    // eight rows' loads issued before they are accumulated (in row order)
    constexpr int U = 8;
    for (long long r = r0 + rsub; r < r1; r += U * rpi) {
      uint4 raw[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const long long rq = r + (long long)q * rpi;
        raw[q] = rq < r1 ? *reinterpret_cast<const uint4*>(z + rq * C + cu * E) : uint4{0, 0, 0, 0};
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        if (r + (long long)q * rpi >= r1) break;
        float v[E];
        unit_to_f<T>(raw[q], v);
#pragma unroll
        for (int i = 0; i < E; ++i) {
          float d = v[i] - K[i];
          s1[i] += d;
          s2[i] += d * d;
        }
      }
    }
  }
  __shared__ float sh[2][256 * 8];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    sh[0][t * E + i] = s1[i];
    sh[1][t * E + i] = s2[i];
  }
  __syncthreads();
  // thread c (< C) sums the rpi partials of channel c in a fixed order
  for (int c = t; c < C; c += 256) {
    int u = c / E, i = c % E;
    float a = 0.f, b = 0.f;
    for (int rs = 0; rs < rpi; ++rs) {
      a += sh[0][(rs * tpr + u) * E + i];
      b += sh[1][(rs * tpr + u) * E + i];
    }
    part[(long long)blockIdx.x * 2 * C + c] = a;
    part[(long long)blockIdx.x * 2 * C + C + c] = b;
  }
}

// Fixed-order sum over chunks of the two partial rows of channel c: one
// block per channel, thread k sums chunks k, k + 256, ... (at most FIN_PER,
// all loads issued before the adds), then the 256 thread sums are added
// pairwise in double in a fixed tree (thread k with k + 128, ...).  Returns
// true for the thread that holds the totals.
constexpr int FIN_CH = 1;
constexpr int FIN_SL = 256;
constexpr int FIN_PER = BN_MAX_CHUNKS / FIN_SL;
__device__ __forceinline__ bool chunk_sums(const float* part, int nchunks, int C, double& a,
                                           double& b) {
  __shared__ double sa[FIN_SL], sb[FIN_SL];
  const int k = threadIdx.x, c = blockIdx.x;
  float x = 0.f, y = 0.f;
  {
    float v1[FIN_PER], v2[FIN_PER];
#pragma unroll
    for (int u = 0; u < FIN_PER; ++u) {
      const int ch = k + FIN_SL * u;
      v1[u] = ch < nchunks ? part[(long long)ch * 2 * C + c] : 0.f;
      v2[u] = ch < nchunks ? part[(long long)ch * 2 * C + C + c] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < FIN_PER; ++u)
      if (k + FIN_SL * u < nchunks) {
        x += v1[u];
        y += v2[u];
      }
  }
  sa[k] = x;
  sb[k] = y;
  __syncthreads();
#pragma unroll
  for (int h = FIN_SL / 2; h >= 1; h >>= 1) {
    if (k < h) {
      sa[k] += sa[k + h];
      sb[k] += sb[k + h];
    }
    __syncthreads();
  }
  if (k != 0) return false;
  a = sa[0];
  b = sb[0];
  return true;
}
static_assert(FIN_CH * FIN_SL == 256, "chunk_sums runs in 256-thread blocks");

template <typename T>
__global__ __launch_bounds__(256) void bn_stats_final(const T* z, const float* part, int nchunks,
                                                      long long M, int C, const float* gamma,
                                                      const float* beta, float* rm, float* rv,
                                                      float* mean, float* invstd, float* scale,
                                                      float* shift) {
  double a, b;
  if (!chunk_sums(part, nchunks, C, a, b)) return;
  const int c = blockIdx.x;
  const double Kc = (double)to_f(z[c]);
  const double d = a / (double)M;
  double var = b / (double)M - d * d;
  if (var < 0.0) var = 0.0;
  const float mu = (float)(Kc + d);
  const float is = (float)(1.0 / sqrt(var + (double)BN_EPS));
  mean[c] = mu;
  invstd[c] = is;
  const float sc = gamma[c] * is;
  scale[c] = sc;
  shift[c] = beta[c] - mu * sc;
  if (rm) {
    const double unb = M > 1 ? var * (double)M / (double)(M - 1) : var;
    rm[c] = (1.f - BN_MOMENTUM) * rm[c] + BN_MOMENTUM * mu;
    rv[c] = (1.f - BN_MOMENTUM) * rv[c] + BN_MOMENTUM * (float)unb;
  }
}

// One thread takes units u0, u0 + S, u0 + 2S, ... (S the grid's thread
// count).  SAME: S is a multiple of the C / E units of a row, so all of a
// thread's units hold the same channels and their coefficients are loaded
// once.  The loads of BN_AU units are issued before any is used.
constexpr int BN_AU = 2;
template <typename T, bool SAME>
__global__ __launch_bounds__(256) void bn_apply_kernel(const T* z, long long units, int C,
                                                       const float* mean, const float* scale,
                                                       const float* beta, const T* res, int relu,
                                                       T* y) {
  constexpr int E = Elt<T>::E;
  const long long S = (long long)gridDim.x * blockDim.x;
  const long long u0 = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  float mu[E], sc[E], be[E];
  auto coefs = [&](int c0) {
    chan_load<E>(mean, c0, mu);
    chan_load<E>(scale, c0, sc);
    chan_load<E>(beta, c0, be);
  };
  if (SAME) coefs((int)((u0 * E) % C));
  for (long long u = u0; u < units; u += BN_AU * S) {
    uint4 rv[BN_AU], rr[BN_AU];
#pragma unroll
    for (int q = 0; q < BN_AU; ++q) {
      const long long uq = u + q * S;
      const bool in = uq < units;
      rv[q] = in ? reinterpret_cast<const uint4*>(z)[uq] : uint4{0, 0, 0, 0};
      rr[q] = (in && res) ? reinterpret_cast<const uint4*>(res)[uq] : uint4{0, 0, 0, 0};
    }
#pragma unroll
    for (int q = 0; q < BN_AU; ++q) {
      const long long uq = u + q * S;
      if (uq >= units) break;
      if (!SAME) coefs((int)((uq * E) % C));
      float v[E], r[E];
      unit_to_f<T>(rv[q], v);
      if (res) unit_to_f<T>(rr[q], r);
#pragma unroll
      for (int i = 0; i < E; ++i) {
        // (z - mean) * scale + beta: no cancellation when invstd is large
        float t = __builtin_fmaf(v[i] - mu[i], sc[i], be[i]);
        if (res) t += r[i];
        if (relu) t = relu_nan(t);
        v[i] = t;
      }
      reinterpret_cast<uint4*>(y)[uq] = f_to_unit<T>(v);
    }
  }
}

// ------------------------------------------- BN, small batches: two launches
// For up to BN_FOLD_MAX_CHUNKS chunks of BN_FOLD_ROWS rows and C a multiple of
// 64: a partial kernel writes per (chunk, 64-channel group) sums, and each
// block of the apply kernel first reduces the chunk sums of its own 64
// channels, in one fixed order (so every block derives the same per-channel
// coefficients), then applies them to its rows.  This replaces the separate
// per-channel final kernel of the general path.
constexpr int BN_FOLD_ROWS = 128;
constexpr int BN_FOLD_MAX_CHUNKS = 64;
constexpr int BN_GROUP = 64;

inline bool bn_fold_ok(long long M, int C) {
  return C % BN_GROUP == 0 && cdivl(M, BN_FOLD_ROWS) <= BN_FOLD_MAX_CHUNKS;
}

// Per (chunk, 64-channel group) partials, in a fixed order.  Forward: the
// chunk's sum S1 and its squared deviations from the chunk mean M2 (rows kept
// in registers for the second pass).  Backward: g = dy [* (y > 0)];
// S1 = sum g, S2 = sum g (z - mean).  Row slices are added in slice order.
template <typename T, bool BWD>
__global__ __launch_bounds__(256) void bn_group_partial(const T* z, const T* dy, const T* y,
                                                        const float* mean, const float* gamma,
                                                        const float* invstd, const float* mb,
                                                        long long M, int C, float* part) {
  constexpr int E = Elt<T>::E, UG = BN_GROUP / E, RI = 256 / UG, RPT = BN_FOLD_ROWS / RI;
  const int t = threadIdx.x, u = t % UG, rs = t / UG;
  const int c0 = blockIdx.y * BN_GROUP + u * E;
  const long long r0 = (long long)blockIdx.x * BN_FOLD_ROWS;
  __shared__ float sh[2][256 * E];
  __shared__ float smean[BN_GROUP];
  float s1[E], s2[E];
#pragma unroll
  for (int i = 0; i < E; ++i) s1[i] = s2[i] = 0.f;
  if constexpr (BWD) {
    float mu[E], msc[E], mbe[E];
    chan_load<E>(mean, c0, mu);
    if (mb) mask_coef<E>(gamma, invstd, mb, c0, msc, mbe);
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const long long r = r0 + rs + (long long)RI * q;
      if (r >= M) break;
      const long long off = r * C + c0;
      float v[E], g[E];
      unit_to_f<T>(*reinterpret_cast<const uint4*>(z + off), v);
      unit_to_f<T>(*reinterpret_cast<const uint4*>(dy + off), g);
      if (y) {
        float yy[E];
        unit_to_f<T>(*reinterpret_cast<const uint4*>(y + off), yy);
#pragma unroll
        for (int i = 0; i < E; ++i) g[i] = yy[i] > 0.f ? g[i] : 0.f;
      } else if (mb) {
        apply_mask<T, E>(msc, mbe, mu, v, g);
      }
#pragma unroll
      for (int i = 0; i < E; ++i) {
        s1[i] += g[i];
        s2[i] += g[i] * (v[i] - mu[i]);
      }
    }
  } else {
    float v[RPT][E];
    const int nk = (int)std::min<long long>(BN_FOLD_ROWS, M - r0);
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const long long r = r0 + rs + (long long)RI * q;
      if (r < M) {
        unit_to_f<T>(*reinterpret_cast<const uint4*>(z + r * C + c0), v[q]);
#pragma unroll
        for (int i = 0; i < E; ++i) s1[i] += v[q][i];
      }
    }
#pragma unroll
    for (int i = 0; i < E; ++i) sh[0][t * E + i] = s1[i];
    __syncthreads();
    if (t < BN_GROUP) {
      float a = 0.f;
      for (int k = 0; k < RI; ++k) a += sh[0][k * BN_GROUP + t];
      smean[t] = a / (float)nk;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const long long r = r0 + rs + (long long)RI * q;
      if (r < M) {
#pragma unroll
        for (int i = 0; i < E; ++i) {
          const float d = v[q][i] - smean[u * E + i];
          s2[i] += d * d;
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < E; ++i) {
    sh[0][t * E + i] = s1[i];
    sh[1][t * E + i] = s2[i];
  }
  __syncthreads();
  if (t < BN_GROUP) {
    float a = 0.f, b = 0.f;
    for (int k = 0; k < RI; ++k) {  // row slices in order
      a += sh[0][k * BN_GROUP + t];
      b += sh[1][k * BN_GROUP + t];
    }
    const int c = blockIdx.y * BN_GROUP + t;
    part[(long long)blockIdx.x * 2 * C + c] = a;
    part[(long long)blockIdx.x * 2 * C + C + c] = b;
  }
}

// Count, mean and sum of squared deviations (n, m, q) of one channel merged
// with those of another set of rows (Chan, Golub and LeVeque's pairwise
// update): stable in float, where the one-pass sum of squares would need
// double.  The weight nb / (n + nb) uses the hardware reciprocal (about one
// ulp).  A set with no rows leaves the state unchanged.
__device__ __forceinline__ void stats_merge(float& n, float& m, float& q, float nb, float mb,
                                            float qb) {
  if (nb == 0.f) return;
  const float nn = n + nb, d = mb - m, f = nb * __builtin_amdgcn_rcpf(nn);
  m += d * f;
  q += qb + d * d * n * f;
  n = nn;
}

// Mean and biased variance of channel c = 64 blockIdx.y + threadIdx.x % 64
// over M rows from forward partials (S1_k, M2_k) of chunks of `crows` rows
// (the last one ragged): chunk k contributes n_k rows of mean S1_k / n_k and
// squared deviations M2_k, merged by stats_merge.  Four slices of chunks
// (k = slice, slice + 4, ...) are merged in k order, then the slices in
// slice order; a slice loads GS_BATCH chunks before merging them, so the
// loads overlap.  The same in every block; true for the thread (one per
// channel) that holds the result.
constexpr int GS_BATCH = 8;
__device__ __forceinline__ bool group_stats(const float* part, int nch, int crows, long long M,
                                            int C, double& mean, double& var) {
  __shared__ float sn[4][BN_GROUP], sm[4][BN_GROUP], sq[4][BN_GROUP];
  const int lc = threadIdx.x % BN_GROUP, sl = threadIdx.x / BN_GROUP;
  const int c = blockIdx.y * BN_GROUP + lc;
  float n = 0.f, m = 0.f, q = 0.f;
  for (int k0 = sl; k0 < nch; k0 += 4 * GS_BATCH) {
    float v1[GS_BATCH], v2[GS_BATCH];
#pragma unroll
    for (int u = 0; u < GS_BATCH; ++u) {
      const int k = k0 + 4 * u;
      v1[u] = k < nch ? part[(long long)k * 2 * C + c] : 0.f;
      v2[u] = k < nch ? part[(long long)k * 2 * C + C + c] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < GS_BATCH; ++u) {
      const int k = k0 + 4 * u;
      if (k < nch) {
        const float nk = (float)std::min<long long>(crows, M - (long long)k * crows);
        stats_merge(n, m, q, nk, v1[u] * __builtin_amdgcn_rcpf(nk), v2[u]);
      }
    }
  }
  sn[sl][lc] = n;
  sm[sl][lc] = m;
  sq[sl][lc] = q;
  __syncthreads();
  if (sl != 0) return false;
#pragma unroll
  for (int k = 1; k < 4; ++k) stats_merge(n, m, q, sn[k][lc], sm[k][lc], sq[k][lc]);
  mean = (double)m;
  var = M > 0 ? std::max(0.0, (double)q / (double)M) : 0.0;
  return true;
}

// Totals of the two partial rows for channel c = 64 blockIdx.y + threadIdx.x % 64:
// four slices of chunks (k = slice, slice + 4, ...) in float, loaded in
// batches as in group_stats, the slices added in order in double.  True for
// the thread (one per channel) that holds them.
__device__ __forceinline__ bool group_sums(const float* part, int nch, int C, double& a,
                                           double& b) {
  __shared__ float sa[4][BN_GROUP], sb[4][BN_GROUP];
  const int lc = threadIdx.x % BN_GROUP, sl = threadIdx.x / BN_GROUP;
  const int c = blockIdx.y * BN_GROUP + lc;
  float x = 0.f, y = 0.f;
  for (int k0 = sl; k0 < nch; k0 += 4 * GS_BATCH) {
    float v1[GS_BATCH], v2[GS_BATCH];
#pragma unroll
    for (int u = 0; u < GS_BATCH; ++u) {
      const int k = k0 + 4 * u;
      v1[u] = k < nch ? part[(long long)k * 2 * C + c] : 0.f;
      v2[u] = k < nch ? part[(long long)k * 2 * C + C + c] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < GS_BATCH; ++u)
      if (k0 + 4 * u < nch) {
        x += v1[u];
        y += v2[u];
      }
  }
  sa[sl][lc] = x;
  sb[sl][lc] = y;
  __syncthreads();
  if (sl != 0) return false;
  a = (((double)sa[0][lc] + (double)sa[1][lc]) + (double)sa[2][lc]) + (double)sa[3][lc];
  b = (((double)sb[0][lc] + (double)sb[1][lc]) + (double)sb[2][lc]) + (double)sb[3][lc];
  return true;
}

// Statistics from the group partials, then y = relu?((z - mean) scale + beta
// [+ res]) on rows [blockIdx.x rpb, +rpb) of the block's 64 channels.  Blocks
// with blockIdx.x == 0 publish mean / invstd / scale / shift and update the
// running statistics.
template <typename T>
__global__ __launch_bounds__(256) void bn_fold_apply(const T* z, const float* part, int nch,
                                                     int crows, long long M, int C, long long rpb,
                                                     const float* gamma, const float* beta,
                                                     float* rm, float* rv, float* mean,
                                                     float* invstd, float* scale, float* shift,
                                                     const T* res, int relu, T* y) {
  constexpr int E = Elt<T>::E, UG = BN_GROUP / E, RI = 256 / UG;
  __shared__ float cf[3][BN_GROUP];
  const int t = threadIdx.x;
  double mean_d, var;
  if (group_stats(part, nch, crows, M, C, mean_d, var)) {
    const int c = blockIdx.y * BN_GROUP + t;
    const float mu = (float)mean_d;
    const float is = (float)(1.0 / sqrt(var + (double)BN_EPS));
    const float sc = gamma[c] * is;
    cf[0][t] = mu;
    cf[1][t] = sc;
    cf[2][t] = beta[c];
    if (blockIdx.x == 0) {
      mean[c] = mu;
      invstd[c] = is;
      scale[c] = sc;
      shift[c] = beta[c] - mu * sc;
      if (rm) {
        const double unb = M > 1 ? var * (double)M / (double)(M - 1) : var;
        rm[c] = (1.f - BN_MOMENTUM) * rm[c] + BN_MOMENTUM * mu;
        rv[c] = (1.f - BN_MOMENTUM) * rv[c] + BN_MOMENTUM * (float)unb;
      }
    }
  }
  __syncthreads();
  const int u = t % UG, rs = t / UG;
  float mu[E], sc[E], be[E];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    mu[i] = cf[0][u * E + i];
    sc[i] = cf[1][u * E + i];
    be[i] = cf[2][u * E + i];
  }
  const long long r0 = blockIdx.x * rpb, r1 = std::min<long long>(M, r0 + rpb);
  const int c0 = blockIdx.y * BN_GROUP + u * E;
  for (long long r = r0 + rs; r < r1; r += RI) {
    const long long off = r * C + c0;
    float v[E], q[E];
    unit_to_f<T>(*reinterpret_cast<const uint4*>(z + off), v);
    if (res) unit_to_f<T>(*reinterpret_cast<const uint4*>(res + off), q);
#pragma unroll
    for (int i = 0; i < E; ++i) {
      float o = __builtin_fmaf(v[i] - mu[i], sc[i], be[i]);
      if (res) o += q[i];
      if (relu) o = relu_nan(o);
      v[i] = o;
    }
    *reinterpret_cast<uint4*>(y + off) = f_to_unit<T>(v);
  }
}

// Backward coefficients from the group partials (dz = a g + b + c (z - mean)),
// then dz (and g if g_out) on the block's rows; blocks with blockIdx.x == 0
// publish dgamma / dbeta.
template <typename T>
__global__ __launch_bounds__(256) void bn_bwd_fold_apply(const T* dy, const T* y, const T* z,
                                                         const float* part, int nch, long long M,
                                                         int C, long long rpb,
                                                         const float* gamma, const float* mean,
                                                         const float* invstd, const float* mb,
                                                         float* dgamma, float* dbeta, T* dz,
                                                         T* g_out) {
  constexpr int E = Elt<T>::E, UG = BN_GROUP / E, RI = 256 / UG;
  __shared__ float cf[4][BN_GROUP];
  const int t = threadIdx.x;
  double sg, sgx;
  if (group_sums(part, nch, C, sg, sgx)) {
    const int c = blockIdx.y * BN_GROUP + t;
    const float is = invstd[c];
    const float db = (float)sg;
    const float dg = (float)(sgx * (double)is);
    const float a = gamma[c] * is;
    cf[0][t] = a;
    cf[1][t] = -a * db / (float)M;
    cf[2][t] = -a * is * dg / (float)M;
    cf[3][t] = mean[c];
    if (blockIdx.x == 0) {
      dbeta[c] = db;
      dgamma[c] = dg;
    }
  }
  __syncthreads();
  const int u = t % UG, rs = t / UG;
  float ca[E], cb[E], cc[E], mu[E];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    ca[i] = cf[0][u * E + i];
    cb[i] = cf[1][u * E + i];
    cc[i] = cf[2][u * E + i];
    mu[i] = cf[3][u * E + i];
  }
  const long long r0 = blockIdx.x * rpb, r1 = std::min<long long>(M, r0 + rpb);
  const int c0 = blockIdx.y * BN_GROUP + u * E;
  float msc[E], mbe[E];
  if (mb) mask_coef<E>(gamma, invstd, mb, c0, msc, mbe);
  for (long long r = r0 + rs; r < r1; r += RI) {
    const long long off = r * C + c0;
    float g[E], zz[E], o[E];
    unit_to_f<T>(*reinterpret_cast<const uint4*>(dy + off), g);
    unit_to_f<T>(*reinterpret_cast<const uint4*>(z + off), zz);
    if (y) {
      float yy[E];
      unit_to_f<T>(*reinterpret_cast<const uint4*>(y + off), yy);
#pragma unroll
      for (int i = 0; i < E; ++i) g[i] = yy[i] > 0.f ? g[i] : 0.f;
    } else if (mb) {
      apply_mask<T, E>(msc, mbe, mu, zz, g);
    }
    if (g_out) *reinterpret_cast<uint4*>(g_out + off) = f_to_unit<T>(g);
#pragma unroll
    for (int i = 0; i < E; ++i) o[i] = ca[i] * g[i] + cb[i] + cc[i] * (zz[i] - mu[i]);
    *reinterpret_cast<uint4*>(dz + off) = f_to_unit<T>(o);
  }
}

// Sum of split-K partials [split][M][C] in split order (+ res), stored in T,
// with the BatchNorm chunk partials of the stored values for the two-launch
// path: one block per chunk of BN_FOLD_ROWS rows and 64 channels, 1024
// threads = 64 row slices x 16 four-channel units (two rows each), partials
// loaded four splits ahead.  Forward: (S1, M2) as bn_group_partial;
// backward: g = out [* (ymask > 0)], (sum g, sum g (z - mean)).
// Sum over the 64 row slices of channel column c (sh[k * 64 + c], k < 64) in a
// fixed order: 16 groups of 4 consecutive slices (all 1024 threads), then
// the 16 group sums; the result in red[c] for c < 64.
__device__ __forceinline__ void slice_sum64(const float* sh, float* grp, float* red) {
  const int t = threadIdx.x, c = t & 63, gi = t >> 6;
  const float* p = sh + (gi * 4) * BN_GROUP + c;
  grp[gi * BN_GROUP + c] = ((p[0] + p[BN_GROUP]) + p[2 * BN_GROUP]) + p[3 * BN_GROUP];
  __syncthreads();
  if (t < BN_GROUP) {
    float a = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) a += grp[k * BN_GROUP + t];
    red[t] = a;
  }
  __syncthreads();
}

constexpr int SBN_SLICES = 64, SBN_RPT = BN_FOLD_ROWS / SBN_SLICES;
template <typename T, bool BWD>
__global__ __launch_bounds__(1024) void split_bn_kernel(const float* part, int splits, long long M,
                                                        int C, const T* res, T* out,
                                                        const T* ymask, const T* z,
                                                        const float* mean, float* bnp) {
  const int t = threadIdx.x, u = t & 15, rs = t >> 4;
  const int c0 = blockIdx.y * BN_GROUP + u * 4;
  const long long r0 = (long long)blockIdx.x * BN_FOLD_ROWS;
  const long long stride = M * C;
  __shared__ float sh[2][1024 * 4];
  __shared__ float grp[16 * BN_GROUP];
  __shared__ float red[2][BN_GROUP];
  bool ok[SBN_RPT];
  long long off[SBN_RPT];
  float v[SBN_RPT][4];
#pragma unroll
  for (int q = 0; q < SBN_RPT; ++q) {
    const long long r = r0 + rs + (long long)SBN_SLICES * q;
    ok[q] = r < M;
    off[q] = (ok[q] ? r : 0) * C + c0;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[q][i] = 0.f;
  }
  for (int sp = 0; sp < splits; sp += 4) {
    float4 p[4][SBN_RPT];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int q = 0; q < SBN_RPT; ++q)
        p[k][q] = (sp + k < splits && ok[q])
                      ? *reinterpret_cast<const float4*>(part + (sp + k) * stride + off[q])
                      : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (sp + k < splits)
#pragma unroll
        for (int q = 0; q < SBN_RPT; ++q) {  // split order per element
          v[q][0] += p[k][q].x;
          v[q][1] += p[k][q].y;
          v[q][2] += p[k][q].z;
          v[q][3] += p[k][q].w;
        }
  }
  float s1[4] = {0.f, 0.f, 0.f, 0.f}, s2[4] = {0.f, 0.f, 0.f, 0.f}, mu[4];
  if (BWD) chan_load<4>(mean, c0, mu);
#pragma unroll
  for (int q = 0; q < SBN_RPT; ++q) {
    if (!ok[q]) continue;
    if (res) {
      float rr[4];
      load4<T>(res + off[q], rr);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[q][i] += rr[i];
    }
    store4<T>(out + off[q], v[q]);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[q][i] = to_f(from_f<T>(v[q][i]));  // the stored values
    if (BWD) {
      float zz[4], g[4] = {v[q][0], v[q][1], v[q][2], v[q][3]};
      load4<T>(z + off[q], zz);
      if (ymask) {
        float yy[4];
        load4<T>(ymask + off[q], yy);
#pragma unroll
        for (int i = 0; i < 4; ++i) g[i] = yy[i] > 0.f ? g[i] : 0.f;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s1[i] += g[i];
        s2[i] += g[i] * (zz[i] - mu[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) s1[i] += v[q][i];
    }
  }
  if (!BWD) {
    const int nk = (int)std::min<long long>(BN_FOLD_ROWS, M - r0);
#pragma unroll
    for (int i = 0; i < 4; ++i) sh[0][t * 4 + i] = s1[i];
    __syncthreads();
    slice_sum64(sh[0], grp, red[0]);
#pragma unroll
    for (int q = 0; q < SBN_RPT; ++q) {
      if (!ok[q]) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float d = v[q][i] - red[0][u * 4 + i] / (float)nk;
        s2[i] += d * d;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) sh[1][t * 4 + i] = s2[i];
    __syncthreads();
    slice_sum64(sh[1], grp, red[1]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sh[0][t * 4 + i] = s1[i];
      sh[1][t * 4 + i] = s2[i];
    }
    __syncthreads();
    slice_sum64(sh[0], grp, red[0]);
    slice_sum64(sh[1], grp, red[1]);
  }
  if (t < BN_GROUP) {
    const int c = blockIdx.y * BN_GROUP + t;
    bnp[(long long)blockIdx.x * 2 * C + c] = red[0][t];
    bnp[(long long)blockIdx.x * 2 * C + C + c] = red[1][t];
  }
}

// Rows per block of the fold apply kernels: about 512 blocks over the
// groups, a whole number of row slices each.
inline long long bn_fold_rpb(long long M, int C, int dt) {
  const int ri = 256 / (BN_GROUP / dtype_vec(dt));
  const long long target = std::max(1, 512 / (C / BN_GROUP));
  return ri * cdivl(cdivl(M, target), ri);
}

// tab row: gamma_off, beta_off, rm_off, rv_off, C, out_off
__global__ void bn_fold_kernel(const float* p, const long long* tab, float* out) {
  const long long* t = tab + 6 * blockIdx.x;
  const int C = (int)t[4];
  for (int c = threadIdx.x; c < C; c += blockDim.x) {
    float sc = p[t[0] + c] / sqrtf(p[t[3] + c] + BN_EPS);
    out[t[5] + c] = sc;
    out[t[5] + C + c] = p[t[1] + c] - p[t[2] + c] * sc;
  }
}

// ------------------------------------------------------------ BN backward
// partials: S_g = sum g, S_gx = sum g * (z - mean), g = dy * [y > 0].
template <typename T>
__global__ __launch_bounds__(256) void bn_bwd_partial(const T* dy, const T* y, const T* z,
                                                      long long M, int C,
                                                      long long rows_per_chunk,
                                                      const float* mean, const float* gamma,
                                                      const float* invstd, const float* mb,
                                                      float* part) {
  constexpr int E = Elt<T>::E;
  const int tpr = C / E;
  const int rpi = 256 / tpr;
  const int t = threadIdx.x;
  const int cu = t % tpr, rsub = t / tpr;
  const long long r0 = blockIdx.x * rows_per_chunk;
  const long long r1 = std::min<long long>(M, r0 + rows_per_chunk);
  float s1[E], s2[E], mu[E], msc[E], mbe[E];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    s1[i] = s2[i] = 0.f;
    mu[i] = mean[cu * E + i];
    msc[i] = mbe[i] = 0.f;
  }
  if (mb) mask_coef<E>(gamma, invstd, mb, cu * E, msc, mbe);
  if (rsub < rpi) {
    // four rows' loads issued before they are accumulated (in row order)
    constexpr int U = 4;
    for (long long r = r0 + rsub; r < r1; r += U * rpi) {
      uint4 rg[U], rz[U], ry[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const long long rq = r + (long long)q * rpi;
        const bool in = rq < r1;
        const long long off = rq * C + cu * E;
        rg[q] = in ? *reinterpret_cast<const uint4*>(dy + off) : uint4{0, 0, 0, 0};
        rz[q] = in ? *reinterpret_cast<const uint4*>(z + off) : uint4{0, 0, 0, 0};
        ry[q] = (in && y) ? *reinterpret_cast<const uint4*>(y + off) : uint4{0, 0, 0, 0};
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        if (r + (long long)q * rpi >= r1) break;
        float g[E], zz[E];
        unit_to_f<T>(rg[q], g);
        unit_to_f<T>(rz[q], zz);
        if (y) {
          float yy[E];
          unit_to_f<T>(ry[q], yy);
#pragma unroll
          for (int i = 0; i < E; ++i) g[i] = yy[i] > 0.f ? g[i] : 0.f;
        } else if (mb) {
          apply_mask<T, E>(msc, mbe, mu, zz, g);
        }
#pragma unroll
        for (int i = 0; i < E; ++i) {
          s1[i] += g[i];
          s2[i] += g[i] * (zz[i] - mu[i]);
        }
      }
    }
  }
  __shared__ float sh[2][256 * 8];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    sh[0][t * E + i] = s1[i];
    sh[1][t * E + i] = s2[i];
  }
  __syncthreads();
  for (int c = t; c < C; c += 256) {
    int u = c / E, i = c % E;
    float a = 0.f, b = 0.f;
    for (int rs = 0; rs < rpi; ++rs) {
      a += sh[0][(rs * tpr + u) * E + i];
      b += sh[1][(rs * tpr + u) * E + i];
    }
    part[(long long)blockIdx.x * 2 * C + c] = a;
    part[(long long)blockIdx.x * 2 * C + C + c] = b;
  }
}

// coef[3C]: dz = a*g + b + c*(z - mean)
__global__ __launch_bounds__(256) void bn_bwd_final(const float* part, int nchunks, long long M,
                                                    int C, const float* gamma, const float* invstd,
                                                    float* dgamma, float* dbeta, float* coef) {
  double sg, sgx;
  if (!chunk_sums(part, nchunks, C, sg, sgx)) return;
  const int c = blockIdx.x;
  const float is = invstd[c];
  const float db = (float)sg;
  const float dg = (float)(sgx * (double)is);
  dbeta[c] = db;
  dgamma[c] = dg;
  const float a = gamma[c] * is;
  coef[c] = a;
  coef[C + c] = -a * db / (float)M;
  coef[2 * C + c] = -a * is * dg / (float)M;
}

// Units per thread as in bn_apply_kernel.
template <typename T, bool SAME>
__global__ __launch_bounds__(256) void bn_bwd_apply(const T* dy, const T* y, const T* z,
                                                    long long units, int C, const float* mean,
                                                    const float* coef, const float* gamma,
                                                    const float* invstd, const float* mb, T* dz,
                                                    T* g_out) {
  constexpr int E = Elt<T>::E;
  const long long S = (long long)gridDim.x * blockDim.x;
  const long long u0 = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  float mu[E], ca[E], cb[E], cc[E], msc[E], mbe[E];
  auto coefs = [&](int c0) {
    chan_load<E>(mean, c0, mu);
    chan_load<E>(coef, c0, ca);
    chan_load<E>(coef + C, c0, cb);
    chan_load<E>(coef + 2 * C, c0, cc);
    if (!y && mb) mask_coef<E>(gamma, invstd, mb, c0, msc, mbe);
  };
  if (SAME) coefs((int)((u0 * E) % C));
  for (long long u = u0; u < units; u += BN_AU * S) {
    uint4 rg[BN_AU], rz[BN_AU], ry[BN_AU];
#pragma unroll
    for (int q = 0; q < BN_AU; ++q) {
      const long long uq = u + q * S;
      const bool in = uq < units;
      rg[q] = in ? reinterpret_cast<const uint4*>(dy)[uq] : uint4{0, 0, 0, 0};
      rz[q] = in ? reinterpret_cast<const uint4*>(z)[uq] : uint4{0, 0, 0, 0};
      ry[q] = (in && y) ? reinterpret_cast<const uint4*>(y)[uq] : uint4{0, 0, 0, 0};
    }
#pragma unroll
    for (int q = 0; q < BN_AU; ++q) {
      const long long uq = u + q * S;
      if (uq >= units) break;
      if (!SAME) coefs((int)((uq * E) % C));
      float g[E], zz[E], o[E];
      unit_to_f<T>(rg[q], g);
      unit_to_f<T>(rz[q], zz);
      if (y) {
        float yy[E];
        unit_to_f<T>(ry[q], yy);
#pragma unroll
        for (int i = 0; i < E; ++i) g[i] = yy[i] > 0.f ? g[i] : 0.f;
      } else if (mb) {
        apply_mask<T, E>(msc, mbe, mu, zz, g);
      }
      if (g_out) reinterpret_cast<uint4*>(g_out)[uq] = f_to_unit<T>(g);
#pragma unroll
      for (int i = 0; i < E; ++i) o[i] = ca[i] * g[i] + cb[i] + cc[i] * (zz[i] - mu[i]);
      reinterpret_cast<uint4*>(dz)[uq] = f_to_unit<T>(o);
    }
  }
}

// ---------------------------------------------------------------- pooling
// E window indices (bytes) of one 16-byte unit, moved as one 4- or 8-byte word.
template <int E> struct ArgWord;
template <> struct ArgWord<8> { using type = uint2; };
template <> struct ArgWord<4> { using type = uint32_t; };
template <int E> __device__ __forceinline__ void arg_load(const uint8_t* p, int (&a)[E]) {
  union {
    typename ArgWord<E>::type w;
    uint8_t b[E];
  } u;
  u.w = *reinterpret_cast<const typename ArgWord<E>::type*>(p);
#pragma unroll
  for (int i = 0; i < E; ++i) a[i] = u.b[i];
}
template <int E> __device__ __forceinline__ void arg_store(uint8_t* p, const int (&a)[E]) {
  union {
    typename ArgWord<E>::type w;
    uint8_t b[E];
  } u;
#pragma unroll
  for (int i = 0; i < E; ++i) u.b[i] = (uint8_t)a[i];
  *reinterpret_cast<typename ArgWord<E>::type*>(p) = u.w;
}

// 3x3 / stride 2 / pad 1 max pool.  One block covers 256 units (pixel x
// 16-byte channel unit) of a pair of output rows p, p + 1 (p even; the
// second absent for the last row of an odd P); bpr blocks per row pair (the
// pair index from the block index is uniform, so no per-lane wide division).
// The two windows of a thread share input row 2p + 1: its five input rows
// are loaded once, and each element converted once.
// BNR: x is a BatchNorm input z and the pooled values are the BatchNorm +
// ReLU outputs relu((z - mean) * scale + beta), rounded to T exactly as the
// standalone apply kernel stores them (so the window maxima and their
// indices are those of the stored activation).
template <typename T, bool BNR = false>
__global__ __launch_bounds__(256) void maxpool_fwd_kernel(const T* x, int N, int H, int W, int C,
                                                          int P, int Q, int bpr, T* y,
                                                          uint8_t* arg, const float* mean,
                                                          const float* scale,
                                                          const float* beta) {
  constexpr int E = Elt<T>::E;
  const int cu = C / E;
  const int PR = (P + 1) / 2;
  const int pair = blockIdx.x / bpr;  // n * PR + p / 2
  const int t = (blockIdx.x - pair * bpr) * 256 + threadIdx.x;
  if (pair >= N * PR || t >= Q * cu) return;
  const int q = t / cu, c0 = (t - q * cu) * E;
  const int n = pair / PR, p = 2 * (pair - n * PR);
  const bool two = p + 1 < P;
  float mu[E], sc[E], be[E];
  if constexpr (BNR) {
    chan_load<E>(mean, c0, mu);
    chan_load<E>(scale, c0, sc);
    chan_load<E>(beta, c0, be);
  }
  float best0[E], best1[E];
  int ba0[E], ba1[E];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    best0[i] = best1[i] = -INFINITY;
    ba0[i] = ba1[i] = 0;
  }
  // all fifteen loads in flight before the comparisons; input row rr is
  // window row rr of output row p and window row rr - 2 of output row p + 1
  uint4 raw[15];
  bool ok[15];
#pragma unroll
  for (int rr = 0; rr < 5; ++rr)
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const int h = 2 * p + rr - 1, w = 2 * q + s - 1;
      ok[3 * rr + s] = (rr < 3 || two) && h >= 0 && h < H && w >= 0 && w < W;
      raw[3 * rr + s] = ok[3 * rr + s]
                            ? *reinterpret_cast<const uint4*>(x + (((long long)n * H + h) * W + w) * C + c0)
                            : uint4{0, 0, 0, 0};
    }
#pragma unroll
  for (int k = 0; k < 15; ++k) {
    if (!ok[k]) continue;
    float v[E];
    unit_to_f<T>(raw[k], v);
    if constexpr (BNR) {
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] = to_f((T)relu_nan(__builtin_fmaf(v[i] - mu[i], sc[i], be[i])));
    }
    if (k < 9) {  // windows in (r, s) order: the first maximum wins
#pragma unroll
      for (int i = 0; i < E; ++i)
        if (v[i] > best0[i]) {
          best0[i] = v[i];
          ba0[i] = k;
        }
    }
    if (k >= 6) {
#pragma unroll
      for (int i = 0; i < E; ++i)
        if (v[i] > best1[i]) {
          best1[i] = v[i];
          ba1[i] = k - 6;
        }
    }
  }
  const long long o = (((long long)n * P + p) * Q + q) * C + c0;
  *reinterpret_cast<uint4*>(y + o) = f_to_unit<T>(best0);
  if (arg) arg_store<E>(arg + o, ba0);
  if (two) {
    const long long o1 = o + (long long)Q * C;
    *reinterpret_cast<uint4*>(y + o1) = f_to_unit<T>(best1);
    if (arg) arg_store<E>(arg + o1, ba1);
  }
}

// Input gradient of the max pool: a gather over the (at most 2 x 2) windows
// that contain the pixel, adding the output gradient of each whose recorded
// maximum is this pixel.  Blocks as in the forward pass, over input rows.
template <typename T>
__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const T* dy, const uint8_t* arg, int N,
                                                          int H, int W, int C, int P, int Q,
                                                          int bpr, T* dx) {
  constexpr int E = Elt<T>::E;
  const int cu = C / E;
  const int row = blockIdx.x / bpr;  // n * H + h
  const int t = (blockIdx.x - row * bpr) * 256 + threadIdx.x;
  if (row >= N * H || t >= W * cu) return;
  const int w = t / cu, c0 = (t - w * cu) * E;
  const int n = row / H, h = row - n * H;
  float acc[E];
#pragma unroll
  for (int i = 0; i < E; ++i) acc[i] = 0.f;
  // window row / column offsets r, s with h + 1 - r and w + 1 - s even: one
  // (even coordinate) or two (odd) of each; all loads in flight before the adds
  const int r0 = (h & 1) ? 0 : 1, nr = (h & 1) ? 2 : 1;
  const int s0 = (w & 1) ? 0 : 1, nsw = (w & 1) ? 2 : 1;
  uint4 graw[4];
  int a[4][E];
  bool ok[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = r0 + 2 * (k >> 1), s = s0 + 2 * (k & 1);
    const int hp = h + 1 - r, wp = w + 1 - s;
    ok[k] = (k >> 1) < nr && (k & 1) < nsw && hp >= 0 && (hp >> 1) < P && wp >= 0 && (wp >> 1) < Q;
    const long long o = (((long long)n * P + (hp >> 1)) * Q + (wp >> 1)) * C + c0;
    if (ok[k]) {
      graw[k] = *reinterpret_cast<const uint4*>(dy + o);
      arg_load<E>(arg + o, a[k]);
    } else {
      graw[k] = uint4{0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < E; ++i) a[k][i] = -1;
    }
  }
  // windows in (r, s) order, as a row-major walk over the 3 x 3 offsets
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (!ok[k]) continue;
    const int r = r0 + 2 * (k >> 1), s = s0 + 2 * (k & 1);
    float g[E];
    unit_to_f<T>(graw[k], g);
#pragma unroll
    for (int i = 0; i < E; ++i)
      if (a[k][i] == r * 3 + s) acc[i] += g[i];
  }
  *reinterpret_cast<uint4*>(dx + ((long long)row * W + w) * C + c0) = f_to_unit<T>(acc);
}

// ------------------------------- max pool backward inside the BatchNorm backward
// For a BatchNorm + ReLU whose output went only into the 3x3 / stride 2 /
// pad 1 max pool (the stem, 64 channels): the gradient at output pixel
// (n, h, w) is gathered from the pooled gradient and window indices exactly as
// maxpool_bwd_kernel computes it (windows in (r, s) order) and rounded to T as
// that kernel stores it; the ReLU mask is recomputed from z.  So every
// element's gradient is the one bn_backward would read after maxpool_bwd
// (the statistics add the same terms, grouped differently), without the
// full-size gradient being written or read.
// Input rows 2p and 2p + 1 take their gradient from pooled rows p and p + 1
// only: a block stages those two pooled rows (gradient and indices) in LDS,
// then gathers from there while it streams the two rows of z.
struct PoolSrc {
  const void* dy;      // pooled gradient [N][P][Q][C]
  const uint8_t* arg;  // window indices, same layout
  int H, W, P, Q;
};
constexpr int POOLBN_C = 64;
constexpr int POOLBN_QMAX = 64;  // pooled width (stem output width up to 128)

template <typename T>
struct PoolRows {
  static constexpr int E = Elt<T>::E, CU = POOLBN_C / E;
  // pooled rows p, p + 1 (zero beyond the image), each Q + 1 columns wide:
  // units [2][Q + 1][CU], indices [2][Q + 1][C]; column Q stays zero, the
  // right neighbour of an odd last input column
  uint4 g[2 * (POOLBN_QMAX + 1) * CU];
  uint8_t a[2 * (POOLBN_QMAX + 1) * POOLBN_C];
};

// Pooled rows p, p + 1 of image n, held in registers between their loads and
// their LDS writes so that a thread's loads are all in flight together: a
// 256-thread block covers the 2 x POOLBN_QMAX x CU gradient units in GPT
// loads per thread and the index units in APT.
template <typename T>
struct PoolRowsRegs {
  static constexpr int CU = POOLBN_C / Elt<T>::E;
  static constexpr int GPT = 2 * POOLBN_QMAX * CU / 256, APT = 2 * POOLBN_QMAX * POOLBN_C / 16 / 256;
  uint4 g[GPT], a[APT];
};

template <typename T>
__device__ __forceinline__ void pool_rows_load(const PoolSrc& ps, int n, int p, int tid,
                                               PoolRowsRegs<T>& r) {
  using R = PoolRowsRegs<T>;
  const int per_g = ps.Q * R::CU, per_a = ps.Q * POOLBN_C / 16;
#pragma unroll
  for (int j = 0; j < R::GPT; ++j) {
    const int i = tid + 256 * j, rr = i >= per_g, rem = i - rr * per_g;
    r.g[j] = i < 2 * per_g && p + rr < ps.P
                 ? reinterpret_cast<const uint4*>(ps.dy)[((long long)n * ps.P + p + rr) * per_g + rem]
                 : uint4{0, 0, 0, 0};
  }
#pragma unroll
  for (int j = 0; j < R::APT; ++j) {
    const int i = tid + 256 * j, rr = i >= per_a, rem = i - rr * per_a;
    r.a[j] = i < 2 * per_a && p + rr < ps.P
                 ? reinterpret_cast<const uint4*>(ps.arg)[((long long)n * ps.P + p + rr) * per_a + rem]
                 : uint4{0, 0, 0, 0};
  }
}

template <typename T>
__device__ __forceinline__ void pool_rows_store(const PoolSrc& ps, const PoolRowsRegs<T>& r, int tid,
                                                PoolRows<T>& sm) {
  using R = PoolRowsRegs<T>;
  const int per_g = ps.Q * R::CU, per_a = ps.Q * POOLBN_C / 16;
#pragma unroll
  for (int j = 0; j < R::GPT; ++j) {
    const int i = tid + 256 * j, rr = i >= per_g;
    if (i < 2 * per_g) sm.g[i + rr * R::CU] = r.g[j];
  }
#pragma unroll
  for (int j = 0; j < R::APT; ++j) {
    const int i = tid + 256 * j, rr = i >= per_a;
    if (i < 2 * per_a) reinterpret_cast<uint4*>(sm.a)[i + rr * (POOLBN_C / 16)] = r.a[j];
  }
}

// The zero column Q of both staged rows (written once; staging never touches it).
template <typename T>
__device__ __forceinline__ void pool_rows_zero_pad(const PoolSrc& ps, PoolRows<T>& sm) {
  constexpr int CU = POOLBN_C / Elt<T>::E, AU = POOLBN_C / 16;
  const int t = threadIdx.x;
  if (t < 2 * CU) sm.g[((t / CU) * (ps.Q + 1) + ps.Q) * CU + t % CU] = uint4{0, 0, 0, 0};
  if (t < 2 * AU)
    reinterpret_cast<uint4*>(sm.a)[((t / AU) * (ps.Q + 1) + ps.Q) * AU + t % AU] = uint4{0, 0, 0, 0};
}

// Gradient of unit cu of input pixel (h = 2p + hh, w), from the staged rows.
// Row parity hh and column parity w & 1 fix which windows hold the pixel: an
// even row only window row r = 1 of pooled row p; an odd row r = 0 of row
// p + 1 and r = 2 of row p; an even column only s = 1 of pooled column w / 2;
// an odd column s = 0 of (w + 1) / 2 and s = 2 of (w - 1) / 2.  Both parities
// are the same across a wave, so the candidates are taken in (r, s) order
// with branches that never split a wave.
template <typename T>
__device__ __forceinline__ void pool_rows_grad(const PoolSrc& ps, const PoolRows<T>& sm, int hh,
                                               int par, int w, int cu, float (&g)[Elt<T>::E]) {
  constexpr int E = Elt<T>::E, CU = POOLBN_C / E;
  float acc[E];
#pragma unroll
  for (int i = 0; i < E; ++i) acc[i] = 0.f;
  const int Q1 = ps.Q + 1;
#pragma unroll
  for (int kr = 0; kr < 2; ++kr) {
    if (kr > hh) break;
    const int r = hh ? 2 * kr : 1, rr = hh ? 1 - kr : 0;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      if (ks > par) break;
      const int s = par ? 2 * ks : 1, q = (w + 1 - s) >> 1;  // q <= Q (the zero column)
      float v[E];
      int a[E];
      unit_to_f<T>(sm.g[(rr * Q1 + q) * CU + cu], v);
      arg_load<E>(sm.a + (rr * Q1 + q) * POOLBN_C + cu * E, a);  // one 4- or 8-byte LDS read
#pragma unroll
      for (int i = 0; i < E; ++i)
        if (a[i] == r * 3 + s) acc[i] += v[i];
    }
  }
#pragma unroll
  for (int i = 0; i < E; ++i) g[i] = to_f((T)acc[i]);
}

// STATS: partial sums S_g, S_gx of block b's rp row pairs into part[b];
// otherwise dz of block b's rp row pairs.
template <typename T, bool STATS>
__global__ __launch_bounds__(256, STATS ? 4 : 1) void bn_bwd_pool_kernel(
    PoolSrc ps, const T* z, int N, int rp, const float* mean, const float* coef,
    const float* gamma, const float* invstd, const float* mb, float* part, T* dz) {
  constexpr int E = Elt<T>::E, CU = POOLBN_C / E;
  __shared__ PoolRows<T> sm;
  const int t = threadIdx.x, cu = t % CU, c0 = cu * E;
  float mu[E], msc[E], mbe[E], ca[E], cb[E], cc[E], s1[E], s2[E];
  chan_load<E>(mean, c0, mu);
  mask_coef<E>(gamma, invstd, mb, c0, msc, mbe);
  if constexpr (!STATS) {
    chan_load<E>(coef, c0, ca);
    chan_load<E>(coef + POOLBN_C, c0, cb);
    chan_load<E>(coef + 2 * POOLBN_C, c0, cc);
  }
#pragma unroll
  for (int i = 0; i < E; ++i) s1[i] = s2[i] = 0.f;
  const int pairs = N * ps.P;
  const int k0 = blockIdx.x * rp, k1 = min(pairs, k0 + rp);
  // units by parity class (hh, w & 1): class c = 2 hh + (w & 1) takes
  // units [c G, c G + G), G = GW x 64 so a wave stays in one class; within a
  // class unit i is column 2 (i / CU) + (w & 1), channel unit i % CU.  A
  // wave's units of a pair are 64 (wave + 4 j) + lane, so its class for
  // step j is (wave + 4 j) / GW, a scalar.
  const int GW = cdiv(cdiv(ps.W, 2) * CU, 64), G = GW * 64;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  constexpr int ZPT = 4 * ((POOLBN_QMAX * CU + 63) / 64) * 64 / 256;
  static_assert(256 % CU == 0 && 64 % CU == 0, "a thread keeps its channel unit");
  pool_rows_zero_pad<T>(ps, sm);  // ordered before any read by the first pair's barriers
  for (int k = k0; k < k1; ++k) {
    const int n = k / ps.P, p = k - n * ps.P;
    // the per-unit offsets and predicates are recomputed each pair from an
    // opaque copy of the thread index: hoisted out of the loop they would
    // occupy most of the register file
    int tl = t;
    asm volatile("" : "+v"(tl));
    const long long base = ((long long)n * ps.H + 2 * p) * ps.W * POOLBN_C + c0;
    // z of the pair and its two pooled rows are loaded together before any is used
    uint4 zr[ZPT];
#pragma unroll
    for (int j = 0; j < ZPT; ++j) {
      const int cls = (wave + 4 * j) / GW, hh = cls >> 1;
      const int w = 2 * ((tl + 256 * j - cls * G) / CU) + (cls & 1);
      zr[j] = cls < 4 && w < ps.W && 2 * p + hh < ps.H
                  ? *reinterpret_cast<const uint4*>(z + base + ((long long)hh * ps.W + w) * POOLBN_C)
                  : uint4{0, 0, 0, 0};
    }
    PoolRowsRegs<T> pr;
    pool_rows_load<T>(ps, n, p, tl, pr);
    __syncthreads();  // the previous pair's staged rows are no longer read
    pool_rows_store<T>(ps, pr, tl, sm);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < ZPT; ++j) {
      const int cls = (wave + 4 * j) / GW, hh = cls >> 1;
      if (cls >= 4 || 2 * p + hh >= ps.H) continue;  // wave-uniform
      const int w = 2 * ((tl + 256 * j - cls * G) / CU) + (cls & 1);
      if (w >= ps.W) continue;
      float g[E], zz[E];
      unit_to_f<T>(zr[j], zz);
      pool_rows_grad<T>(ps, sm, hh, cls & 1, w, cu, g);
      apply_mask<T, E>(msc, mbe, mu, zz, g);
      if constexpr (STATS) {
#pragma unroll
        for (int i = 0; i < E; ++i) {
          s1[i] += g[i];
          s2[i] += g[i] * (zz[i] - mu[i]);
        }
      } else {
        float o[E];
#pragma unroll
        for (int i = 0; i < E; ++i) o[i] = ca[i] * g[i] + cb[i] + cc[i] * (zz[i] - mu[i]);
        *reinterpret_cast<uint4*>(dz + base + ((long long)hh * ps.W + w) * POOLBN_C) = f_to_unit<T>(o);
      }
      // one unit's LDS reads at a time: hoisting them all costs the whole register file
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if constexpr (STATS) {
    // threads t, t + CU, ... share channel unit cu: added in thread order
    __syncthreads();
    float* sh = reinterpret_cast<float*>(&sm);  // 2 x 256 x E floats (<= the staging area)
#pragma unroll
    for (int i = 0; i < E; ++i) {
      sh[t * E + i] = s1[i];
      sh[256 * E + t * E + i] = s2[i];
    }
    __syncthreads();
    if (t < POOLBN_C) {
      const int u = t / E, i = t % E;
      float a = 0.f, bsum = 0.f;
      for (int j = u; j < 256; j += CU) {
        a += sh[j * E + i];
        bsum += sh[256 * E + j * E + i];
      }
      part[(long long)blockIdx.x * 2 * POOLBN_C + t] = a;
      part[(long long)blockIdx.x * 2 * POOLBN_C + POOLBN_C + t] = bsum;
    }
  }
}
static_assert(sizeof(PoolRows<float>) >= 2 * 256 * 4 * sizeof(float), "reduction fits the staging area");
static_assert(sizeof(PoolRows<bf16>) >= 2 * 256 * 8 * sizeof(float), "reduction fits the staging area");

template <typename T>
__global__ void avgpool_fwd_kernel(const T* x, int N, int HW, int C, float* f) {
  const long long n_out = (long long)N * C;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n_out;
       i += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(i % C);
    const long long n = i / C;
    float s = 0.f;
    for (int k = 0; k < HW; ++k) s += to_f(x[(n * HW + k) * C + c]);
    f[i] = s / (float)HW;
  }
}

template <typename T>
__global__ void avgpool_bwd_kernel(const float* df, int N, int HW, int C, T* dx) {
  const long long n_el = (long long)N * HW * C;
  const float inv = 1.f / (float)HW;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n_el;
       i += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(i % C);
    const long long n = i / ((long long)HW * C);
    dx[i] = from_f<T>(df[n * C + c] * inv);
  }
}

// ------------------------------------------------------------- classifier
// One block per row: each thread takes a strided slice of the features for 8
// classes at a time, then a fixed-order wave and block reduction.
__global__ __launch_bounds__(256) void fc_fwd_kernel(const float* f, const float* W, const float* b,
                                                     int N, int I, int J, float* z) {
  __shared__ float red[4][8];
  const int n = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* fr = f + (long long)n * I;
  for (int j0 = 0; j0 < J; j0 += 8) {
    float s[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) s[k] = 0.f;
    for (int i = t; i < I; i += 256) {
      const float x = fr[i];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (j0 + k < J) s[k] += x * W[(long long)(j0 + k) * I + i];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float v = s[k];
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
      if (lane == 0) red[wave][k] = v;
    }
    __syncthreads();
    if (t < 8 && j0 + t < J)
      z[(long long)n * J + j0 + t] = ((red[0][t] + red[1][t]) + (red[2][t] + red[3][t])) + b[j0 + t];
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void softmax_ce_kernel(const float* z, const int32_t* labels,
                                                         const int32_t* idx, int N, int J,
                                                         float* dz, float* out) {
  __shared__ float sl[256];
  __shared__ int sc[256];
  __shared__ int sn[256];
  float loss = 0.f;
  int correct = 0, bad = 0;
  for (int n = threadIdx.x; n < N; n += 256) {
    const float* zr = z + (long long)n * J;
    const int y = labels[idx ? idx[n] : n];
    if (y < 0 || y >= J) {  // invalid label: flag it, no gradient from this row
      bad = 1;
      for (int j = 0; j < J; ++j) dz[(long long)n * J + j] = 0.f;
      continue;
    }
    float m = zr[0];
    int am = 0;
    for (int j = 1; j < J; ++j)
      if (zr[j] > m) {
        m = zr[j];
        am = j;
      }
    float se = 0.f;
    for (int j = 0; j < J; ++j) se += expf(zr[j] - m);
    const float lse = m + logf(se);
    const float l = lse - zr[y];
    if (!isfinite(l)) bad = 1;
    loss += l;
    correct += (am == y);
    for (int j = 0; j < J; ++j)
      dz[(long long)n * J + j] = (expf(zr[j] - lse) - (j == y ? 1.f : 0.f)) / (float)N;
  }
  sl[threadIdx.x] = loss;
  sc[threadIdx.x] = correct;
  sn[threadIdx.x] = bad;
  __syncthreads();
  if (threadIdx.x == 0) {
    float L = 0.f;
    int C = 0, B = 0;
    for (int t = 0; t < 256; ++t) {
      L += sl[t];
      C += sc[t];
      B |= sn[t];
    }
    out[0] = L / (float)N;
    out[1] = (float)C;
    out[2] = (float)B;
  }
}

__global__ void fc_bwd_w_kernel(const float* dz, const float* f, int N, int I, int J, float* dW,
                                float* db) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < J * I) {
    const int j = t / I, i = t % I;
    float s = 0.f;
    for (int n = 0; n < N; ++n) s += dz[(long long)n * J + j] * f[(long long)n * I + i];
    dW[t] = s;
  }
  if (t < J) {
    float s = 0.f;
    for (int n = 0; n < N; ++n) s += dz[(long long)n * J + t];
    db[t] = s;
  }
}

__global__ void fc_bwd_x_kernel(const float* dz, const float* W, int N, int I, int J, float* df) {
  const long long t = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (t >= (long long)N * I) return;
  const int n = (int)(t / I), i = (int)(t % I);
  float s = 0.f;
  for (int j = 0; j < J; ++j) s += dz[(long long)n * J + j] * W[(long long)j * I + i];
  df[t] = s;
}

// ----------------------------------------------------- fused classifier head
// Forward: one block per sample: pooled[n][c] = mean over the HW pixels of
// x[n] (or the given features f when x is null), then the logits as in
// fc_fwd_kernel.  Backward: one launch for softmax cross-entropy, the
// classifier's weight and bias gradients and the average-pool backward.
// Every block recomputes the (6-wide) softmax rows it needs from the logits,
// so no intermediate dz array or extra launch is needed.
template <typename T, int NW, int IMAX>
__global__ __launch_bounds__(NW * 64) void head_fwd_kernel(const T* x, int HW, const float* fin,
                                                           const float* W, const float* b, int I,
                                                           int J, float* pooled, float* z) {
  constexpr int E = Elt<T>::E;
  __shared__ float fl[IMAX];
  __shared__ float red[NW][8];
  __shared__ float ps[NW][IMAX];
  const int n = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  if (x) {
    // thread: one 16-byte unit of channels x one of NW pixel slices (pixels
    // wave, wave + NW, ...), four pixels' loads in flight, added in pixel
    // order; the slices added in order
    const int units = I / E;
    for (int u = lane; u < units; u += 64) {
      float acc[E];
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = 0.f;
      const T* xp = x + (long long)n * HW * I + u * E;
      int k = wave;
      for (; k + 3 * NW < HW; k += 4 * NW) {
        float v[4][E];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          unit_to_f<T>(*reinterpret_cast<const uint4*>(xp + (long long)(k + q * NW) * I), v[q]);
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < E; ++e) acc[e] += v[q][e];
      }
      for (; k < HW; k += NW) {
        float v[E];
        unit_to_f<T>(*reinterpret_cast<const uint4*>(xp + (long long)k * I), v);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] += v[e];
      }
#pragma unroll
      for (int e = 0; e < E; ++e) ps[wave][u * E + e] = acc[e];
    }
    __syncthreads();
    for (int i = t; i < I; i += NW * 64) {
      float v = ps[0][i];
#pragma unroll
      for (int w = 1; w < NW; ++w) v += ps[w][i];
      v /= (float)HW;
      pooled[(long long)n * I + i] = v;
      fl[i] = v;
    }
  } else {
    for (int i = t; i < I; i += NW * 64) fl[i] = fin[(long long)n * I + i];
  }
  __syncthreads();
  for (int j0 = 0; j0 < J; j0 += 8) {
    float s[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) s[k] = 0.f;
    for (int i = t; i < I; i += NW * 64) {
      const float xv = fl[i];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (j0 + k < J) s[k] += xv * W[(long long)(j0 + k) * I + i];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float v = s[k];
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
      if (lane == 0) red[wave][k] = v;
    }
    __syncthreads();
    if (t < 8 && j0 + t < J) {
      float v = red[0][t];
#pragma unroll
      for (int w = 1; w < NW; ++w) v += red[w][t];
      z[(long long)n * J + j0 + t] = v + b[j0 + t];
    }
    __syncthreads();
  }
}

constexpr int HEAD_JMAX = 16;  // classes handled by the fused backward (else the separate kernels)
constexpr int HEAD_WB = 8;     // blocks of 64 features for the weight gradient (I = 512)
constexpr int HEAD_PC = 8;     // pixels per block of the pooled-feature gradient

// Softmax cross-entropy gradient of one row (J <= HEAD_JMAX): dz[j] =
// (softmax_j - [j == y]) / N, zero for j >= J; false (dz = 0) for a label
// outside [0, J).  The logits are loaded up front.
__device__ __forceinline__ bool ce_row(const float* zr, int y, int J, int N,
                                       float (&dz)[HEAD_JMAX], float& loss, int& correct) {
  float v[HEAD_JMAX];
#pragma unroll
  for (int j = 0; j < HEAD_JMAX; ++j) v[j] = j < J ? zr[j] : 0.f;
  if (y < 0 || y >= J) {
#pragma unroll
    for (int j = 0; j < HEAD_JMAX; ++j) dz[j] = 0.f;
    loss = 0.f;
    correct = 0;
    return false;
  }
  float m = v[0], vy = v[0];
  int am = 0;
#pragma unroll
  for (int j = 1; j < HEAD_JMAX; ++j) {
    if (j < J && v[j] > m) {
      m = v[j];
      am = j;
    }
    if (j == y) vy = v[j];
  }
  float se = 0.f;
#pragma unroll
  for (int j = 0; j < HEAD_JMAX; ++j)
    if (j < J) se += expf(v[j] - m);
  const float lse = m + logf(se);
  loss = lse - vy;
  correct = (am == y);
#pragma unroll
  for (int j = 0; j < HEAD_JMAX; ++j)
    dz[j] = j < J ? (expf(v[j] - lse) - (j == y ? 1.f : 0.f)) / (float)N : 0.f;
  return true;
}

// Blocks [0, HEAD_WB): classifier gradients dW (64 features per block) and,
// in block 0, db / mean loss / correct count / non-finite flag.  Blocks
// after: the pooled-feature gradient spread over the HW pixels,
// dout[n][p][c] = (sum_j dz_j W[j][c]) / HW, one sample and HEAD_PC pixels
// per block.
// BNP: the pooled-feature gradient blocks instead cover 64-row chunks x 64
// channels of dout (rows n HW + p) and also leave the backward BatchNorm
// partials of the block output's BatchNorm in `bp.part` (chunk k: sum g and
// sum g (z - mean), g = dout * [ymask > 0], as bn_group_partial in 64-row
// chunks), so that BatchNorm's backward needs no partials pass.
struct HeadBnArgs {
  const void* ymask;
  const void* z;
  const float* mean;
  float* part;
};

template <typename T, bool BNP>
__global__ __launch_bounds__(256) void head_bwd_kernel(const float* z, const int32_t* labels,
                                                       const int32_t* idx, int N, int J,
                                                       const float* f, const float* W, int I,
                                                       float* dW, float* db, T* dout, int HW,
                                                       float* out, HeadBnArgs bp) {
  constexpr int E = Elt<T>::E;
  const int t = threadIdx.x;
  __shared__ float rdz[256][HEAD_JMAX];
  __shared__ float rl[256];
  __shared__ int rc[256], rb[256];
  float dz[HEAD_JMAX];
  if (blockIdx.x < (unsigned)HEAD_WB) {
    // features i = 64 b + t % 64; samples of each 256-row chunk in 4 slices,
    // the slices added in order
    __shared__ float part[4][HEAD_JMAX][64];
    const int il = t & 63, sl = t >> 6;
    const int i = blockIdx.x * 64 + il;
    float acc[HEAD_JMAX], dsum = 0.f, L = 0.f;
    int C = 0, bad = 0;
#pragma unroll
    for (int j = 0; j < HEAD_JMAX; ++j) acc[j] = 0.f;
    for (int n0 = 0; n0 < N; n0 += 256) {
      const int cnt = min(256, N - n0);
      __syncthreads();
      if (t < cnt) {
        float l;
        int c;
        const bool ok = ce_row(z + (long long)(n0 + t) * J, labels[idx ? idx[n0 + t] : n0 + t], J,
                               N, dz, l, c);
#pragma unroll
        for (int j = 0; j < HEAD_JMAX; ++j) rdz[t][j] = dz[j];
        rl[t] = l;
        rc[t] = c;
        rb[t] = (!ok || !isfinite(l)) ? 1 : 0;
      }
      __syncthreads();
      const int per = (cnt + 3) / 4;
      const int k0 = sl * per, k1 = min(cnt, k0 + per);
      for (int k = k0; k < k1; k += 8) {  // eight samples' features loaded up front
        float fv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q)
          fv[q] = (k + q < k1 && i < I) ? f[(long long)(n0 + k + q) * I + i] : 0.f;
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (k + q < k1)
#pragma unroll
            for (int j = 0; j < HEAD_JMAX; ++j)
              if (j < J) acc[j] += rdz[k + q][j] * fv[q];
      }
      if (blockIdx.x == 0) {  // sample sums in sample order, one quantity per wave
        if (t < J) {
          for (int k = 0; k < cnt; ++k) dsum += rdz[k][t];
        } else if (t == 64) {
          for (int k = 0; k < cnt; ++k) L += rl[k];
        } else if (t == 128) {
          for (int k = 0; k < cnt; ++k) C += rc[k];
        } else if (t == 192) {
          for (int k = 0; k < cnt; ++k) bad |= rb[k];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < HEAD_JMAX; ++j) part[sl][j][il] = acc[j];
    __syncthreads();
    if (sl == 0 && i < I)
      for (int j = 0; j < J; ++j)
        dW[(long long)j * I + i] = ((part[0][j][il] + part[1][j][il]) + part[2][j][il]) + part[3][j][il];
    if (blockIdx.x == 0) {
      if (t < J) db[t] = dsum;
      if (t == 64) out[0] = L / (float)N;
      if (t == 128) out[1] = (float)C;
      if (t == 192) out[2] = (float)bad;
    }
    return;
  }
  if (!dout) return;
  if constexpr (BNP) {
    constexpr int UG = BN_GROUP / E, RI = 256 / UG, RPT = 64 / RI;
    const int G = I / BN_GROUP;
    const long long Mr = (long long)N * HW;
    const int bb = blockIdx.x - HEAD_WB, k = bb / G, cg = bb % G;
    const long long r0 = (long long)k * 64, r1 = std::min<long long>(Mr, r0 + 64);
    if (r0 >= Mr) return;
    const int u = t % UG, rs = t / UG, c0 = cg * BN_GROUP + u * E;
    const T* ymask = reinterpret_cast<const T*>(bp.ymask);
    const T* zb = reinterpret_cast<const T*>(bp.z);
    // the rows' ReLU mask and BatchNorm input, loaded before the softmax rows
    uint4 ym[RPT], zr[RPT];
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const long long r = r0 + rs + (long long)RI * q;
      if (r < r1) {
        ym[q] = *reinterpret_cast<const uint4*>(ymask + r * I + c0);
        zr[q] = *reinterpret_cast<const uint4*>(zb + r * I + c0);
      }
    }
    const int n_lo = (int)(r0 / HW), nsm = (int)((r1 - 1) / HW) - n_lo + 1;  // <= 64 samples
    if (t < nsm) {
      float l;
      int c;
      const int n = n_lo + t;
      ce_row(z + (long long)n * J, labels[idx ? idx[n] : n], J, N, dz, l, c);
#pragma unroll
      for (int j = 0; j < HEAD_JMAX; ++j) rdz[t][j] = dz[j];
    }
    __syncthreads();
    __shared__ float dp[64][BN_GROUP];
    const float inv = 1.f / (float)HW;
    for (int i = t; i < nsm * BN_GROUP; i += 256) {
      const int sm = i / BN_GROUP, c = i % BN_GROUP;
      float d = 0.f;
      for (int j = 0; j < J; ++j) d += rdz[sm][j] * W[(long long)j * I + cg * BN_GROUP + c];
      dp[sm][c] = d * inv;
    }
    __syncthreads();
    float mu[E], s1[E], s2[E];
    chan_load<E>(bp.mean, c0, mu);
#pragma unroll
    for (int e = 0; e < E; ++e) s1[e] = s2[e] = 0.f;
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const long long r = r0 + rs + (long long)RI * q;
      if (r < r1) {
        const int sm = (int)(r / HW) - n_lo;
        float d[E], gs[E], yv[E], zv[E];
#pragma unroll
        for (int e = 0; e < E; ++e) d[e] = dp[sm][u * E + e];
        const uint4 v = f_to_unit<T>(d);
        *reinterpret_cast<uint4*>(dout + r * I + c0) = v;
        unit_to_f<T>(v, gs);
        unit_to_f<T>(ym[q], yv);
        unit_to_f<T>(zr[q], zv);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float g = yv[e] > 0.f ? gs[e] : 0.f;
          s1[e] += g;
          s2[e] += g * (zv[e] - mu[e]);
        }
      }
    }
    __shared__ float red[2][RI][BN_GROUP];  // row slices added in slice order
#pragma unroll
    for (int e = 0; e < E; ++e) {
      red[0][rs][u * E + e] = s1[e];
      red[1][rs][u * E + e] = s2[e];
    }
    __syncthreads();
    if (t < BN_GROUP) {
      float a = 0.f, b = 0.f;
      for (int q = 0; q < RI; ++q) {
        a += red[0][q][t];
        b += red[1][q][t];
      }
      bp.part[(long long)k * 2 * I + cg * BN_GROUP + t] = a;
      bp.part[(long long)k * 2 * I + I + cg * BN_GROUP + t] = b;
    }
    return;
  }
  const int nchunk = (HW + HEAD_PC - 1) / HEAD_PC;
  const int bb = blockIdx.x - HEAD_WB, n = bb / nchunk, pc = bb % nchunk;
  if (n >= N) return;
  if (t == 0) {
    float l;
    int c;
    ce_row(z + (long long)n * J, labels[idx ? idx[n] : n], J, N, dz, l, c);
#pragma unroll
    for (int j = 0; j < HEAD_JMAX; ++j) rdz[0][j] = dz[j];
  }
  __syncthreads();
  const int units = I / E, u = t % units, ps = t / units, nsl = 256 / units;
  const float inv = 1.f / (float)HW;
  float d[E];
#pragma unroll
  for (int e = 0; e < E; ++e) d[e] = 0.f;
#pragma unroll
  for (int j = 0; j < HEAD_JMAX; ++j)
    if (j < J) {
      const float w = rdz[0][j];
      float wv[E];
      chan_load<E>(W + (long long)j * I, u * E, wv);
#pragma unroll
      for (int e = 0; e < E; ++e) d[e] += w * wv[e];
    }
#pragma unroll
  for (int e = 0; e < E; ++e) d[e] *= inv;
  const uint4 v = f_to_unit<T>(d);
  const int p1 = min(HW, (pc + 1) * HEAD_PC);
  for (int p = pc * HEAD_PC + ps; p < p1; p += nsl)
    reinterpret_cast<uint4*>(dout + ((long long)n * HW + p) * I)[u] = v;
}

__global__ __launch_bounds__(256) void count_correct_kernel(const float* z, const int32_t* labels,
                                                            int N, int J, int32_t* count) {
  __shared__ int sc[256];
  int c = 0;
  for (int n = threadIdx.x; n < N; n += 256) {
    const float* zr = z + (long long)n * J;
    float m = zr[0];
    int am = 0;
    for (int j = 1; j < J; ++j)
      if (zr[j] > m) {
        m = zr[j];
        am = j;
      }
    c += (am == labels[n]);
  }
  sc[threadIdx.x] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int t = 0; t < 256; ++t) s += sc[t];
    *count += s;
  }
}

__global__ void argmax_kernel(const float* z, int N, int J, int32_t* out) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const float* zr = z + (long long)n * J;
  float m = zr[0];
  int am = 0;
  for (int j = 1; j < J; ++j)
    if (zr[j] > m) {
      m = zr[j];
      am = j;
    }
  out[n] = am;
}

// --------------------------------------------------------------- optimiser
__global__ void sgd_kernel(float* w, float* v, const float* g, long long n, float lr, float mu) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    const float vn = mu * v[i] + g[i];
    v[i] = vn;
    w[i] = w[i] - lr * vn;
  }
}

// ----------------------------------------------------------- data movement
__global__ void gather_rows_kernel(const uint4* src, const int32_t* idx, int n, long long row_units,
                                   uint4* dst) {
  const long long total = (long long)n * row_units;
  for (long long t = blockIdx.x * (long long)blockDim.x + threadIdx.x; t < total;
       t += (long long)gridDim.x * blockDim.x) {
    const long long r = t / row_units, u = t % row_units;
    const long long sr = idx ? idx[r] : r;
    dst[t] = src[sr * row_units + u];
  }
}

template <typename T>
__global__ void frames_to_padded_kernel(const T* src, const int32_t* idx, int n, long long hw,
                                        int Cp, T* dst) {
  const long long total = (long long)n * hw;
  for (long long t = blockIdx.x * (long long)blockDim.x + threadIdx.x; t < total;
       t += (long long)gridDim.x * blockDim.x) {
    const long long f = t / hw, p = t % hw;
    const long long sf = idx ? idx[f] : f;
    const T* s = src + (sf * hw + p) * 3;
    T* d = dst + t * Cp;
    for (int c = 0; c < Cp; ++c) d[c] = c < 3 ? s[c] : from_f<T>(0.f);
  }
}

// 2-byte elements, 8 stored channels, an even pixel count per frame: a lane
// expands two adjacent pixels (three dwords of 3-channel input, 4-byte
// aligned) into two 16-byte pixels; blockIdx.y is the frame.
__global__ void frames_to_padded8_kernel(const uint32_t* src, const int32_t* idx, int pairs,
                                         uint4* dst) {
  const int f = blockIdx.y;
  const long long sf = idx ? idx[f] : f;
  const uint32_t* s = src + sf * pairs * 3;
  uint4* d = dst + (long long)f * pairs * 2;
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < pairs; t += gridDim.x * blockDim.x) {
    const uint32_t a = s[3 * t], b = s[3 * t + 1], c = s[3 * t + 2];
    d[2 * t] = make_uint4(a, b & 0xFFFFu, 0u, 0u);
    d[2 * t + 1] = make_uint4((b >> 16) | (c << 16), c >> 16, 0u, 0u);
  }
}

__device__ __forceinline__ void src_coord(int dst, int n_in, int n_out, int& i0, int& i1,
                                          float& lam) {
  float s = ((float)dst + 0.5f) * ((float)n_in / (float)n_out) - 0.5f;
  if (s < 0.f) s = 0.f;
  i0 = min((int)floorf(s), n_in - 1);
  i1 = min(i0 + 1, n_in - 1);
  lam = s - (float)i0;
}

template <typename T>
__global__ void resize_kernel(const T* src, int n, int H, int W, int r, int Cp, T* dst) {
  const long long total = (long long)n * r * r;
  for (long long t = blockIdx.x * (long long)blockDim.x + threadIdx.x; t < total;
       t += (long long)gridDim.x * blockDim.x) {
    const int ox = (int)(t % r), oy = (int)((t / r) % r);
    const long long f = t / ((long long)r * r);
    int y0, y1, x0, x1;
    float ly, lx;
    src_coord(oy, H, r, y0, y1, ly);
    src_coord(ox, W, r, x0, x1, lx);
    const T* s = src + f * H * W * 3;
    T* d = dst + t * Cp;
    for (int c = 0; c < Cp; ++c) {
      if (c >= 3) {
        d[c] = from_f<T>(0.f);
        continue;
      }
      const float a = to_f(s[((long long)y0 * W + x0) * 3 + c]);
      const float b = to_f(s[((long long)y0 * W + x1) * 3 + c]);
      const float cc = to_f(s[((long long)y1 * W + x0) * 3 + c]);
      const float dd = to_f(s[((long long)y1 * W + x1) * 3 + c]);
      const float top0 = a * (1.f - ly) + cc * ly;   // rows first, then columns
      const float top1 = b * (1.f - ly) + dd * ly;
      d[c] = from_f<T>(top0 * (1.f - lx) + top1 * lx);
    }
  }
}

template <typename T>
__global__ void cast_kernel(const float* src, long long n, T* dst) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    dst[i] = from_f<T>(src[i]);
}

// ------------------------------------------------------- weight repacking
// tab row: src_off, K, R, S, C0, Cp, krsc_off, crsk_off.  Both copies are
// written in their own element order (coalesced); the [C][R][S][K] copy reads
// the fp32 master with a stride.
// One 64 x 64 tile (output channels k x input channels c) of one tap (r, s)
// of a conv per iteration: the fp32 master tile is read once along c, the
// [K][R][S][Cp] copy written along c and, through LDS, the [C][R][S][K] copy
// along k -- every global access coalesced.
// tab row: master offset, K, R, S, C0, Cp, krsc offset, crsk offset (-1: none)
template <typename T>
__global__ __launch_bounds__(256) void pack_conv_kernel(const float* master, const long long* tab,
                                                        T* shadow) {
  const long long* t = tab + 8 * blockIdx.y;
  const int K = (int)t[1], RS = (int)(t[2] * t[3]), C0 = (int)t[4], Cp = (int)t[5];
  const float* src = master + t[0];
  T* krsc = shadow + t[6];
  T* crsk = t[7] >= 0 ? shadow + t[7] : nullptr;
  const int tk = cdiv(K, 64), tc = cdiv(Cp, 64);
  const int ntiles = RS * tk * tc;
  const int cc = threadIdx.x & 63, kr = threadIdx.x >> 6;
  __shared__ float tile[64][65];
  for (int bt = blockIdx.x; bt < ntiles; bt += gridDim.x) {
    const int rs = bt / (tk * tc), rem = bt % (tk * tc);
    const int k0 = (rem / tc) * 64, c0 = (rem % tc) * 64;
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
      const int k = k0 + kr + 4 * i, c = c0 + cc;
      const float v = (k < K && c < C0) ? src[((long long)k * RS + rs) * C0 + c] : 0.f;
      tile[kr + 4 * i][cc] = v;
      if (k < K && c < Cp) krsc[((long long)k * RS + rs) * Cp + c] = from_f<T>(v);
    }
    if (crsk) {
      __syncthreads();
#pragma unroll 4
      for (int i = 0; i < 16; ++i) {
        const int c = c0 + kr + 4 * i, k = k0 + cc;
        if (c < C0 && k < K) crsk[((long long)c * RS + rs) * K + k] = from_f<T>(tile[cc][kr + 4 * i]);
      }
    }
    __syncthreads();
  }
}

// Momentum SGD of one convolution's weights from its weight-gradient split
// partials, and its low-precision copies.  A block takes 16 output x 64 input
// channels of one filter tap, 4 elements per thread: g = sum of the splits in
// split order (as the separate reduction adds them), loads four splits ahead;
// v = mu v + g, w = w - lr v on the fp32 [K][RS][C] master, then the
// [K][RS][C] copy directly and the [C][RS][K] copy through an LDS transpose.
constexpr int UPD_K = 16;
// Splits a split-group pass adds up before the momentum step (above it).
constexpr int UPD_GROUP = 16;
template <typename T>
__global__ __launch_bounds__(256) void conv_update_kernel(const float* part, int splits, int K,
                                                          int RS, int C, float* w, float* v,
                                                          float lr, float mu, T* krsc, T* crsk) {
  const int tk = K / UPD_K, tc = C / 64;
  const int ntiles = RS * tk * tc;
  const long long stride = (long long)K * RS * C;
  const int cc = threadIdx.x & 63, kr = threadIdx.x >> 6;
  __shared__ float tile[UPD_K][65];
  for (int bt = blockIdx.x; bt < ntiles; bt += gridDim.x) {
    const int rs = bt / (tk * tc), rem = bt % (tk * tc);
    const int k0 = (rem / tc) * UPD_K, c0 = (rem % tc) * 64;
    int o[4];
    float g[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[i] = ((k0 + kr + 4 * i) * RS + rs) * C + c0 + cc;
      g[i] = 0.f;
    }
    for (int sp = 0; sp < splits; sp += 4) {
      float t[4][4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) t[q][i] = sp + q < splits ? part[(sp + q) * stride + o[i]] : 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (sp + q < splits) g[i] += t[q][i];
    }
    float vv[4], ww[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      vv[i] = v[o[i]];
      ww[i] = w[o[i]];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float vn = mu * vv[i] + g[i];
      const float wn = ww[i] - lr * vn;
      v[o[i]] = vn;
      w[o[i]] = wn;
      krsc[o[i]] = from_f<T>(wn);
      tile[kr + 4 * i][cc] = wn;
    }
    __syncthreads();
    // [C][RS][K]: thread -> input channel c0 + t / 4, output channels 4 (t % 4) .. + 3
    const int c = c0 + (threadIdx.x >> 2), kq = (threadIdx.x & 3) * 4;
    T* dst = crsk + ((long long)c * RS + rs) * K + k0 + kq;
#pragma unroll
    for (int i = 0; i < 4; ++i) dst[i] = from_f<T>(tile[kq + i][c - c0]);
    __syncthreads();
  }
}

// SGD with momentum over the ranges (offset, length) of a table, one range per
// blockIdx.y.
__global__ void sgd_ranges_kernel(float* w, float* v, const float* g, const long long* tab,
                                  float lr, float mu) {
  const long long off = tab[2 * blockIdx.y], n = tab[2 * blockIdx.y + 1];
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    const long long o = off + i;
    const float vn = mu * v[o] + g[o];
    v[o] = vn;
    w[o] = w[o] - lr * vn;
  }
}

// tab row: off, K, C, R, S
__global__ void permute_kernel(const float* src, float* dst, const long long* tab, int ntab,
                               long long total, int to_internal) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    int lo = 0, hi = ntab - 1;  // last row with off <= i
    while (lo < hi) {
      int mid = (lo + hi + 1) >> 1;
      if (tab[5 * mid] <= i) lo = mid; else hi = mid - 1;
    }
    const long long* t = tab + 5 * lo;
    const long long off = t[0], l = i - off;
    const int C = (int)t[2], R = (int)t[3], S = (int)t[4];
    if (R * S * C == 1 || (R == 1 && S == 1)) {  // no reordering needed
      dst[i] = src[i];
      continue;
    }
    if (to_internal) {
      // l indexes [K][C][R][S]; destination [K][R][S][C]
      const int s = (int)(l % S), r = (int)((l / S) % R), c = (int)((l / ((long long)S * R)) % C);
      const long long k = l / ((long long)S * R * C);
      dst[off + ((k * R + r) * S + s) * C + c] = src[i];
    } else {
      // l indexes [K][R][S][C]; destination [K][C][R][S]
      const int c = (int)(l % C), s = (int)((l / C) % S), r = (int)((l / ((long long)C * S)) % R);
      const long long k = l / ((long long)C * S * R);
      dst[off + ((k * C + c) * R + r) * S + s] = src[i];
    }
  }
}

template <typename F>
hipError_t by_type(int dt, F&& f) {
  if (dt == DT_F32) f((float*)nullptr); else f((bf16*)nullptr);
  return hipGetLastError();
}

}  // namespace

// Room for every chunking that writes partials of an M x C BatchNorm: the
// large-M path (bn_chunks), and -- where the two-launch path applies (at most
// BN_FOLD_MAX_CHUNKS chunks of BN_FOLD_ROWS rows) -- the 128-row chunks of its
// partial kernel and the 64-row chunks GEMM epilogues and the classifier-head
// backward leave; plus the per-channel coefficients of the large-M backward.
size_t bn_partials_floats(long long M, int C) {
  long long ch = bn_chunks(M, C);
  if (bn_fold_ok(M, C)) ch = std::max(ch, cdivl(M, 64));
  return (size_t)ch * 2 * C + 3 * C;
}

hipError_t bn_train_stats(int dt, const void* z, long long M, int C, const float* gamma,
                          const float* beta, float* rm, float* rv, float* mean, float* invstd,
                          float* scale, float* shift, float* partials, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int nch = bn_chunks(M, C);
  const long long rpc = cdivl(M, nch);
  return by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(bn_stats_partial<T>, dim3(nch), dim3(256), 0, stream, (const T*)z, M, C,
                       rpc, partials);
    hipLaunchKernelGGL(bn_stats_final<T>, dim3(cdiv(C, FIN_CH)), dim3(256), 0, stream, (const T*)z,
                       partials, nch, M, C, gamma, beta, rm, rv, mean, invstd, scale, shift);
  });
}

bool bn_fold_path(long long M, int C) { return bn_fold_ok(M, C); }

hipError_t split_reduce_bn(int dt, const float* part, int splits, long long M, int C,
                           const void* res, void* out, const BnStatsSink& sink,
                           hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (!bn_fold_ok(M, C) || splits < 1 || !sink.part ||
      (sink.bwd && (!sink.z || !sink.mean)))
    return hipErrorInvalidValue;
  const dim3 grid((unsigned)cdivl(M, BN_FOLD_ROWS), C / BN_GROUP);
  const double act = (double)M * C * dtype_size(dt);
  // fp32 partials of every split read, the sum written; the backward variant
  // also reads the ReLU mask and the BatchNorm input (and a residual)
  const double bytes = (double)M * C * 4 * splits + act * (1 + (res ? 1 : 0) + (sink.bwd ? 2 : 0));
  TimedLaunch tl(stream);
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    if (sink.bwd)
      hipLaunchKernelGGL((split_bn_kernel<T, true>), grid, dim3(1024), 0, stream, part, splits, M,
                         C, (const T*)res, (T*)out, (const T*)sink.ymask, (const T*)sink.z,
                         sink.mean, sink.part);
    else
      hipLaunchKernelGGL((split_bn_kernel<T, false>), grid, dim3(1024), 0, stream, part, splits, M,
                         C, (const T*)res, (T*)out, (const T*)nullptr, (const T*)nullptr,
                         (const float*)nullptr, sink.part);
  }), "split_reduce_bn", bytes);
}

hipError_t bn_train_forward(int dt, const void* z, long long M, int C, const float* gamma,
                            const float* beta, float* rm, float* rv, float* mean, float* invstd,
                            float* scale, float* shift, const void* res, int relu, void* y,
                            float* partials, hipStream_t stream, int ready_rows) {
  if (M == 0) return hipSuccess;
  if (ready_rows != 0 && ((ready_rows != 64 && ready_rows != BN_FOLD_ROWS) || !bn_fold_ok(M, C)))
    return hipErrorInvalidValue;
  const double act = (double)M * C * dtype_size(dt);  // bytes of one activation tensor
  if (!bn_fold_ok(M, C)) {
    TimedLaunch ts(stream);
    hipError_t e = ts.done(bn_train_stats(dt, z, M, C, gamma, beta, rm, rv, mean, invstd, scale,
                                          shift, partials, stream),
                           "bn_fwd_stats", act);
    if (e != hipSuccess) return e;
    TimedLaunch ta(stream);
    return ta.done(bn_apply(dt, z, M, C, mean, scale, beta, res, relu, y, stream), "bn_fwd_apply",
                   act * (res ? 3 : 2));
  }
  const int crows = ready_rows ? ready_rows : BN_FOLD_ROWS;
  const int nch = (int)cdivl(M, crows), groups = C / BN_GROUP;
  const long long rpb = bn_fold_rpb(M, C, dt);
  if (!ready_rows) {
    TimedLaunch tp_(stream);
    hipError_t e = tp_.done(by_type(dt, [&](auto* tp) {
      using T = std::remove_pointer_t<decltype(tp)>;
      hipLaunchKernelGGL((bn_group_partial<T, false>), dim3(nch, groups), dim3(256), 0, stream,
                         (const T*)z, (const T*)nullptr, (const T*)nullptr, (const float*)nullptr,
                         (const float*)nullptr, (const float*)nullptr, (const float*)nullptr, M, C,
                         partials);
    }), "bn_fwd_stats", act);
    if (e != hipSuccess) return e;
  }
  TimedLaunch ta(stream);
  return ta.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(bn_fold_apply<T>, dim3((unsigned)cdivl(M, rpb), groups), dim3(256), 0,
                       stream, (const T*)z, partials, nch, crows, M, C, rpb, gamma, beta, rm, rv, mean,
                       invstd, scale, shift, (const T*)res, relu, (T*)y);
  }), "bn_fwd_apply", act * (res ? 3 : 2));
}

hipError_t bn_apply(int dt, const void* z, long long M, int C, const float* mean,
                    const float* scale, const float* beta, const void* res, int relu, void* y,
                    hipStream_t stream) {
  const long long units = M * C / dtype_vec(dt);
  if (units == 0) return hipSuccess;
  return by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    const int grid = grid_for(units, 256 * BN_AU);
    const int upr = C / Elt<T>::E;  // units per row
    if ((256LL * grid) % upr == 0)
      hipLaunchKernelGGL((bn_apply_kernel<T, true>), dim3(grid), dim3(256), 0, stream, (const T*)z,
                         units, C, mean, scale, beta, (const T*)res, relu, (T*)y);
    else
      hipLaunchKernelGGL((bn_apply_kernel<T, false>), dim3(grid), dim3(256), 0, stream,
                         (const T*)z, units, C, mean, scale, beta, (const T*)res, relu, (T*)y);
  });
}

hipError_t bn_fold(const float* params, const long long* tab, int n, float* out,
                   hipStream_t stream) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(bn_fold_kernel, dim3(n), dim3(256), 0, stream, params, tab, out);
  return hipGetLastError();
}

hipError_t bn_backward(int dt, const void* dy, const void* y, const void* z, long long M, int C,
                       const float* gamma, const float* mean, const float* invstd, float* dgamma,
                       float* dbeta, void* dz, void* g_out, float* partials, hipStream_t stream,
                       int ready_rows, const float* relu_beta) {
  if (M == 0) return hipSuccess;
  if (y && relu_beta) return hipErrorInvalidValue;
  if (ready_rows != 0 && ((ready_rows != 64 && ready_rows != BN_FOLD_ROWS) || !bn_fold_ok(M, C)))
    return hipErrorInvalidValue;
  const double act = (double)M * C * dtype_size(dt);
  // reads dy, z (and y), writes dz (and g)
  const double apply_bytes = act * (3 + (y ? 1 : 0) + (g_out ? 1 : 0));
  if (bn_fold_ok(M, C)) {
    const int nf = (int)cdivl(M, ready_rows ? ready_rows : BN_FOLD_ROWS), groups = C / BN_GROUP;
    const long long rpb = bn_fold_rpb(M, C, dt);
    if (!ready_rows) {
      TimedLaunch tp_(stream);
      hipError_t e = tp_.done(by_type(dt, [&](auto* tp) {
        using T = std::remove_pointer_t<decltype(tp)>;
        hipLaunchKernelGGL((bn_group_partial<T, true>), dim3(nf, groups), dim3(256), 0, stream,
                           (const T*)z, (const T*)dy, (const T*)y, mean, gamma, invstd, relu_beta,
                           M, C, partials);
      }), "bn_bwd_stats", act * (y ? 3 : 2));
      if (e != hipSuccess) return e;
    }
    TimedLaunch ta(stream);
    return ta.done(by_type(dt, [&](auto* tp) {
      using T = std::remove_pointer_t<decltype(tp)>;
      hipLaunchKernelGGL(bn_bwd_fold_apply<T>, dim3((unsigned)cdivl(M, rpb), groups), dim3(256), 0,
                         stream, (const T*)dy, (const T*)y, (const T*)z, partials, nf, M, C, rpb,
                         gamma, mean, invstd, relu_beta, dgamma, dbeta, (T*)dz, (T*)g_out);
    }), "bn_bwd_apply", apply_bytes);
  }
  const int nch = bn_chunks(M, C);
  const long long rpc = cdivl(M, nch);
  float* coef = partials + (size_t)nch * 2 * C;
  const long long units = M * C / dtype_vec(dt);
  TimedLaunch ts(stream);
  hipError_t e = ts.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(bn_bwd_partial<T>, dim3(nch), dim3(256), 0, stream, (const T*)dy,
                       (const T*)y, (const T*)z, M, C, rpc, mean, gamma, invstd, relu_beta,
                       partials);
    hipLaunchKernelGGL(bn_bwd_final, dim3(cdiv(C, FIN_CH)), dim3(256), 0, stream, partials, nch, M, C,
                       gamma, invstd, dgamma, dbeta, coef);
  }), "bn_bwd_stats", act * (y ? 3 : 2));
  if (e != hipSuccess) return e;
  TimedLaunch ta(stream);
  return ta.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    const int grid = grid_for(units, 256 * BN_AU);
    const int upr = C / Elt<T>::E;  // units per row
    if ((256LL * grid) % upr == 0)
      hipLaunchKernelGGL((bn_bwd_apply<T, true>), dim3(grid), dim3(256), 0, stream, (const T*)dy,
                         (const T*)y, (const T*)z, units, C, mean, coef, gamma, invstd, relu_beta,
                         (T*)dz, (T*)g_out);
    else
      hipLaunchKernelGGL((bn_bwd_apply<T, false>), dim3(grid), dim3(256), 0, stream, (const T*)dy,
                         (const T*)y, (const T*)z, units, C, mean, coef, gamma, invstd, relu_beta,
                         (T*)dz, (T*)g_out);
  }), "bn_bwd_apply", apply_bytes);
}

bool bn_backward_pool_ok(int C, int H, int W) {
  return C == POOLBN_C && W <= 2 * POOLBN_QMAX && H >= 1 && W >= 1;
}

hipError_t bn_backward_pool_stats(int dt, const void* dy_pool, const uint8_t* arg, const void* z,
                                  int N, int H, int W, int C, const float* gamma, const float* beta,
                                  const float* mean, const float* invstd, float* dgamma,
                                  float* dbeta, float* partials, const float** coef_out,
                                  hipStream_t stream) {
  const long long M = (long long)N * H * W;
  *coef_out = partials;
  if (M == 0) return hipSuccess;
  if (M >= (1LL << 31) || !bn_backward_pool_ok(C, H, W)) return hipErrorInvalidValue;
  const int P = (H - 1) / 2 + 1, Q = (W - 1) / 2 + 1;
  const PoolSrc ps{dy_pool, arg, H, W, P, Q};
  const int pairs = N * P;
  // at most as many partial rows as bn_partials_floats(M, C) provides
  const int rp = cdiv(pairs, bn_chunks(M, C)), nch = cdiv(pairs, rp);
  float* coef = partials + (size_t)nch * 2 * C;
  *coef_out = coef;
  const size_t es = dtype_size(dt);
  const double act = (double)M * C * es, pooled = (double)N * P * Q * C * (es + 1);
  TimedLaunch ts(stream);  // z; the pooled gradient and its window indices
  return ts.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL((bn_bwd_pool_kernel<T, true>), dim3(nch), dim3(256), 0, stream, ps,
                       (const T*)z, N, rp, mean, (const float*)nullptr, gamma, invstd, beta,
                       partials, (T*)nullptr);
    hipLaunchKernelGGL(bn_bwd_final, dim3(cdiv(C, FIN_CH)), dim3(256), 0, stream, partials, nch, M, C,
                       gamma, invstd, dgamma, dbeta, coef);
  }), "bn_bwd_pool_stats", act + pooled);
}

hipError_t bn_backward_pool(int dt, const void* dy_pool, const uint8_t* arg, const void* z, int N,
                            int H, int W, int C, const float* gamma, const float* beta,
                            const float* mean, const float* invstd, float* dgamma, float* dbeta,
                            void* dz, float* partials, hipStream_t stream) {
  const long long M = (long long)N * H * W;
  if (M == 0) return hipSuccess;
  const float* coef = nullptr;
  hipError_t e = bn_backward_pool_stats(dt, dy_pool, arg, z, N, H, W, C, gamma, beta, mean, invstd,
                                        dgamma, dbeta, partials, &coef, stream);
  if (e != hipSuccess) return e;
  const int P = (H - 1) / 2 + 1, Q = (W - 1) / 2 + 1;
  const PoolSrc ps{dy_pool, arg, H, W, P, Q};
  const int pairs = N * P;
  const size_t es = dtype_size(dt);
  const double act = (double)M * C * es, pooled = (double)N * P * Q * C * (es + 1);
  TimedLaunch ta(stream);  // z and the pooled gradient read, dz written
  return ta.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL((bn_bwd_pool_kernel<T, false>), dim3(pairs), dim3(256), 0, stream, ps,
                       (const T*)z, N, 1, mean, coef, gamma, invstd, beta, (float*)nullptr, (T*)dz);
  }), "bn_bwd_pool_apply", 2 * act + pooled);
}

hipError_t maxpool_fwd(int dt, const void* x, int N, int H, int W, int C, void* y, uint8_t* arg,
                       hipStream_t stream) {
  const int P = (H - 1) / 2 + 1, Q = (W - 1) / 2 + 1;
  const long long units = (long long)N * P * Q * C / dtype_vec(dt);
  if (units == 0) return hipSuccess;
  const size_t es = dtype_size(dt);
  TimedLaunch tl(stream);  // input once; output (and its window index)
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    const int bpr = cdiv(Q * (C / Elt<T>::E), 256);
    hipLaunchKernelGGL(maxpool_fwd_kernel<T>, dim3((unsigned)((long long)N * ((P + 1) / 2) * bpr)),
                       dim3(256), 0,
                       stream, (const T*)x, N, H, W, C, P, Q, bpr, (T*)y, arg,
                       (const float*)nullptr, (const float*)nullptr, (const float*)nullptr);
  }), "maxpool_fwd", (double)N * C * ((double)H * W * es + (double)P * Q * (es + (arg ? 1 : 0))));
}

hipError_t bn_relu_maxpool_train(int dt, const void* z, int N, int H, int W, int C,
                                 const float* gamma, const float* beta, float* rm, float* rv,
                                 float* mean, float* invstd, float* scale, float* shift,
                                 float* partials, void* y, uint8_t* arg, hipStream_t stream) {
  const long long M = (long long)N * H * W;
  if (M == 0) return hipSuccess;
  const int P = (H - 1) / 2 + 1, Q = (W - 1) / 2 + 1;
  const size_t es = dtype_size(dt);
  TimedLaunch ts(stream);
  hipError_t e = ts.done(bn_train_stats(dt, z, M, C, gamma, beta, rm, rv, mean, invstd, scale,
                                        shift, partials, stream),
                         "bn_fwd_stats", (double)M * C * es);
  if (e != hipSuccess) return e;
  TimedLaunch tl(stream);  // BatchNorm input once; pooled output and its window index
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    const int bpr = cdiv(Q * (C / Elt<T>::E), 256);
    hipLaunchKernelGGL((maxpool_fwd_kernel<T, true>), dim3((unsigned)((long long)N * ((P + 1) / 2) * bpr)),
                       dim3(256), 0, stream, (const T*)z, N, H, W, C, P, Q, bpr, (T*)y, arg, mean,
                       scale, beta);
  }), "bn_relu_maxpool", (double)N * C * ((double)H * W * es + (double)P * Q * (es + (arg ? 1 : 0))));
}

hipError_t maxpool_bwd(int dt, const void* dy, const uint8_t* arg, int N, int H, int W, int C,
                       void* dx, hipStream_t stream) {
  const int P = (H - 1) / 2 + 1, Q = (W - 1) / 2 + 1;
  const long long units = (long long)N * H * W * C / dtype_vec(dt);
  if (units == 0) return hipSuccess;
  const size_t es = dtype_size(dt);
  TimedLaunch tl(stream);  // output gradient and window index once; input gradient
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    const int bpr = cdiv(W * (C / Elt<T>::E), 256);
    hipLaunchKernelGGL(maxpool_bwd_kernel<T>, dim3((unsigned)((long long)N * H * bpr)), dim3(256), 0,
                       stream, (const T*)dy, arg, N, H, W, C, P, Q, bpr, (T*)dx);
  }), "maxpool_bwd", (double)N * C * ((double)P * Q * (es + 1) + (double)H * W * es));
}

hipError_t avgpool_fwd(int dt, const void* x, int N, int HW, int C, float* f, hipStream_t stream) {
  const long long n = (long long)N * C;
  if (n == 0) return hipSuccess;
  return by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(avgpool_fwd_kernel<T>, dim3(grid_for(n)), dim3(256), 0, stream, (const T*)x,
                       N, HW, C, f);
  });
}

hipError_t avgpool_bwd(int dt, const float* df, int N, int HW, int C, void* dx,
                       hipStream_t stream) {
  const long long n = (long long)N * HW * C;
  if (n == 0) return hipSuccess;
  return by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(avgpool_bwd_kernel<T>, dim3(grid_for(n)), dim3(256), 0, stream, df, N, HW,
                       C, (T*)dx);
  });
}

hipError_t fc_fwd(const float* f, const float* W, const float* b, int N, int I, int J, float* z,
                  hipStream_t stream) {
  if (N == 0) return hipSuccess;
  hipLaunchKernelGGL(fc_fwd_kernel, dim3(N), dim3(256), 0, stream, f, W, b, N, I, J, z);
  return hipGetLastError();
}

hipError_t softmax_ce(const float* z, const int32_t* labels, const int32_t* idx, int N, int J,
                      float* dz, float* out, hipStream_t stream) {
  hipLaunchKernelGGL(softmax_ce_kernel, dim3(1), dim3(256), 0, stream, z, labels, idx, N, J, dz,
                     out);
  return hipGetLastError();
}

hipError_t fc_bwd(const float* dz, const float* f, const float* W, int N, int I, int J, float* dW,
                  float* db, float* df, hipStream_t stream) {
  hipLaunchKernelGGL(fc_bwd_w_kernel, dim3(cdiv(J * I, 256)), dim3(256), 0, stream, dz, f, N, I, J,
                     dW, db);
  if (df) {
    hipLaunchKernelGGL(fc_bwd_x_kernel, dim3(grid_for((long long)N * I)), dim3(256), 0, stream, dz,
                       W, N, I, J, df);
  }
  return hipGetLastError();
}

hipError_t head_forward(int dt, const void* x, int HW, const float* f, const float* W,
                        const float* b, int N, int I, int J, float* pooled, float* z,
                        hipStream_t stream) {
  if (N == 0) return hipSuccess;
  if (I > 2048 || I % dtype_vec(dt) != 0) return hipErrorInvalidValue;
  TimedLaunch tl(stream);
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    if (I <= 512)  // ResNet18's 512 features: 16 waves per sample
      hipLaunchKernelGGL((head_fwd_kernel<T, 16, 512>), dim3(N), dim3(1024), 0, stream,
                         (const T*)x, HW, f, W, b, I, J, pooled, z);
    else
      hipLaunchKernelGGL((head_fwd_kernel<T, 4, 2048>), dim3(N), dim3(256), 0, stream,
                         (const T*)x, HW, f, W, b, I, J, pooled, z);
  }), "head_fwd", x ? (double)N * HW * I * dtype_size(dt) : (double)N * I * 4);
}

bool head_backward_fused(int J, int I) { return J <= HEAD_JMAX && I <= 64 * HEAD_WB; }

hipError_t head_backward(int dt, const float* z, const int32_t* labels, const int32_t* idx, int N,
                         int J, const float* f, const float* W, int I, float* dW, float* db,
                         void* dout, int HW, float* out, hipStream_t stream, HeadBnSink* bn) {
  if (bn) bn->rows = 0;
  if (!head_backward_fused(J, I) || I % dtype_vec(dt) != 0 || 256 % (I / dtype_vec(dt)) != 0)
    return hipErrorInvalidValue;
  const long long Mr = (long long)N * HW;
  const bool bnp = dout && bn && bn->ymask && bn->z && bn->mean && bn->part && Mr > 0 &&
                   bn_fold_ok(Mr, I);
  const int dblocks =
      !dout ? 0 : bnp ? (int)cdivl(Mr, 64) * (I / BN_GROUP) : N * cdiv(HW, HEAD_PC);
  const HeadBnArgs ha = bnp ? HeadBnArgs{bn->ymask, bn->z, bn->mean, bn->part}
                            : HeadBnArgs{nullptr, nullptr, nullptr, nullptr};
  // the pooled-feature gradient spread over the block's output (and, with
  // the BatchNorm partials, that block's ReLU mask and BatchNorm input read)
  TimedLaunch tl(stream);
  hipError_t e = tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    if (bnp)
      hipLaunchKernelGGL((head_bwd_kernel<T, true>), dim3(HEAD_WB + dblocks), dim3(256), 0, stream,
                         z, labels, idx, N, J, f, W, I, dW, db, (T*)dout, HW, out, ha);
    else
      hipLaunchKernelGGL((head_bwd_kernel<T, false>), dim3(HEAD_WB + dblocks), dim3(256), 0,
                         stream, z, labels, idx, N, J, f, W, I, dW, db, (T*)dout, HW, out, ha);
  }), "head_bwd", (double)Mr * I * dtype_size(dt) * (bnp ? 3 : 1) + (double)N * I * 4);
  if (e == hipSuccess && bnp) bn->rows = 64;
  return e;
}

hipError_t count_correct(const float* z, const int32_t* labels, int N, int J, int32_t* count,
                         hipStream_t stream) {
  hipLaunchKernelGGL(count_correct_kernel, dim3(1), dim3(256), 0, stream, z, labels, N, J, count);
  return hipGetLastError();
}

hipError_t argmax_rows(const float* z, int N, int J, int32_t* out, hipStream_t stream) {
  if (N == 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(cdiv(N, 256)), dim3(256), 0, stream, z, N, J, out);
  return hipGetLastError();
}

hipError_t sgd_momentum(float* w, float* v, const float* g, long long n, float lr, float mu,
                        hipStream_t stream) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(sgd_kernel, dim3(grid_for(n)), dim3(256), 0, stream, w, v, g, n, lr, mu);
  return hipGetLastError();
}

hipError_t gather_rows(const void* src, const int32_t* idx, int n, long long row_bytes, void* dst,
                       hipStream_t stream) {
  const long long ru = row_bytes / 16;
  if (n == 0 || ru == 0) return hipSuccess;
  TimedLaunch tl(stream);
  hipLaunchKernelGGL(gather_rows_kernel, dim3(grid_for(n * ru)), dim3(256), 0, stream,
                     (const uint4*)src, idx, n, ru, (uint4*)dst);
  return tl.done(hipGetLastError(), "gather_rows", 2.0 * n * row_bytes);
}

hipError_t frames_to_padded(int dt, const void* frames, const int32_t* idx, int n, int H, int W,
                            int Cp, void* dst, hipStream_t stream) {
  const long long hw = (long long)H * W;
  if (n == 0) return hipSuccess;
  TimedLaunch tl(stream);
  const double bytes = (double)n * hw * (3 + Cp) * dtype_size(dt);
  if (dtype_size(dt) == 2 && Cp == 8 && hw % 2 == 0 && hw / 2 <= INT_MAX / 3 &&
      (reinterpret_cast<uintptr_t>(frames) & 3) == 0 && (reinterpret_cast<uintptr_t>(dst) & 15) == 0 &&
      n <= 65535) {
    const int pairs = (int)(hw / 2);
    hipLaunchKernelGGL(frames_to_padded8_kernel, dim3(std::min(cdiv(pairs, 256), 4096), n), dim3(256),
                       0, stream, (const uint32_t*)frames, idx, pairs, (uint4*)dst);
    return tl.done(hipGetLastError(), "frames_to_padded", bytes);
  }
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(frames_to_padded_kernel<T>, dim3(grid_for(n * hw)), dim3(256), 0, stream,
                       (const T*)frames, idx, n, hw, Cp, (T*)dst);
  }), "frames_to_padded", bytes);
}

hipError_t resize_to_padded(int dt, const void* frames, int n, int H, int W, int r, int Cp,
                            void* dst, hipStream_t stream) {
  const long long total = (long long)n * r * r;
  if (total == 0) return hipSuccess;
  TimedLaunch tl(stream);  // every source pixel once, every padded output pixel
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(resize_kernel<T>, dim3(grid_for(total)), dim3(256), 0, stream,
                       (const T*)frames, n, H, W, r, Cp, (T*)dst);
  }), "resize", (double)n * ((double)H * W * 3 + (double)r * r * Cp) * dtype_size(dt));
}

hipError_t cast_from_f32(int dt, const float* src, long long n, void* dst, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  return by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(cast_kernel<T>, dim3(grid_for(n)), dim3(256), 0, stream, src, n, (T*)dst);
  });
}

hipError_t pack_conv_weights(int dt, const float* master, const long long* tab, int n,
                             void* shadow, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  return by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(pack_conv_kernel<T>, dim3(256, n), dim3(256), 0, stream, master, tab,
                       (T*)shadow);
  });
}

// out[g][i] = sum of part[s][i] over the splits s of group g (UPD_GROUP
// consecutive splits, added in split order), four floats per thread.
__global__ __launch_bounds__(256) void split_group_kernel(const float* part, int splits,
                                                          long long n, float* out) {
  const long long n4 = n / 4;
  const int g = blockIdx.y, s0 = g * UPD_GROUP, s1 = min(splits, s0 + UPD_GROUP);
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < n4; i += (long long)gridDim.x * 256) {
    float4 acc = reinterpret_cast<const float4*>(part + (long long)s0 * n)[i];
    for (int s = s0 + 1; s < s1; ++s) {
      const float4 t = reinterpret_cast<const float4*>(part + (long long)s * n)[i];
      acc.x += t.x;
      acc.y += t.y;
      acc.z += t.z;
      acc.w += t.w;
    }
    reinterpret_cast<float4*>(out + (long long)g * n)[i] = acc;
  }
}

int conv_update_groups(int splits) { return splits > UPD_GROUP ? cdiv(splits, UPD_GROUP) : 0; }

hipError_t split_group_sum(const float* part, int splits, long long n, float* out,
                           hipStream_t stream) {
  const int groups = conv_update_groups(splits);
  if (groups == 0 || n % 4 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(split_group_kernel,
                     dim3((unsigned)std::min<long long>(cdivl(n / 4, 256), 1024), groups), dim3(256),
                     0, stream, part, splits, n, out);
  return hipGetLastError();
}

hipError_t conv_weight_update(int dt, const float* part, int splits, int K, int RS, int C,
                              float* w, float* v, float lr, float mu, void* krsc, void* crsk,
                              hipStream_t stream) {
  if (K % 64 != 0 || C % 64 != 0 || splits < 1 || (long long)K * RS * C >= (1LL << 31))
    return hipErrorInvalidValue;
  const int groups = conv_update_groups(splits);
  if (groups > 0) {
    // many splits (the all-taps weight gradient of small convolutions): add
    // them in groups first, spread over the whole GPU, into the scratch
    // after the partials; the momentum step then reads the group sums
    const long long nw = (long long)K * RS * C;
    float* sums = const_cast<float*>(part) + (long long)splits * nw;
    TimedLaunch tg(stream);
    hipLaunchKernelGGL(split_group_kernel,
                       dim3((unsigned)std::min<long long>(cdivl(nw / 4, 256), 1024), groups),
                       dim3(256), 0, stream, part, splits, nw, sums);
    EKYA_HIP(tg.done(hipGetLastError(), "conv_update_group",
                     (double)nw * 4.0 * (splits + groups)));
    part = sums;
    splits = groups;
  }
  const int ntiles = RS * (K / UPD_K) * (C / 64);
  // per weight: the split partials, master and momentum read; master and
  // momentum written, and the two low-precision copies
  const double n = (double)K * RS * C;
  TimedLaunch tl(stream);
  return tl.done(by_type(dt, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    hipLaunchKernelGGL(conv_update_kernel<T>, dim3(std::min(ntiles, 4096)), dim3(256), 0, stream,
                       part, splits, K, RS, C, w, v, lr, mu, (T*)krsc, (T*)crsk);
  }), "conv_update", n * (4.0 * splits + 16 + 2 * dtype_size(dt)));
}

hipError_t sgd_momentum_ranges(float* w, float* v, const float* g, const long long* tab, int n,
                               long long max_len, float lr, float mu, hipStream_t stream) {
  if (n == 0 || max_len == 0) return hipSuccess;
  hipLaunchKernelGGL(sgd_ranges_kernel, dim3(grid_for(max_len, 256, 1024), n), dim3(256), 0, stream,
                     w, v, g, tab, lr, mu);
  return hipGetLastError();
}

hipError_t permute_weights(const float* src, float* dst, const long long* tab, int n,
                           long long total, int to_internal, hipStream_t stream) {
  hipLaunchKernelGGL(permute_kernel, dim3(grid_for(total)), dim3(256), 0, stream, src, dst, tab, n,
                     total, to_internal);
  return hipGetLastError();
}

__global__ void relu_f32_kernel(float* y, const float* x, const float* mask, long long n) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    y[i] = mask ? (mask[i] > 0.f ? x[i] : 0.f) : fmaxf(x[i], 0.f);
}

hipError_t relu_f32(float* y, const float* x, const float* mask, long long n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(relu_f32_kernel, dim3(grid_for(n)), dim3(256), 0, stream, y, x, mask, n);
  return hipGetLastError();
}

// Hardware registers read with s_getreg_b32 (hwreg(id, offset, size) is
// id | offset << 6 | (size - 1) << 11): HW_ID (4) holds the CU in bits 11:8,
// the shader array in bit 12 and the shader engine in bits 14:13; XCC_ID (20)
// the die in bits 3:0.
__global__ void __launch_bounds__(64) cu_ids_kernel(uint32_t* out, int n) {
  const uint32_t hw = __builtin_amdgcn_s_getreg(4 | (0 << 6) | (31 << 11));
  const uint32_t xcc = __builtin_amdgcn_s_getreg(20 | (0 << 6) | (3 << 11));
  // stay resident for about 20 us (wall clock at 100 MHz, at most 2^20
  // polls) so that the workgroups spread over every CU the queue may use
  const uint64_t t0 = wall_clock64();
  for (int i = 0; i < (1 << 20) && wall_clock64() - t0 < 2000; ++i) __builtin_amdgcn_s_sleep(1);
  if (threadIdx.x == 0 && (int)blockIdx.x < n)
    out[blockIdx.x] = (xcc & 15u) << 10 | ((hw >> 12) & 1u) << 8 | ((hw >> 13) & 3u) << 4 |
                      ((hw >> 8) & 15u);
}

hipError_t cu_ids(int n, uint32_t* out, hipStream_t stream) {
  if (n < 1 || n > (1 << 20)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(cu_ids_kernel, dim3(n), dim3(64), 0, stream, out, n);
  return hipGetLastError();
}

}  // namespace ekya
