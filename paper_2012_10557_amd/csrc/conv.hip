// Convolution forward, data-gradient and weight-gradient as implicit GEMMs on
// MFMA (gfx950).  One block-tiled main loop (256 threads, 2 x 2 waves, LDS
// double buffering of 16-byte k-contiguous units) is shared by three operand
// policies:
//   forward : D[k][pix]   = sum_(r,s,c)  w[k][r][s][c]  * x(pix; r,s,c)
//   dgrad   : D[c][pix]   = sum_(r,s,k)  wT[c][r][s][k] * dy(pix; r,s,k)
//   wgrad   : D[rsc][k]   = sum_(pix)    x(pix; rsc)    * dy[pix][k]
// Rows of D are MFMA rows (the lane's four accumulator values are four
// consecutive rows), so forward/dgrad lanes own four consecutive NHWC channels
// and wgrad lanes own four consecutive (r,s,c) entries of one output channel.
#include <algorithm>

#include "kernels.hpp"

namespace ekya {
namespace {

constexpr int NT = 256;

template <typename T> __device__ __forceinline__ void store4(T* dst, const float (&v)[4]);
template <> __device__ __forceinline__ void store4<float>(float* dst, const float (&v)[4]) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
}
template <> __device__ __forceinline__ void store4<bf16>(bf16* dst, const float (&v)[4]) {
  union {
    uint2 u;
    bf16 e[4];
  } p;
#pragma unroll
  for (int i = 0; i < 4; ++i) p.e[i] = (bf16)v[i];
  *reinterpret_cast<uint2*>(dst) = p.u;
}
template <typename T> __device__ __forceinline__ void load4(const T* src, float (&v)[4]);
template <> __device__ __forceinline__ void load4<float>(const float* src, float (&v)[4]) {
  float4 t = *reinterpret_cast<const float4*>(src);
  v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
}
template <> __device__ __forceinline__ void load4<bf16>(const bf16* src, float (&v)[4]) {
  union {
    uint2 u;
    bf16 e[4];
  } p;
  p.u = *reinterpret_cast<const uint2*>(src);
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (float)p.e[i];
}

// ------------------------------------------------------------------ forward
template <typename T> struct FwdArgs {
  ConvGeom g;
  const T* x;
  const T* w;
  T* y;
  ConvEpilogue epi;
};

template <typename T, int BM, int BN>
struct FwdPolicy {
  static constexpr int E = Elt<T>::E;
  static constexpr int KU = 4;
  static constexpr int UA = BM * KU / NT;
  static constexpr int UB = BN * KU / NT;
  using Args = FwdArgs<T>;

  int Ktot, m0, n0;
  const T* arow[UA];
  int au[UA];
  const T* bimg[UB];
  int bh0[UB], bw0[UB], bu[UB];
  bool bok[UB];
  uint4 ra[UA], rb[UB];

  __device__ void init(const Args& a, int m0_, int n0_, int /*split*/) {
    const ConvGeom& g = a.g;
    m0 = m0_;
    n0 = n0_;
    Ktot = g.R * g.S * g.C;
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int q = threadIdx.x + NT * i, row = q / KU;
      au[i] = q % KU;
      int k = m0 + row;
      arow[i] = (k < g.K) ? a.w + (long long)k * Ktot : nullptr;
    }
    const int npix = g.N * g.P * g.Q;
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      int q = threadIdx.x + NT * i, row = q / KU;
      bu[i] = q % KU;
      int pix = n0 + row;
      bok[i] = pix < npix;
      int pp = bok[i] ? pix : 0;
      int n = pp / (g.P * g.Q), rem = pp % (g.P * g.Q);
      int p = rem / g.Q, qq = rem % g.Q;
      bimg[i] = a.x + (long long)n * g.H * g.W * g.C;
      bh0[i] = p * g.stride - g.pad;
      bw0[i] = qq * g.stride - g.pad;
    }
  }
  __device__ int num_stages(const Args&) const { return cdiv(Ktot, KU * E); }
  __device__ void fetch(const Args& a, int st) {
    const ConvGeom& g = a.g;
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int k = st * KU * E + au[i] * E;
      ra[i] = (arow[i] && k < Ktot) ? *reinterpret_cast<const uint4*>(arow[i] + k) : zero_unit();
    }
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      int k = st * KU * E + bu[i] * E;
      uint4 v = zero_unit();
      if (bok[i] && k < Ktot) {
        int c = k % g.C, rs = k / g.C;
        int r = rs / g.S, s = rs % g.S;
        int h = bh0[i] + r, w = bw0[i] + s;
        if (h >= 0 && h < g.H && w >= 0 && w < g.W)
          v = *reinterpret_cast<const uint4*>(bimg[i] + ((long long)h * g.W + w) * g.C + c);
      }
      rb[i] = v;
    }
  }
  template <int PITCH>
  __device__ void commit(uint4* As, uint4* Bs) {
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int q = threadIdx.x + NT * i;
      As[(q / KU) * PITCH + q % KU] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      int q = threadIdx.x + NT * i;
      Bs[(q / KU) * PITCH + q % KU] = rb[i];
    }
  }
  // row = output channel, col = output pixel; v = 4 consecutive channels
  __device__ void out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    if (row >= g.K || col >= g.N * g.P * g.Q) return;
    const ConvEpilogue& e = a.epi;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (e.scale) v[i] *= e.scale[row + i];
      if (e.shift) v[i] += e.shift[row + i];
    }
    long long off = (long long)col * g.K + row;
    if (e.res) {
      float r[4];
      load4<T>(reinterpret_cast<const T*>(e.res) + off, r);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += r[i];
    }
    if (e.relu) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = fmaxf(v[i], 0.0f);
    }
    store4<T>(a.y + off, v);
  }
};

// ------------------------------------------------------------------- dgrad
template <typename T> struct DgradArgs {
  ConvGeom g;
  const T* dy;
  const T* wt;  // [C][R][S][K]
  T* dx;
  const T* res;
};

template <typename T, int BM, int BN>
struct DgradPolicy {
  static constexpr int E = Elt<T>::E;
  static constexpr int KU = 4;
  static constexpr int UA = BM * KU / NT;
  static constexpr int UB = BN * KU / NT;
  using Args = DgradArgs<T>;

  int Ktot, m0, n0;
  const T* arow[UA];
  int au[UA];
  const T* bimg[UB];
  int bh[UB], bw[UB], bu[UB];
  bool bok[UB];
  uint4 ra[UA], rb[UB];

  __device__ void init(const Args& a, int m0_, int n0_, int) {
    const ConvGeom& g = a.g;
    m0 = m0_;
    n0 = n0_;
    Ktot = g.R * g.S * g.K;
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int q = threadIdx.x + NT * i, row = q / KU;
      au[i] = q % KU;
      int c = m0 + row;
      arow[i] = (c < g.C) ? a.wt + (long long)c * Ktot : nullptr;
    }
    const int npix = g.N * g.H * g.W;
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      int q = threadIdx.x + NT * i, row = q / KU;
      bu[i] = q % KU;
      int pix = n0 + row;
      bok[i] = pix < npix;
      int pp = bok[i] ? pix : 0;
      int n = pp / (g.H * g.W), rem = pp % (g.H * g.W);
      bimg[i] = a.dy + (long long)n * g.P * g.Q * g.K;
      bh[i] = rem / g.W + g.pad;
      bw[i] = rem % g.W + g.pad;
    }
  }
  __device__ int num_stages(const Args&) const { return cdiv(Ktot, KU * E); }
  __device__ void fetch(const Args& a, int st) {
    const ConvGeom& g = a.g;
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int k = st * KU * E + au[i] * E;
      ra[i] = (arow[i] && k < Ktot) ? *reinterpret_cast<const uint4*>(arow[i] + k) : zero_unit();
    }
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      int k = st * KU * E + bu[i] * E;
      uint4 v = zero_unit();
      if (bok[i] && k < Ktot) {
        int kk = k % g.K, rs = k / g.K;
        int r = rs / g.S, s = rs % g.S;
        int hp = bh[i] - r, wp = bw[i] - s;
        if (hp >= 0 && wp >= 0 && hp % g.stride == 0 && wp % g.stride == 0) {
          int p = hp / g.stride, q = wp / g.stride;
          if (p < g.P && q < g.Q)
            v = *reinterpret_cast<const uint4*>(bimg[i] + ((long long)p * g.Q + q) * g.K + kk);
        }
      }
      rb[i] = v;
    }
  }
  template <int PITCH>
  __device__ void commit(uint4* As, uint4* Bs) {
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int q = threadIdx.x + NT * i;
      As[(q / KU) * PITCH + q % KU] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      int q = threadIdx.x + NT * i;
      Bs[(q / KU) * PITCH + q % KU] = rb[i];
    }
  }
  __device__ void out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    if (row >= g.C || col >= g.N * g.H * g.W) return;
    long long off = (long long)col * g.C + row;
    if (a.res) {
      float r[4];
      load4<T>(a.res + off, r);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += r[i];
    }
    store4<T>(a.dx + off, v);
  }
};

// ------------------------------------------------------------------- wgrad
// Reduction over output pixels; both operands arrive pixel-major (channels
// contiguous), so each thread loads an E x E block (E pixels x E channels),
// transposes it in registers and writes E k-contiguous units.
template <typename T> struct WgradArgs {
  ConvGeom g;
  const T* x;
  const T* dy;
  float* part;  // [split][K][R*S*C]
  int m_per_split;
};

template <typename T, int BM, int BN>
struct WgradPolicy {
  static constexpr int E = Elt<T>::E;
  static constexpr int KU = E;               // units (of E pixels) per row per stage
  static constexpr int NA = (BM / E) * KU;   // = BM blocks for operand A
  static constexpr int NB = (BN / E) * KU;
  static constexpr int NBLK = (NA + NB + NT - 1) / NT;
  using Args = WgradArgs<T>;

  int m0, n0, mb, me, RSC;
  uint4 rv[NBLK][E];
  // A-block geometry (x side)
  int ar[NBLK], as_[NBLK], ac[NBLK];
  bool aok[NBLK];

  __device__ void init(const Args& a, int m0_, int n0_, int split) {
    const ConvGeom& g = a.g;
    m0 = m0_;
    n0 = n0_;
    RSC = g.R * g.S * g.C;
    const int M = g.N * g.P * g.Q;
    mb = split * a.m_per_split;
    me = min(M, mb + a.m_per_split);
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      int b = threadIdx.x + NT * j;
      aok[j] = false;
      if (b < NA) {
        int rg = b % (BM / E);
        int i0 = m0 + rg * E;
        if (i0 < RSC) {
          aok[j] = true;
          int rs = i0 / g.C;
          ac[j] = i0 % g.C;
          ar[j] = rs / g.S;
          as_[j] = rs % g.S;
        }
      }
    }
  }
  __device__ int num_stages(const Args&) const {
    return me > mb ? cdiv(me - mb, KU * E) : 0;
  }
  __device__ void fetch(const Args& a, int st) {
    const ConvGeom& g = a.g;
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      int b = threadIdx.x + NT * j;
#pragma unroll
      for (int e = 0; e < E; ++e) rv[j][e] = zero_unit();
      if (b < NA) {
        if (!aok[j]) continue;
        int u = b / (BM / E);
        int m = mb + st * KU * E + u * E;
        if (m >= me) continue;
        int PQ = g.P * g.Q;
        int n = m / PQ, rem = m % PQ;
        int p = rem / g.Q, q = rem % g.Q;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if (m + e < me) {
            int h = p * g.stride - g.pad + ar[j], w = q * g.stride - g.pad + as_[j];
            if (h >= 0 && h < g.H && w >= 0 && w < g.W)
              rv[j][e] = *reinterpret_cast<const uint4*>(
                  a.x + (((long long)n * g.H + h) * g.W + w) * g.C + ac[j]);
          }
          if (++q == g.Q) {
            q = 0;
            if (++p == g.P) {
              p = 0;
              ++n;
            }
          }
        }
        transpose_block(rv[j], (T*)nullptr);
      } else if (b < NA + NB) {
        int bb = b - NA;
        int rg = bb % (BN / E), u = bb / (BN / E);
        int k0 = n0 + rg * E;
        int m = mb + st * KU * E + u * E;
        if (k0 >= g.K) continue;
#pragma unroll
        for (int e = 0; e < E; ++e)
          if (m + e < me)
            rv[j][e] = *reinterpret_cast<const uint4*>(a.dy + (long long)(m + e) * g.K + k0);
        transpose_block(rv[j], (T*)nullptr);
      }
    }
  }
  template <int PITCH>
  __device__ void commit(uint4* As, uint4* Bs) {
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      int b = threadIdx.x + NT * j;
      if (b < NA) {
        int rg = b % (BM / E), u = b / (BM / E);
#pragma unroll
        for (int e = 0; e < E; ++e) As[(rg * E + e) * PITCH + u] = rv[j][e];
      } else if (b < NA + NB) {
        int bb = b - NA;
        int rg = bb % (BN / E), u = bb / (BN / E);
#pragma unroll
        for (int e = 0; e < E; ++e) Bs[(rg * E + e) * PITCH + u] = rv[j][e];
      }
    }
  }
  // row = (r,s,c) index, col = output channel k
  __device__ void out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    if (row >= RSC || col >= g.K) return;
    float* dst = a.part + ((long long)blockIdx.z * g.K + col) * RSC + row;
    *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

// ---------------------------------------------------------------- main loop
template <typename T, int BM, int BN, class Pol>
__global__ __launch_bounds__(NT) void gemm_kernel(typename Pol::Args args) {
  constexpr int KU = Pol::KU;
  constexpr int PITCH = KU + 1;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TI = WM / 16, TJ = WN / 16;
  __shared__ uint4 smem[2 * (BM + BN) * PITCH];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 15, lg = lane >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;

  Pol pol;
  pol.init(args, m0, n0, blockIdx.z);
  const int ns = pol.num_stages(args);

  f32x4 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (ns > 0) {
    pol.fetch(args, 0);
    pol.template commit<PITCH>(smem, smem + BM * PITCH);
  }
  __syncthreads();
  for (int st = 0; st < ns; ++st) {
    uint4* As = smem + (st & 1) * (BM + BN) * PITCH;
    uint4* Bs = As + BM * PITCH;
    if (st + 1 < ns) pol.fetch(args, st + 1);
#pragma unroll
    for (int u0 = 0; u0 < KU; u0 += 4) {
      uint4 fa[TI], fb[TJ];
#pragma unroll
      for (int i = 0; i < TI; ++i) fa[i] = As[(wm * WM + i * 16 + lr) * PITCH + u0 + lg];
#pragma unroll
      for (int j = 0; j < TJ; ++j) fb[j] = Bs[(wn * WN + j * 16 + lr) * PITCH + u0 + lg];
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) mma_unit(acc[i][j], fa[i], fb[j], (T*)nullptr);
    }
    if (st + 1 < ns) {
      uint4* An = smem + ((st + 1) & 1) * (BM + BN) * PITCH;
      pol.template commit<PITCH>(An, An + BM * PITCH);
    }
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      pol.out4(args, m0 + wm * WM + i * 16 + 4 * lg, n0 + wn * WN + j * 16 + lr, v);
    }
}

template <typename T>
__global__ void wgrad_reduce_kernel(const float* part, int splits, int K, int RS, int C, int C0,
                                    float* dw) {
  long long n = (long long)K * RS * C0;
  long long stride = (long long)K * RS * C;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    int c = i % C0;
    long long krs = i / C0;
    long long src = krs * C + c;
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += part[z * stride + src];
    dw[i] = s;
  }
}

// -------------------------------------------------------------- launching
template <typename T, template <typename, int, int> class PolT, int BM, int BN>
hipError_t launch_gemm(const typename PolT<T, BM, BN>::Args& args, int rows, int cols, int splits,
                       hipStream_t stream) {
  dim3 grid(cdiv(cols, BN), cdiv(rows, BM), splits);
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, PolT<T, BM, BN>>), grid, dim3(NT), 0, stream, args);
  return hipGetLastError();
}

// Choose the tile for a rows x cols output: 128 rows when there are >= 128
// rows; 128 columns only when that still leaves enough blocks for the chip.
inline void pick_tile(int rows, int cols, int& bm, int& bn) {
  bm = rows >= 128 ? 128 : 64;
  long long blocks128 = (long long)cdiv(cols, 128) * cdiv(rows, bm);
  bn = blocks128 >= 512 ? 128 : 64;
}

template <typename T, template <typename, int, int> class PolT>
hipError_t dispatch_tile(const typename PolT<T, 64, 64>::Args& args, int rows, int cols,
                         hipStream_t stream) {
  int bm, bn;
  pick_tile(rows, cols, bm, bn);
#define EKYA_TILE(BM_, BN_) \
  if (bm == BM_ && bn == BN_) return launch_gemm<T, PolT, BM_, BN_>(args, rows, cols, 1, stream);
  EKYA_TILE(64, 64)
  EKYA_TILE(64, 128)
  EKYA_TILE(128, 64)
  EKYA_TILE(128, 128)
#undef EKYA_TILE
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t conv_fwd_t(const ConvGeom& g, const void* x, const void* w, void* y,
                      const ConvEpilogue& epi, hipStream_t stream) {
  // All tile variants share one Args layout.
  FwdArgs<T> a{g, (const T*)x, (const T*)w, (T*)y, epi};
  return dispatch_tile<T, FwdPolicy>(a, g.K, g.N * g.P * g.Q, stream);
}

template <typename T>
hipError_t conv_dgrad_t(const ConvGeom& g, const void* dy, const void* wt, void* dx,
                        const void* res, hipStream_t stream) {
  DgradArgs<T> a{g, (const T*)dy, (const T*)wt, (T*)dx, (const T*)res};
  return dispatch_tile<T, DgradPolicy>(a, g.C, g.N * g.H * g.W, stream);
}

int wgrad_stage_m(int dt) { return dt == DT_F32 ? 16 : 64; }

}  // namespace

int conv_wgrad_splits(int dt, const ConvGeom& g) {
  const long long M = (long long)g.N * g.P * g.Q;
  const int rows = g.R * g.S * g.C;
  const int bn = g.K >= 128 ? 128 : 64;
  const long long tiles = (long long)cdiv(rows, 128) * cdiv(g.K, bn);
  const long long by_work = cdivl(M, 4LL * wgrad_stage_m(dt));  // >= 4 stages per split
  long long s = cdivl(1024, tiles);
  if (s > by_work) s = by_work;
  if (s < 1) s = 1;
  if (s > 1024) s = 1024;
  return (int)s;
}

size_t conv_wgrad_workspace_floats(int dt, const ConvGeom& g) {
  return (size_t)conv_wgrad_splits(dt, g) * g.K * g.R * g.S * g.C;
}

hipError_t conv_fwd(int dt, const ConvGeom& g, const void* x, const void* w, void* y,
                    const ConvEpilogue& epi, hipStream_t stream) {
  if (g.N * g.P * g.Q == 0) return hipSuccess;
  return dt == DT_F32 ? conv_fwd_t<float>(g, x, w, y, epi, stream)
                      : conv_fwd_t<bf16>(g, x, w, y, epi, stream);
}

hipError_t conv_dgrad(int dt, const ConvGeom& g, const void* dy, const void* wt, void* dx,
                      const void* res, hipStream_t stream) {
  if (g.N * g.H * g.W == 0) return hipSuccess;
  return dt == DT_F32 ? conv_dgrad_t<float>(g, dy, wt, dx, res, stream)
                      : conv_dgrad_t<bf16>(g, dy, wt, dx, res, stream);
}

hipError_t conv_wgrad(int dt, const ConvGeom& g, const void* x, const void* dy, float* partials,
                      float* dw, int C0, hipStream_t stream) {
  const int splits = conv_wgrad_splits(dt, g);
  const long long M = (long long)g.N * g.P * g.Q;
  const int stage = wgrad_stage_m(dt);
  const int mps = (int)(cdivl(cdivl(M, splits), stage) * stage);
  const int rows = g.R * g.S * g.C;
  const int bn = g.K >= 128 ? 128 : 64;
  hipError_t e;
  if (dt == DT_F32) {
    if (bn == 128) {
      WgradArgs<float> a{g, (const float*)x, (const float*)dy, partials, mps};
      e = launch_gemm<float, WgradPolicy, 128, 128>(a, rows, g.K, splits, stream);
    } else {
      WgradArgs<float> a{g, (const float*)x, (const float*)dy, partials, mps};
      e = launch_gemm<float, WgradPolicy, 128, 64>(a, rows, g.K, splits, stream);
    }
  } else {
    if (bn == 128) {
      WgradArgs<bf16> a{g, (const bf16*)x, (const bf16*)dy, partials, mps};
      e = launch_gemm<bf16, WgradPolicy, 128, 128>(a, rows, g.K, splits, stream);
    } else {
      WgradArgs<bf16> a{g, (const bf16*)x, (const bf16*)dy, partials, mps};
      e = launch_gemm<bf16, WgradPolicy, 128, 64>(a, rows, g.K, splits, stream);
    }
  }
  if (e != hipSuccess) return e;
  long long n = (long long)g.K * g.R * g.S * C0;
  int blocks = (int)std::min<long long>(cdivl(n, 256), 4096);
  hipLaunchKernelGGL(wgrad_reduce_kernel<float>, dim3(blocks), dim3(256), 0, stream, partials,
                     splits, g.K, g.R * g.S, g.C, C0, dw);
  return hipGetLastError();
}

}  // namespace ekya
