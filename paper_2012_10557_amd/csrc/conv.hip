// Convolution forward, data-gradient and weight-gradient as implicit GEMMs on
// MFMA (gfx950).  One block-tiled main loop (256 threads, 2 x 2 waves, LDS
// double buffering of 16-byte k-contiguous units, one stage of global->register
// prefetch) is shared by three operand policies:
//   forward : D[k][pix]   = sum_(r,s,c)  w[k][r][s][c]  * x(pix; r,s,c)
//   dgrad   : D[c][pix]   = sum_(r,s,k)  wT[c][r][s][k] * dy(pix; r,s,k)
//   wgrad   : D[rsc][k]   = sum_(pix)    x(pix; rsc)    * dy[pix][k]
// Rows of D are MFMA rows (the lane's four accumulator values are four
// consecutive rows), so forward/dgrad lanes own four consecutive NHWC channels
// and wgrad lanes own four consecutive (r,s,c) entries of one output channel.
//
// A stage covers KU units (KU*E reduction elements) of every tile row.  When
// the channel count is a multiple of that, a stage never straddles a filter
// tap, so the tap (r, s) and channel offset are block-uniform scalars that
// advance incrementally and the per-unit address is a bounds test plus an add.
// Forward and dgrad split the reduction over blockIdx.z when the output has too
// few tiles to fill the chip; partial sums go to an fp32 buffer that a second
// kernel adds up in a fixed order (deterministic) and finishes with the epilogue.
#include <algorithm>

#include "kernels.hpp"

namespace ekya {
namespace {

constexpr int NT = 256;

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// Quotient of non-negative a < 2^22 by d > 0, with inv = 1.0f / d.
__device__ __forceinline__ int fdiv(int a, int d, float inv) {
  int q = (int)((float)a * inv);
  if (q * d > a) --q;
  if ((q + 1) * d <= a) ++q;
  return q;
}

// Split-K output: partial sums in [split][col][row] fp32 (col = pixel).
struct SplitOut {
  float* part;
  int splits;
  int stages_per_split;
};

// BatchNorm chunk partials an unsplit GEMM leaves from its epilogue (part
// null: none); see wave_epilogue.
struct BnEpi {
  float* part = nullptr;
  const bf16* ymask = nullptr;
  const bf16* z = nullptr;
  const float* mean = nullptr;
  int bwd = 0;
};

// Stores v as bf16 and leaves the stored (rounded) values in v.
__device__ __forceinline__ void store4_keep(bf16* dst, float (&v)[4]) {
  store4<bf16>(dst, v);
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (float)(bf16)v[i];
}

// ------------------------------------------------------------------ forward
template <typename T> struct FwdArgs {
  ConvGeom g;
  const T* x;
  const T* w;
  T* y;
  ConvEpilogue epi;
  SplitOut so;
};

template <typename T, int BM, int BN, int KU_, bool UT>
struct FwdPolicy {
  static constexpr int E = Elt<T>::E;
  static constexpr int KU = KU_;
  static constexpr int UA = BM * KU / NT;
  static constexpr int UB = BN * KU / NT;
  using Args = FwdArgs<T>;

  int Ktot, m0, n0, s_begin, s_end;
  const T* arow[UA];
  const T* bptr[UB];   // UT: pixel origin + this unit's channel offset
  int bh0[UB], bw0[UB], bu[UB];
  bool bok[UB];
  int tr, ts, tc;      // UT: tap and channel offset of the next stage to fetch
  uint4 ra[UA], rb[UB];

  __device__ void init(const Args& a, int m0_, int n0_, int split) {
    const ConvGeom& g = a.g;
    m0 = m0_;
    n0 = n0_;
    Ktot = g.R * g.S * g.C;
    const int ns = cdiv(Ktot, KU * E);
    s_begin = min(ns, split * a.so.stages_per_split);
    s_end = min(ns, s_begin + a.so.stages_per_split);
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      const int q = threadIdx.x + NT * i, k = m0 + q / KU;
      arow[i] = (k < g.K) ? a.w + (long long)k * Ktot + (q % KU) * E : nullptr;
    }
    const int npix = g.N * g.P * g.Q;
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      const int q = threadIdx.x + NT * i, pix = n0 + q / KU;
      bu[i] = q % KU;
      bok[i] = pix < npix;
      const int pp = bok[i] ? pix : 0;
      const int n = pp / (g.P * g.Q), rem = pp % (g.P * g.Q);
      const int p = rem / g.Q, qq = rem % g.Q;
      bh0[i] = p * g.stride - g.pad;
      bw0[i] = qq * g.stride - g.pad;
      bptr[i] = a.x + (long long)n * g.H * g.W * g.C;
      if (UT) bptr[i] += ((long long)bh0[i] * g.W + bw0[i]) * g.C + bu[i] * E;
    }
    if (UT) {
      const int k0 = s_begin * KU * E;
      const int rs = k0 / g.C;
      tc = k0 - rs * g.C;
      tr = rs / g.S;
      ts = rs - tr * g.S;
    }
  }
  __device__ int first_stage() const { return s_begin; }
  __device__ int end_stage() const { return s_end; }
  __device__ void fetch(const Args& a, int st) {
    const ConvGeom& g = a.g;
    const int k0 = st * KU * E;
#pragma unroll
    for (int i = 0; i < UA; ++i)
      ra[i] = (arow[i] && (UT || k0 + (int)((threadIdx.x + NT * i) % KU) * E < Ktot))
                  ? ld16(arow[i] + k0) : zero_unit();
    if (UT) {
      const long long off = ((long long)tr * g.W + ts) * g.C + tc;
#pragma unroll
      for (int i = 0; i < UB; ++i) {
        const bool in = bok[i] && (unsigned)(bh0[i] + tr) < (unsigned)g.H &&
                        (unsigned)(bw0[i] + ts) < (unsigned)g.W;
        rb[i] = in ? ld16(bptr[i] + off) : zero_unit();
      }
      tc += KU * E;
      if (tc >= g.C) {
        tc = 0;
        if (++ts == g.S) {
          ts = 0;
          ++tr;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < UB; ++i) {
        const int k = k0 + bu[i] * E;
        uint4 v = zero_unit();
        if (bok[i] && k < Ktot) {
          const int c = k % g.C, rs = k / g.C;
          const int r = rs / g.S, s = rs % g.S;
          const int h = bh0[i] + r, w = bw0[i] + s;
          if (h >= 0 && h < g.H && w >= 0 && w < g.W)
            v = ld16(bptr[i] + ((long long)h * g.W + w) * g.C + c);
        }
        rb[i] = v;
      }
    }
  }
  template <int PITCH>
  __device__ void commit(uint4* As, uint4* Bs) {
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      const int q = threadIdx.x + NT * i;
      As[(q / KU) * PITCH + q % KU] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      const int q = threadIdx.x + NT * i;
      Bs[(q / KU) * PITCH + q % KU] = rb[i];
    }
  }
  // row = output channel, col = output pixel; v = 4 consecutive channels
  __device__ void out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    const int npix = g.N * g.P * g.Q;
    if (row >= g.K || col >= npix) return;
    const long long off = (long long)col * g.K + row;
    if (a.so.splits > 1) {
      float* dst = a.so.part + (long long)blockIdx.z * npix * g.K + off;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      return;
    }
    const ConvEpilogue& e = a.epi;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (e.scale) v[i] *= e.scale[row + i];
      if (e.shift) v[i] += e.shift[row + i];
    }
    if (e.res) {
      float r[4];
      load4<T>(reinterpret_cast<const T*>(e.res) + off, r);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += r[i];
    }
    if (e.relu) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = relu_nan(v[i]);
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
  SplitOut so;
};

// Requires K % (KU*E) == 0 (every stage within one tap) and stride 1 or 2.
template <typename T, int BM, int BN, int KU_, bool UT>
struct DgradPolicy {
  static constexpr int E = Elt<T>::E;
  static constexpr int KU = KU_;
  static constexpr int UA = BM * KU / NT;
  static constexpr int UB = BN * KU / NT;
  using Args = DgradArgs<T>;

  int Ktot, m0, n0, s_begin, s_end;
  const T* arow[UA];
  const T* bimg[UB];   // image base + this unit's channel offset
  int bh[UB], bw[UB];  // input pixel + pad
  bool bok[UB];
  int tr, ts, tk;
  uint4 ra[UA], rb[UB];

  __device__ void init(const Args& a, int m0_, int n0_, int split) {
    const ConvGeom& g = a.g;
    m0 = m0_;
    n0 = n0_;
    Ktot = g.R * g.S * g.K;
    const int ns = cdiv(Ktot, KU * E);
    s_begin = min(ns, split * a.so.stages_per_split);
    s_end = min(ns, s_begin + a.so.stages_per_split);
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      const int q = threadIdx.x + NT * i, c = m0 + q / KU;
      arow[i] = (c < g.C) ? a.wt + (long long)c * Ktot + (q % KU) * E : nullptr;
    }
    const int npix = g.N * g.H * g.W;
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      const int q = threadIdx.x + NT * i, pix = n0 + q / KU;
      bok[i] = pix < npix;
      const int pp = bok[i] ? pix : 0;
      const int n = pp / (g.H * g.W), rem = pp % (g.H * g.W);
      bimg[i] = a.dy + (long long)n * g.P * g.Q * g.K + (q % KU) * E;
      bh[i] = rem / g.W + g.pad;
      bw[i] = rem % g.W + g.pad;
    }
    const int k0 = s_begin * KU * E;
    const int rs = k0 / g.K;
    tk = k0 - rs * g.K;
    tr = rs / g.S;
    ts = rs - tr * g.S;
  }
  __device__ int first_stage() const { return s_begin; }
  __device__ int end_stage() const { return s_end; }
  __device__ void fetch(const Args& a, int st) {
    const ConvGeom& g = a.g;
    const int k0 = st * KU * E;
#pragma unroll
    for (int i = 0; i < UA; ++i) ra[i] = arow[i] ? ld16(arow[i] + k0) : zero_unit();
    const int sh = g.stride == 2 ? 1 : 0;
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      const int hp = bh[i] - tr, wp = bw[i] - ts;
      const int p = hp >> sh, q = wp >> sh;
      const bool in = bok[i] && hp >= 0 && wp >= 0 && ((hp | wp) & sh) == 0 && p < g.P && q < g.Q;
      rb[i] = in ? ld16(bimg[i] + ((long long)p * g.Q + q) * g.K + tk) : zero_unit();
    }
    tk += KU * E;
    if (tk >= g.K) {
      tk = 0;
      if (++ts == g.S) {
        ts = 0;
        ++tr;
      }
    }
  }
  template <int PITCH>
  __device__ void commit(uint4* As, uint4* Bs) {
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      const int q = threadIdx.x + NT * i;
      As[(q / KU) * PITCH + q % KU] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < UB; ++i) {
      const int q = threadIdx.x + NT * i;
      Bs[(q / KU) * PITCH + q % KU] = rb[i];
    }
  }
  __device__ void out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    const int npix = g.N * g.H * g.W;
    if (row >= g.C || col >= npix) return;
    const long long off = (long long)col * g.C + row;
    if (a.so.splits > 1) {
      float* dst = a.so.part + (long long)blockIdx.z * npix * g.C + off;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      return;
    }
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

template <typename T, int BM, int BN, int KU_, bool UT_>
struct WgradPolicy {
  static constexpr int E = Elt<T>::E;
  static constexpr int KU = E;               // units (of E pixels) per row per stage
  static constexpr int NA = (BM / E) * KU;   // = BM blocks for operand A
  static constexpr int NB = (BN / E) * KU;
  static constexpr int NBLK = (NA + NB + NT - 1) / NT;
  using Args = WgradArgs<T>;

  int m0, n0, mb, me, RSC;
  float inv_pq, inv_q;
  uint4 rv[NBLK][E];
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
    inv_pq = 1.0f / (float)(g.P * g.Q);
    inv_q = 1.0f / (float)g.Q;
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      const int b = threadIdx.x + NT * j;
      aok[j] = false;
      if (b < NA) {
        const int i0 = m0 + (b % (BM / E)) * E;
        if (i0 < RSC) {
          aok[j] = true;
          const int rs = i0 / g.C;
          ac[j] = i0 % g.C;
          ar[j] = rs / g.S;
          as_[j] = rs % g.S;
        }
      }
    }
  }
  __device__ int first_stage() const { return 0; }
  __device__ int end_stage() const { return me > mb ? cdiv(me - mb, KU * E) : 0; }
  __device__ void fetch(const Args& a, int st) {
    const ConvGeom& g = a.g;
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      const int b = threadIdx.x + NT * j;
#pragma unroll
      for (int e = 0; e < E; ++e) rv[j][e] = zero_unit();
      if (b < NA) {
        if (!aok[j]) continue;
        const int u = b / (BM / E);
        const int m = mb + st * KU * E + u * E;
        if (m >= me) continue;
        const int PQ = g.P * g.Q;
        int n = fdiv(m, PQ, inv_pq);
        const int rem = m - n * PQ;
        int p = fdiv(rem, g.Q, inv_q);
        int q = rem - p * g.Q;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if (m + e < me) {
            const int h = p * g.stride - g.pad + ar[j], w = q * g.stride - g.pad + as_[j];
            if ((unsigned)h < (unsigned)g.H && (unsigned)w < (unsigned)g.W)
              rv[j][e] = ld16(a.x + (((long long)n * g.H + h) * g.W + w) * g.C + ac[j]);
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
        const int bb = b - NA;
        const int k0 = n0 + (bb % (BN / E)) * E;
        const int m = mb + st * KU * E + (bb / (BN / E)) * E;
        if (k0 >= g.K) continue;
#pragma unroll
        for (int e = 0; e < E; ++e)
          if (m + e < me) rv[j][e] = ld16(a.dy + (long long)(m + e) * g.K + k0);
        transpose_block(rv[j], (T*)nullptr);
      }
    }
  }
  template <int PITCH>
  __device__ void commit(uint4* As, uint4* Bs) {
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      const int b = threadIdx.x + NT * j;
      if (b < NA) {
        const int rg = b % (BM / E), u = b / (BM / E);
#pragma unroll
        for (int e = 0; e < E; ++e) As[(rg * E + e) * PITCH + u] = rv[j][e];
      } else if (b < NA + NB) {
        const int bb = b - NA;
        const int rg = bb % (BN / E), u = bb / (BN / E);
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
  const int s0 = pol.first_stage(), s1 = pol.end_stage();

  f32x4 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (s0 < s1) {
    pol.fetch(args, s0);
    pol.template commit<PITCH>(smem, smem + BM * PITCH);
  }
  __syncthreads();
  for (int st = s0; st < s1; ++st) {
    uint4* As = smem + ((st - s0) & 1) * (BM + BN) * PITCH;
    uint4* Bs = As + BM * PITCH;
    if (st + 1 < s1) pol.fetch(args, st + 1);
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
    if (st + 1 < s1) {
      uint4* An = smem + ((st + 1 - s0) & 1) * (BM + BN) * PITCH;
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

// Sum of split-K partials [split][npix][C] in split order, then the epilogue.
template <typename T>
__global__ void split_reduce_kernel(const float* part, int splits, long long npix, int C,
                                    ConvEpilogue e, T* y) {
  const long long n4 = npix * C / 4;
  const long long stride = npix * C;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n4;
       i += (long long)gridDim.x * blockDim.x) {
    const long long off = i * 4;
    const int row = (int)(off % C);
    float4 s = *reinterpret_cast<const float4*>(part + off);
    for (int z = 1; z < splits; ++z) {
      const float4 t = *reinterpret_cast<const float4*>(part + z * stride + off);
      s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
    }
    float v[4] = {s.x, s.y, s.z, s.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (e.scale) v[k] *= e.scale[row + k];
      if (e.shift) v[k] += e.shift[row + k];
    }
    if (e.res) {
      float r[4];
      load4<T>(reinterpret_cast<const T*>(e.res) + off, r);
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] += r[k];
    }
    if (e.relu) {
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = relu_nan(v[k]);
    }
    store4<T>(y + off, v);
  }
}

__global__ void wgrad_reduce_kernel(const float* part, int splits, int K, int RS, int C, int C0,
                                    float* dw) {
  const long long n = (long long)K * RS * C0;
  const long long stride = (long long)K * RS * C;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(i % C0);
    const long long src = (i / C0) * C + c;
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += part[z * stride + src];
    dw[i] = s;
  }
}

// ------------------------------------------------- direct-to-LDS main loop
// bf16 forward and data-gradient GEMMs whose reduction runs in 64-element
// stages that never straddle a filter tap (C, resp. K, a multiple of 64).
// Operands go from global memory straight into LDS with
// global_load_lds_dwordx4 (16 bytes per lane; lane i's unit lands at the
// instruction's LDS base + 16 i), through an NST-deep ring of stages.  A stage
// holds BM A-rows then BN B-rows of 8 units (64 elements) each; unit u of row
// r sits at slot u ^ (r & 7), so that one instruction fills 8 whole rows
// (8 lanes read one 128-byte line) and the MFMA fragment reads (lane = 16-row
// index + 16 * k-unit) hit distinct banks.  Lanes whose row or tap lies
// outside the operand read a zero unit instead.
typedef __attribute__((address_space(3))) void lds_void;

__device__ __align__(16) uint4 g_zero_unit[1];

__device__ __forceinline__ void dma16(const void* src, uint4* lds_dst) {
  const uint32_t m0 = (uint32_t)(uintptr_t)(lds_void*)lds_dst;
  // inline asm: the compiler would otherwise make every later LDS read wait
  // for all outstanding loads; completion is tracked with explicit vmcnt waits
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(m0) : "memory");
}

// Barrier without __syncthreads' fence (which would wait for every
// outstanding global load); the vmcnt wait before it orders the LDS writes.
// The wave's own LDS reads are completed first: right after the barrier
// another wave may refill the slot they read.  (Left to itself the compiler
// sinks the last MFMAs of a stage, and the waits for their operands, below
// the barrier, so a slot could be overwritten while reads of it were still in
// flight -- harmless on an idle GPU, wrong results under contention.)
__device__ __forceinline__ void stage_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] at [15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2); give every XCD a contiguous range of tiles, rows of the output fastest,
// so the blocks sharing a column panel of the B operand share an L2.
__host__ __device__ __forceinline__ int xcd_tile(int L, int total) {
  const int x = L & 7, k = L >> 3;
  return x * (total >> 3) + min(x, total & 7) + k;
}

struct DmaFwdArgs {
  ConvGeom g;
  const bf16* x;
  const bf16* w;  // [K][R][S][C]
  bf16* y;
  ConvEpilogue epi;
  SplitOut so;
  int tiles_m, tiles_n;
  BnEpi bn;
};

template <int BM, int BN>
struct DmaFwdOp {
  static constexpr int GA = BM / 8, IPW = (BM + BN) / 32;  // row octets per wave
  using Args = DmaFwdArgs;
  int s_begin, s_end;
  long long Ktot;
  const bf16* ptr[IPW];
  int h0[IPW], w0[IPW];
  int rowoff[IPW];  // input pixel (h0, w0) within its image, in elements (may be negative)
  bool ok[IPW];
  int tr, ts, tc;
  int split;

  // reduction stages [s0, s1) of a split: 64-element steps of R*S*C
  static __device__ void stage_range(const Args& a, int split, int n0, int& s0, int& s1) {
    const int ns = a.g.R * a.g.S * a.g.C / 64;
    s0 = min(ns, split * a.so.stages_per_split);
    s1 = min(ns, s0 + a.so.stages_per_split);
  }

  __device__ void init(const Args& a, int m0, int n0, int split_, int wave, int lane) {
    const ConvGeom& g = a.g;
    split = split_;
    Ktot = (long long)g.R * g.S * g.C;
    stage_range(a, split, n0, s_begin, s_end);
    const int npix = g.N * g.P * g.Q;
    const int r8 = lane >> 3, u = (lane & 7) ^ r8;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int oct = wave + 4 * j;
      if (oct < GA) {
        const int row = m0 + oct * 8 + r8;
        ok[j] = row < g.K;
        ptr[j] = a.w + (ok[j] ? row : 0) * Ktot + u * 8;
        h0[j] = w0[j] = rowoff[j] = 0;
      } else {
        const int pix = n0 + (oct - GA) * 8 + r8;
        ok[j] = pix < npix;
        const int pp = ok[j] ? pix : 0;
        const int n = pp / (g.P * g.Q), rem = pp % (g.P * g.Q);
        const int p = rem / g.Q, q = rem % g.Q;
        h0[j] = p * g.stride - g.pad;
        w0[j] = q * g.stride - g.pad;
        rowoff[j] = (h0[j] * g.W + w0[j]) * g.C;
        ptr[j] = a.x + (long long)n * g.H * g.W * g.C + u * 8;
      }
    }
    const int k0 = s_begin * 64;
    const int rs = k0 / g.C;
    tc = k0 - rs * g.C;
    tr = rs / g.S;
    ts = rs - tr * g.S;
  }
  // Per load: two adds and two unsigned compares for the padding test, one
  // 32-bit offset; the tap's part (tr W + ts) C + tc is wave-uniform.
  __device__ void issue(const Args& a, int st, uint4* slot, int wave, const void* zero) {
    const ConvGeom& g = a.g;
    const long long k0 = (long long)st * 64;
    const int tap = (tr * g.W + ts) * g.C + tc;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int oct = wave + 4 * j;
      const void* src;
      if (oct < GA) {
        src = ok[j] ? (const void*)(ptr[j] + k0) : zero;
      } else {
        const int h = h0[j] + tr, w = w0[j] + ts;
        const bool in = ok[j] && (unsigned)h < (unsigned)g.H && (unsigned)w < (unsigned)g.W;
        src = in ? (const void*)(ptr[j] + (rowoff[j] + tap)) : zero;
      }
      dma16(src, slot + oct * 64);
    }
    tc += 64;
    if (tc >= g.C) {
      tc = 0;
      if (++ts == g.S) {
        ts = 0;
        ++tr;
      }
    }
  }
  static __device__ int chans(const Args& a) { return a.g.K; }
  static __device__ int pixels(const Args& a) { return a.g.N * a.g.P * a.g.Q; }
  // True when it stored bf16 outputs (then v holds the stored values).
  __device__ bool out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    const int npix = g.N * g.P * g.Q;
    if (row >= g.K || col >= npix) return false;
    const long long off = (long long)col * g.K + row;
    if (a.so.splits > 1) {
      float* dst = a.so.part + (long long)split * npix * g.K + off;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      return false;
    }
    const ConvEpilogue& e = a.epi;
    if (e.scale) {
      const float4 s = *reinterpret_cast<const float4*>(e.scale + row);
      v[0] *= s.x; v[1] *= s.y; v[2] *= s.z; v[3] *= s.w;
    }
    if (e.shift) {
      const float4 s = *reinterpret_cast<const float4*>(e.shift + row);
      v[0] += s.x; v[1] += s.y; v[2] += s.z; v[3] += s.w;
    }
    if (e.res) {
      float r[4];
      load4<bf16>(reinterpret_cast<const bf16*>(e.res) + off, r);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += r[i];
    }
    if (e.relu) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = relu_nan(v[i]);
    }
    store4_keep(a.y + off, v);
    return true;
  }
};

struct DmaDgradArgs {
  ConvGeom g;
  const bf16* dy;
  const bf16* wt;  // [C][R][S][K]
  bf16* dx;
  const bf16* res;
  SplitOut so;
  int tiles_m, tiles_n;
  BnEpi bn;
};

// dx[pix][c] = sum_(r,s,k) wt[c][r][s][k] dy(pix; r,s,k), stride 1 or 2.
template <int BM, int BN>
struct DmaDgradOp {
  static constexpr int GA = BM / 8, IPW = (BM + BN) / 32;
  using Args = DmaDgradArgs;
  int s_begin, s_end;
  long long Ktot;
  const bf16* ptr[IPW];
  int hp[IPW], wp[IPW];  // input pixel + pad
  int rowoff[IPW];       // stride 1: output-gradient pixel (hp, wp), in elements
  bool ok[IPW];
  int tr, ts, tk;
  int split;

  // reduction stages [s0, s1) of a split: 64-element steps of R*S*K
  static __device__ void stage_range(const Args& a, int split, int n0, int& s0, int& s1) {
    const int ns = a.g.R * a.g.S * a.g.K / 64;
    s0 = min(ns, split * a.so.stages_per_split);
    s1 = min(ns, s0 + a.so.stages_per_split);
  }

  __device__ void init(const Args& a, int m0, int n0, int split_, int wave, int lane) {
    const ConvGeom& g = a.g;
    split = split_;
    Ktot = (long long)g.R * g.S * g.K;
    stage_range(a, split, n0, s_begin, s_end);
    const int npix = g.N * g.H * g.W;
    const int r8 = lane >> 3, u = (lane & 7) ^ r8;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int oct = wave + 4 * j;
      if (oct < GA) {
        const int row = m0 + oct * 8 + r8;
        ok[j] = row < g.C;
        ptr[j] = a.wt + (ok[j] ? row : 0) * Ktot + u * 8;
        hp[j] = wp[j] = rowoff[j] = 0;
      } else {
        const int pix = n0 + (oct - GA) * 8 + r8;
        ok[j] = pix < npix;
        const int pp = ok[j] ? pix : 0;
        const int n = pp / (g.H * g.W), rem = pp % (g.H * g.W);
        hp[j] = rem / g.W + g.pad;
        wp[j] = rem % g.W + g.pad;
        rowoff[j] = (hp[j] * g.Q + wp[j]) * g.K;
        ptr[j] = a.dy + (long long)n * g.P * g.Q * g.K + u * 8;
      }
    }
    const int k0 = s_begin * 64;
    const int rs = k0 / g.K;
    tk = k0 - rs * g.K;
    tr = rs / g.S;
    ts = rs - tr * g.S;
  }
  // Stride 1: output-gradient pixel (hp - tr, wp - ts), the lane's row offset
  // plus a wave-uniform one; stride 2: (h / 2, w / 2) for even h and w.
  __device__ void issue(const Args& a, int st, uint4* slot, int wave, const void* zero) {
    const ConvGeom& g = a.g;
    const long long k0 = (long long)st * 64;
    const int tap = tk - (tr * g.Q + ts) * g.K;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int oct = wave + 4 * j;
      const void* src;
      if (oct < GA) {
        src = ok[j] ? (const void*)(ptr[j] + k0) : zero;
      } else {
        const int h = hp[j] - tr, w = wp[j] - ts;
        if (g.stride == 1) {
          const bool in = ok[j] && (unsigned)h < (unsigned)g.P && (unsigned)w < (unsigned)g.Q;
          src = in ? (const void*)(ptr[j] + (rowoff[j] + tap)) : zero;
        } else {
          const int p = h >> 1, q = w >> 1;
          const bool in = ok[j] && h >= 0 && w >= 0 && ((h | w) & 1) == 0 && p < g.P && q < g.Q;
          src = in ? (const void*)(ptr[j] + ((p * g.Q + q) * g.K + tk)) : zero;
        }
      }
      dma16(src, slot + oct * 64);
    }
    tk += 64;
    if (tk >= g.K) {
      tk = 0;
      if (++ts == g.S) {
        ts = 0;
        ++tr;
      }
    }
  }
  static __device__ int chans(const Args& a) { return a.g.C; }
  static __device__ int pixels(const Args& a) { return a.g.N * a.g.H * a.g.W; }
  __device__ bool out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    const int npix = g.N * g.H * g.W;
    if (row >= g.C || col >= npix) return false;
    const long long off = (long long)col * g.C + row;
    if (a.so.splits > 1) {
      float* dst = a.so.part + (long long)split * npix * g.C + off;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      return false;
    }
    if (a.res) {
      float r[4];
      load4<bf16>(a.res + off, r);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += r[i];
    }
    store4_keep(a.dx + off, v);
    return true;
  }
};

// Stride-2 data gradient by parity class.  Input pixel (h, w) = (2 i + ph,
// 2 j + pw) receives exactly the taps r = r0, r0 + 2, ... (r0 = (ph + pad)
// mod 2) and s = s0, s0 + 2, ..., from output-gradient pixel
// (i + (ph + pad - r) / 2, j + (pw + pad - s) / 2); the taps in between would
// only multiply zeros.  Each parity class (ph, pw) is its own GEMM over the
// class's pixels with a reduction over its own taps only: column tile ct
// belongs to class ct mod 4 (so every range of tiles mixes the light and
// heavy classes), class-local column (ct / 4) * BN + offset.  A class with no
// taps (1x1 kernels, odd pixels) writes zeros (plus the residual).
// With dy2: a 1x1 / stride-2 / pad-0 convolution on the same input (a
// projection shortcut) adds its data gradient, which reaches only the class
// (0, 0) pixels (2 i, 2 j): from its output-gradient pixel (i, j), the same
// pixel as that class's single 3x3 tap (pad 1) -- so the class's reduction
// runs K2 / 64 more stages over [dy2 | wt2] and no residual is read.
struct DmaDgradS2Args {
  ConvGeom g;
  const bf16* dy;
  const bf16* wt;  // [C][R][S][K]
  bf16* dx;
  const bf16* res;
  SplitOut so;
  int tiles_m, tiles_n;
  BnEpi bn;        // unused (no BatchNorm-statistics epilogue on this path)
  const bf16* dy2 = nullptr;  // shortcut output gradient [N][P][Q][K2]
  const bf16* wt2 = nullptr;  // shortcut weights [C][1][1][K2]
  int K2 = 0;
};

struct S2Class {
  int ph, pw, hc, wc, r0, nr, s0, nsc;
};
__host__ __device__ inline S2Class s2_class(const ConvGeom& g, int cls) {
  S2Class k;
  k.ph = cls >> 1;
  k.pw = cls & 1;
  k.hc = (g.H - k.ph + 1) / 2;  // rows h = 2 i + ph < H
  k.wc = (g.W - k.pw + 1) / 2;
  k.r0 = (k.ph + g.pad) & 1;
  k.nr = (g.R - k.r0 + 1) / 2;
  k.s0 = (k.pw + g.pad) & 1;
  k.nsc = (g.S - k.s0 + 1) / 2;
  return k;
}

template <int BM, int BN>
struct DmaDgradS2Op {
  static constexpr int GA = BM / 8, IPW = (BM + BN) / 32;
  using Args = DmaDgradS2Args;
  int s_begin, s_end;
  long long Ktot;
  const bf16* ptr[IPW];
  const bf16* ptr2[IPW];  // the shortcut's operands (class (0, 0) with dy2)
  int pi[IPW], qj[IPW];  // output-gradient pixel of the class's first tap (r0, s0)
  bool ok[IPW];
  int tr, ts, tk;        // tap (r0 + 2 tr, s0 + 2 ts), channel offset
  int r0, s0, nr, nsc;
  bool ext;              // in the shortcut's stages
  int split;

  // stages of a column tile's class: 64-element steps over the class's taps
  // x K, then (class (0, 0) with dy2) over K2
  static __device__ int class_stages(const Args& a, int ct) {
    const S2Class k = s2_class(a.g, ct & 3);
    return k.nr * k.nsc * a.g.K / 64 + ((ct & 3) == 0 && a.dy2 ? a.K2 / 64 : 0);
  }
  // reduction stages [s0, s1) of a split
  static __device__ void stage_range(const Args& a, int split, int n0, int& s0, int& s1) {
    const int ns = class_stages(a, n0 / BN);
    s0 = min(ns, split * a.so.stages_per_split);
    s1 = min(ns, s0 + a.so.stages_per_split);
  }

  __device__ void init(const Args& a, int m0, int n0, int split_, int wave, int lane) {
    const ConvGeom& g = a.g;
    split = split_;
    Ktot = (long long)g.R * g.S * g.K;
    stage_range(a, split, n0, s_begin, s_end);
    const int ct = n0 / BN;
    const S2Class k = s2_class(g, ct & 3);
    r0 = k.r0;
    s0 = k.s0;
    nr = k.nr;
    nsc = k.nsc;
    const bool sc = (ct & 3) == 0 && a.dy2;
    const int mc = g.N * k.hc * k.wc, lbase = (ct >> 2) * BN;
    const int r8 = lane >> 3, u = (lane & 7) ^ r8;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int oct = wave + 4 * j;
      if (oct < GA) {
        const int row = m0 + oct * 8 + r8;
        ok[j] = row < g.C;
        ptr[j] = a.wt + (ok[j] ? row : 0) * Ktot + u * 8;
        ptr2[j] = sc ? a.wt2 + (long long)(ok[j] ? row : 0) * a.K2 + u * 8 : a.wt;
        pi[j] = qj[j] = 0;
      } else {
        const int l = lbase + (oct - GA) * 8 + r8;
        ok[j] = l < mc;
        const int ll = ok[j] ? l : 0;
        const int n = ll / (k.hc * k.wc), rem = ll - n * (k.hc * k.wc);
        const int i = rem / k.wc, jj = rem - i * k.wc;
        pi[j] = i + (k.ph + g.pad - k.r0) / 2;
        qj[j] = jj + (k.pw + g.pad - k.s0) / 2;
        ptr[j] = a.dy + (long long)n * g.P * g.Q * g.K + u * 8;
        ptr2[j] = sc ? a.dy2 + (long long)n * g.P * g.Q * a.K2 + u * 8 : a.dy;
      }
    }
    const int k0 = s_begin * 64, kmain = nr * nsc * g.K;
    ext = k0 >= kmain;
    if (ext) {
      tk = k0 - kmain;
      tr = ts = 0;
    } else {
      const int rs = k0 / g.K;
      tk = k0 - rs * g.K;
      tr = rs / max(nsc, 1);
      ts = rs - tr * max(nsc, 1);
    }
  }
  __device__ void issue(const Args& a, int st, uint4* slot, int wave, const void* zero) {
    const ConvGeom& g = a.g;
    (void)st;
    if (ext) {
      // the shortcut: output-gradient pixel (i, j) = the class's tap pixel
#pragma unroll
      for (int j = 0; j < IPW; ++j) {
        const int oct = wave + 4 * j;
        const void* src;
        if (oct < GA) {
          src = ok[j] ? (const void*)(ptr2[j] + tk) : zero;
        } else {
          const int p = pi[j], q = qj[j];
          const bool in = ok[j] && (unsigned)p < (unsigned)g.P && (unsigned)q < (unsigned)g.Q;
          src = in ? (const void*)(ptr2[j] + ((p * g.Q + q) * a.K2 + tk)) : zero;
        }
        dma16(src, slot + oct * 64);
      }
      tk += 64;
      return;
    }
    const int woff = ((r0 + 2 * tr) * g.S + (s0 + 2 * ts)) * g.K + tk;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int oct = wave + 4 * j;
      const void* src;
      if (oct < GA) {
        src = ok[j] ? (const void*)(ptr[j] + woff) : zero;
      } else {
        const int p = pi[j] - tr, q = qj[j] - ts;
        const bool in = ok[j] && (unsigned)p < (unsigned)g.P && (unsigned)q < (unsigned)g.Q;
        src = in ? (const void*)(ptr[j] + ((p * g.Q + q) * g.K + tk)) : zero;
      }
      dma16(src, slot + oct * 64);
    }
    tk += 64;
    if (tk >= g.K) {
      tk = 0;
      if (++ts == nsc) {
        ts = 0;
        if (++tr == nr) ext = true;  // (tk = 0: the shortcut's first stage)
      }
    }
  }
  static __device__ int chans(const Args& a) { return a.g.C; }
  static __device__ int pixels(const Args& a) { return a.g.N * a.g.H * a.g.W; }
  __device__ bool out4(const Args& a, int row, int col, float (&v)[4]) {
    const ConvGeom& g = a.g;
    const int ct = col / BN;
    const S2Class k = s2_class(g, ct & 3);
    const int l = (ct >> 2) * BN + (col - ct * BN);
    if (row >= g.C || l >= g.N * k.hc * k.wc) return false;
    const int n = l / (k.hc * k.wc), rem = l - n * (k.hc * k.wc);
    const int i = rem / k.wc, jj = rem - i * k.wc;
    const long long pix = ((long long)n * g.H + 2 * i + k.ph) * g.W + 2 * jj + k.pw;
    const long long off = pix * g.C + row;
    if (a.so.splits > 1) {
      const long long npix = (long long)g.N * g.H * g.W;
      float* dst = a.so.part + (long long)split * npix * g.C + off;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      return false;
    }
    if (a.res) {
      float r[4];
      load4<bf16>(a.res + off, r);
#pragma unroll
      for (int i2 = 0; i2 < 4; ++i2) v[i2] += r[i2];
    }
    store4_keep(a.dx + off, v);
    return true;
  }
};

// Four bf16 (8 bytes) to float.
__device__ __forceinline__ void unpack4(uint2 u, float (&v)[4]) {
  v[0] = __uint_as_float(u.x << 16);
  v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16);
  v[3] = __uint_as_float(u.y & 0xffff0000u);
}

// x of the lane n places lower in the same 16-lane row (DPP row_ror:n).
template <int N> __device__ __forceinline__ float row_ror(float x) {
  static_assert(N >= 1 && N <= 15, "row_ror range");
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x120 + N, 0xF, 0xF,
                                                    false));
}

// Sum over the 16 lanes of a row (lanes 16 r .. 16 r + 15): adding the value
// rotated by 8, 4, 2, 1 lanes pairs the same two partial sums in both lanes
// of each pair, so every lane of the row ends with the same value.
__device__ __forceinline__ float row_sum16(float x) {
  x += row_ror<8>(x);
  x += row_ror<4>(x);
  x += row_ror<2>(x);
  x += row_ror<1>(x);
  return x;
}

// Output of one wave's TI x TJ fragments: channels row0 + 16 i + 4 (lane / 16)
// + 0..3 at pixel col0 + 16 j + lane % 16.  In the BNS variant with
// a.bn.part set (TJ = 4, so the wave covers the 64 pixels [col0, col0 + 64):
// BatchNorm chunk col0 / 64 of 64 rows) it also writes that chunk's per-channel partials of the stored
// values, in the layout of the standalone BatchNorm kernels (row pair k:
// first sums, then second sums, C each).  Forward: the sum and the squared
// deviations from the chunk mean.  Backward, with g = out [* (ymask > 0)]:
// sum g and sum g (z - mean).  A lane adds its own fragments in order, then
// the 16 lanes of a row (one channel's pixels) are combined by row_sum16.
template <int TI, int TJ, bool BNS, class Op>
__device__ __forceinline__ void wave_epilogue(const typename Op::Args& a, Op& op,
                                              f32x4 (&acc)[TI][TJ], int row0, int col0,
                                              int lane) {
  const int lr = lane & 15, lg = lane >> 4;
  if constexpr (BNS && TJ == 4) {
    if (a.bn.part) {
      const int C = Op::chans(a), npix = Op::pixels(a);
      // backward: the BatchNorm input z and the ReLU mask of the lane's
      // outputs, loaded before the stores (clamped in range; out-of-range
      // outputs are excluded below).  The loads are issued as inline asm and
      // waited for explicitly: loads the compiler tracks anywhere in this
      // kernel make it add full vmcnt waits to the loader waves' copy loop.
      uint2 zr[TI][TJ], yr[TI][TJ];
      if (a.bn.bwd) {
        const bf16* ym = a.bn.ymask ? a.bn.ymask : a.bn.z;
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) {
            const int row = min(row0 + i * 16 + 4 * lg, C - 4);
            const int col = min(col0 + j * 16 + lr, npix - 1);
            const long long off = (long long)col * C + row;
            asm volatile("global_load_dwordx2 %0, %1, off" : "=v"(zr[i][j]) : "v"(a.bn.z + off)
                         : "memory");
            asm volatile("global_load_dwordx2 %0, %1, off" : "=v"(yr[i][j]) : "v"(ym + off)
                         : "memory");
          }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) {
            asm volatile("" : "+v"(zr[i][j]));
            asm volatile("" : "+v"(yr[i][j]));
            if (!a.bn.ymask) yr[i][j] = make_uint2(0x3f803f80u, 0x3f803f80u);  // 1.0 each
          }
      }
      // store, keeping the stored values in acc
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
          op.out4(a, row0 + i * 16 + 4 * lg, col0 + j * 16 + lr, v);
          acc[i][j] = f32x4{v[0], v[1], v[2], v[3]};
        }
      if (col0 >= npix) return;
      float* p = a.bn.part + (long long)(col0 / 64) * 2 * C;
      const float nk = (float)min(64, npix - col0);
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int row = row0 + i * 16 + 4 * lg;
        if (!a.bn.bwd) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float x = 0.f;
#pragma unroll
            for (int j = 0; j < TJ; ++j) x += col0 + j * 16 + lr < npix ? acc[i][j][e] : 0.f;
            const float s1 = row_sum16(x);
            const float mu = s1 / nk;
            float y = 0.f;
#pragma unroll
            for (int j = 0; j < TJ; ++j) {
              const float d = acc[i][j][e] - mu;
              y += col0 + j * 16 + lr < npix ? d * d : 0.f;
            }
            const float s2 = row_sum16(y);
            if (lr == 0 && row < C) {
              p[row + e] = s1;
              p[C + row + e] = s2;
            }
          }
        } else {
          float mu[4] = {0.f, 0.f, 0.f, 0.f};
          if (row < C) {
#pragma unroll
            for (int e = 0; e < 4; ++e) mu[e] = a.bn.mean[row + e];
          }
          float x[4] = {0.f, 0.f, 0.f, 0.f}, y[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < TJ; ++j) {
            const bool in = row < C && col0 + j * 16 + lr < npix;
            float zz[4], yy[4];
            unpack4(zr[i][j], zz);
            unpack4(yr[i][j], yy);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float g = (in && yy[e] > 0.f) ? acc[i][j][e] : 0.f;
              x[e] += g;
              y[e] += g * (zz[e] - mu[e]);
            }
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float s1 = row_sum16(x[e]), s2 = row_sum16(y[e]);
            if (lr == 0 && row < C) {
              p[row + e] = s1;
              p[C + row + e] = s2;
            }
          }
        }
      }
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      op.out4(a, row0 + i * 16 + 4 * lg, col0 + j * 16 + lr, v);
    }
}

// 4 waves as WGM x (4 / WGM); each wave owns a (BM/WGM) x (BN*WGM/4) block of
// 16x16 MFMA tiles.  Stage st waits for its own loads (vmcnt), a barrier makes
// every wave's loads visible and retires the slot read in the previous
// iteration, which then receives stage st + NST - 1.
template <int BM, int BN, int WGM, int NST, class Op, bool BNS = false>
__global__ __launch_bounds__(NT) void gemm_dma_kernel(typename Op::Args a) {
  constexpr int WGN = 4 / WGM;
  static_assert((BM + BN) % 32 == 0, "row octets split over 4 waves");
  constexpr int LPS = Op::IPW;            // loads per lane per stage
  constexpr int SU = (BM + BN) * 8;       // 16-byte units per stage
  constexpr int WM = BM / WGM, WN = BN / WGN, TI = WM / 16, TJ = WN / 16;
  __shared__ uint4 smem[NST * SU];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  // one-dimensional grid of (split, tile) items, split-major, each XCD a
  // contiguous range: the blocks of an XCD share one slice of the reduction
  const int tiles = a.tiles_m * a.tiles_n;
  const int item = xcd_tile(blockIdx.x, tiles * a.so.splits);
  const int split = item / tiles, t = item - split * tiles;
  const int m0 = (t % a.tiles_m) * BM, n0 = (t / a.tiles_m) * BN;
  // lane's unit within a 16-row fragment: row fr, k-unit kf * 4 + fkc
  const int fr = lane & 15, fkc = lane >> 4;
  const int off0 = fr * 8 + (fkc ^ (fr & 7));
  const int off1 = fr * 8 + ((4 + fkc) ^ (fr & 7));

  Op op;
  op.init(a, m0, n0, split, wave, lane);
  const int s0 = op.s_begin, s1 = op.s_end;
  const void* zero = g_zero_unit;
  asm volatile("" : "+s"(zero));  // keep it in registers rather than re-deriving it per load

  f32x4 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int p = 0; p < NST - 1; ++p)
    if (s0 + p < s1) op.issue(a, s0 + p, smem + p * SU, wave, zero);

  int slot = 0;
  for (int st = s0; st < s1; ++st) {
    if (st + NST - 2 < s1)
      wait_vmcnt<LPS * (NST - 2)>();
    else
      wait_vmcnt<0>();
    stage_barrier();
    if (st + NST - 1 < s1) {
      const int nslot = slot == 0 ? NST - 1 : slot - 1;
      op.issue(a, st + NST - 1, smem + nslot * SU, wave, zero);
    }
    const uint4* As = smem + slot * SU + (wm * WM) * 8;
    const uint4* Bs = smem + slot * SU + (BM + wn * WN) * 8;
#pragma unroll
    for (int kf = 0; kf < 2; ++kf) {
      const int off = kf == 0 ? off0 : off1;
      uint4 fa[TI], fb[TJ];
#pragma unroll
      for (int i = 0; i < TI; ++i) fa[i] = As[i * 128 + off];
#pragma unroll
      for (int j = 0; j < TJ; ++j) fb[j] = Bs[j * 128 + off];
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) mma_unit(acc[i][j], fa[i], fb[j], (bf16*)nullptr);
    }
    if (++slot == NST) slot = 0;
  }

  wave_epilogue<TI, TJ, BNS>(a, op, acc, m0 + wm * WM, n0 + wn * WN, lane);
}

// Warp-specialised variant: (BM / WTM) x (BN / WTN) compute waves (each a
// WTM x WTN block of 16x16 MFMA tiles) and four loader waves.  The
// loader waves keep the copies of the next NST - 1 stages in flight (the
// CU's vector-memory path, not the MFMAs, is what a wave issuing its own
// copies waits on); the compute waves only read LDS fragments and issue
// MFMAs.  One barrier per stage: before it the loaders have waited for stage
// st + 1 and the compute waves have finished reading stage st, whose slot the
// loaders refill after it.  Every wave executes the same barriers.
constexpr int WS_LOADERS = 4;

template <int BM, int BN, int WTM, int WTN, int NST, class Op, bool BNS = false>
__global__ __launch_bounds__((BM / WTM) * (BN / WTN) * 64 + WS_LOADERS * 64) void gemm_ws_kernel(
    typename Op::Args a) {
  constexpr int WGN = BN / WTN, CW = (BM / WTM) * WGN;
  constexpr int TI = WTM / 16, TJ = WTN / 16;
  constexpr int LPS = Op::IPW;            // copies per loader lane per stage
  constexpr int SU = (BM + BN) * 8;       // 16-byte units per stage
  static_assert(LPS * (NST - 2) < 64, "vmcnt range");
  __shared__ uint4 smem[NST * SU];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tiles = a.tiles_m * a.tiles_n;
  const int item = xcd_tile(blockIdx.x, tiles * a.so.splits);
  const int split = item / tiles, t = item - split * tiles;
  const int m0 = (t % a.tiles_m) * BM, n0 = (t / a.tiles_m) * BN;
  int s0, s1;
  Op::stage_range(a, split, n0, s0, s1);

  // The two roles run separate loops (their registers are never live
  // together) with the same barrier count: one before the loop, one per stage.
  if (wave >= CW) {
    const int lw = wave - CW;
    Op op;
    op.init(a, m0, n0, split, lw, lane);
    const void* zero = g_zero_unit;
    asm volatile("" : "+s"(zero));
#pragma unroll
    for (int p = 0; p < NST - 1; ++p)
      if (s0 + p < s1) op.issue(a, s0 + p, smem + p * SU, lw, zero);
    if (s0 + NST - 2 < s1)
      wait_vmcnt<LPS * (NST - 2)>();
    else
      wait_vmcnt<0>();
    stage_barrier();
    int slot = 0;
    for (int st = s0; st < s1; ++st) {
      if (st + NST - 1 < s1) {
        const int nslot = slot == 0 ? NST - 1 : slot - 1;
        op.issue(a, st + NST - 1, smem + nslot * SU, lw, zero);
        wait_vmcnt<LPS * (NST - 2)>();  // stage st + 1 has landed
      } else {
        wait_vmcnt<0>();
      }
      stage_barrier();
      if (++slot == NST) slot = 0;
    }
    return;
  }

  const int wm = wave / WGN, wn = wave % WGN;
  const int fr = lane & 15, fkc = lane >> 4;
  const int off0 = fr * 8 + (fkc ^ (fr & 7));
  const int off1 = fr * 8 + ((4 + fkc) ^ (fr & 7));
  f32x4 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  stage_barrier();
  int slot = 0;
  for (int st = s0; st < s1; ++st) {
    const uint4* As = smem + slot * SU + (wm * WTM) * 8;
    const uint4* Bs = smem + slot * SU + (BM + wn * WTN) * 8;
#pragma unroll
    for (int kf = 0; kf < 2; ++kf) {
      const int off = kf == 0 ? off0 : off1;
      uint4 fa[TI], fb[TJ];
#pragma unroll
      for (int i = 0; i < TI; ++i) fa[i] = As[i * 128 + off];
#pragma unroll
      for (int j = 0; j < TJ; ++j) fb[j] = Bs[j * 128 + off];
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) mma_unit(acc[i][j], fa[i], fb[j], (bf16*)nullptr);
    }
    stage_barrier();
    if (++slot == NST) slot = 0;
  }

  Op op;
  op.split = split;
  wave_epilogue<TI, TJ, BNS>(a, op, acc, m0 + wm * WTM, n0 + wn * WTN, lane);
}

// ------------------------------------------- direct-to-LDS weight gradient
// bf16 D[rsc][k] = sum_pix x(pix; r,s,c) dy[pix][k] with C and K multiples of
// 64.  A tile's rows are BM channels of one tap.  A stage is 64 pixels: 64
// gathered input-pixel rows of BM channels (zero where the tap falls in the
// padding), then 64 rows of BN output-gradient channels, both pixel-major as
// in memory and loaded by global_load_lds_dwordx4; 32-byte segment s of
// pixel row p is stored at s ^ (p mod segments-per-row).  The MFMA operands
// need 8 consecutive pixels of one channel per lane: ds_read_b64_tr_b16
// reads a 4-pixel x 16-channel block per 16-lane group (member m supplies
// the address of pixel m / 4, channels 4 (m % 4) .. +3) and hands lane i the
// 4 pixels of channel i; two such reads make one operand.
typedef short v4i16 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 lds_read_tr16(const char* p) {
  v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(__attribute__((address_space(3))) char*)p);
  return __builtin_bit_cast(uint2, v);
}

struct WgDmaArgs {
  ConvGeom g;
  const bf16* x;
  const bf16* dy;
  float* out;       // [split][K][R*S*C], or dw itself with one split
  int m_per_split;  // pixels per split, a multiple of 64
  int tiles_m, tiles_n;
  int splits;
};

template <int BM, int BN>
__global__ __launch_bounds__(NT) void wgrad_dma_kernel(WgDmaArgs a) {
  constexpr int NST = 2;
  constexpr int UA = BM / 8, UB = BN / 8;     // 16-byte units per pixel row
  constexpr int RA = 64 / UA, RB = 64 / UB;   // pixel rows per DMA instruction
  constexpr int IA = 64 / RA, IB = 64 / RB;   // DMA instructions per stage
  constexpr int LPS = (IA + IB) / 4, LA = IA / 4;
  static_assert(IA % 4 == 0 && IB % 4 == 0, "instructions split over 4 waves");
  constexpr int SA = BM / 16, SB = BN / 16;   // 32-byte segments per row
  constexpr int STAGE_BYTES = 64 * (BM + BN) * 2;
  constexpr int WM = BM / 2, WN = BN / 2, TI = WM / 16, TJ = WN / 16;
  __shared__ __align__(16) char smem[NST * STAGE_BYTES];

  const ConvGeom& g = a.g;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int t = xcd_tile(blockIdx.x, a.tiles_m * a.tiles_n);
  const int m0 = (t % a.tiles_m) * BM, n0 = (t / a.tiles_m) * BN;
  const int rs = m0 / g.C, c0 = m0 - rs * g.C;
  const int tr = rs / g.S, ts = rs - tr * g.S;
  const int M = g.N * g.P * g.Q, PQ = g.P * g.Q;
  const int mb = blockIdx.y * a.m_per_split;
  const int me = min(M, mb + a.m_per_split);
  const int ns = me > mb ? (me - mb + 63) / 64 : 0;

  // A rows of this lane advance by 64 pixels per stage: (n, p, q) is stepped
  int an[LA], ap[LA], aq[LA], am[LA];
  const int dq = 64 % g.Q, dp = (64 / g.Q) % g.P, dn = 64 / PQ;
#pragma unroll
  for (int j = 0; j < LA; ++j) {
    const int pr = (wave + 4 * j) * RA + lane / UA;
    am[j] = mb + pr;
    const int m = am[j] < M ? am[j] : 0;
    an[j] = m / PQ;
    const int rem = m - an[j] * PQ;
    ap[j] = rem / g.Q;
    aq[j] = rem - ap[j] * g.Q;
  }
  auto issue = [&](int st, char* slot) {
#pragma unroll
    for (int j = 0; j < LPS; ++j) {
      const int ins = wave + 4 * j;
      if (j < LA) {
        const int pr = ins * RA + lane / UA, sl = lane % UA;
        const int u = 2 * ((sl >> 1) ^ (pr % SA)) + (sl & 1);
        const int h = ap[j] * g.stride - g.pad + tr, w = aq[j] * g.stride - g.pad + ts;
        const bool in = am[j] < me && (unsigned)h < (unsigned)g.H && (unsigned)w < (unsigned)g.W;
        const bf16* src = a.x + (((long long)an[j] * g.H + h) * g.W + w) * g.C + c0 + u * 8;
        dma16(in ? (const void*)src : (const void*)g_zero_unit,
              reinterpret_cast<uint4*>(slot + ins * 1024));
        am[j] += 64;
        aq[j] += dq;
        int cy = aq[j] >= g.Q;
        aq[j] -= cy ? g.Q : 0;
        ap[j] += dp + cy;
        cy = ap[j] >= g.P;
        ap[j] -= cy ? g.P : 0;
        an[j] += dn + cy;
      } else {
        const int ib = ins - IA;
        const int pr = ib * RB + lane / UB, sl = lane % UB;
        const int u = 2 * ((sl >> 1) ^ (pr % SB)) + (sl & 1);
        const int m = mb + st * 64 + pr;
        const void* src = m < me ? (const void*)(a.dy + (long long)m * g.K + n0 + u * 8)
                                 : (const void*)g_zero_unit;
        dma16(src, reinterpret_cast<uint4*>(slot + 64 * BM * 2 + ib * 1024));
      }
    }
  };

  f32x4 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (ns > 0) issue(0, smem);
  const int gq = lane >> 4, jr = (lane & 15) >> 2, qd = lane & 3;
  int slot = 0;
  for (int st = 0; st < ns; ++st) {
    wait_vmcnt<0>();
    stage_barrier();
    if (st + 1 < ns) issue(st + 1, smem + (slot ^ 1) * STAGE_BYTES);
    const char* As = smem + slot * STAGE_BYTES;
    const char* Bs = As + 64 * BM * 2;
#pragma unroll
    for (int kf = 0; kf < 2; ++kf) {
      uint4 fa[TI], fb[TJ];
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int pr = kf * 32 + gq * 8 + half * 4 + jr;
#pragma unroll
        for (int i = 0; i < TI; ++i) {
          const int ch = wm * WM + i * 16 + 4 * qd;
          const uint2 v = lds_read_tr16(As + pr * (BM * 2) + (((ch >> 4) ^ (pr % SA)) * 32) +
                                        (ch & 15) * 2);
          if (half == 0) { fa[i].x = v.x; fa[i].y = v.y; } else { fa[i].z = v.x; fa[i].w = v.y; }
        }
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          const int ch = wn * WN + j * 16 + 4 * qd;
          const uint2 v = lds_read_tr16(Bs + pr * (BN * 2) + (((ch >> 4) ^ (pr % SB)) * 32) +
                                        (ch & 15) * 2);
          if (half == 0) { fb[j].x = v.x; fb[j].y = v.y; } else { fb[j].z = v.x; fb[j].w = v.y; }
        }
      }
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) mma_unit(acc[i][j], fa[i], fb[j], (bf16*)nullptr);
    }
    slot ^= 1;
  }

  const int RSC = g.R * g.S * g.C;
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int row = m0 + wm * WM + i * 16 + 4 * lg, col = n0 + wn * WN + j * 16 + lr;
      float* dst = a.out + ((long long)blockIdx.y * g.K + col) * RSC + row;
      *reinterpret_cast<float4*>(dst) =
          make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
}

// ----------------------------------- weight gradient of a 3x3 / stride 1 conv
// All nine taps at once: a block owns 64 input channels x 64 output channels
// x 9 taps (576 x 64 outputs) and reduces over 8 x 8 patches of output
// pixels.  A stage is one patch: its 10 x 10 input pixels (the patch grown by
// the filter's reach, zero outside the image) and its 64 output-gradient
// pixels (zero outside the image) go to LDS once, and each tap reads the
// input at its own offset -- one load of the input serves nine taps, where a
// tap-at-a-time tiling loads it nine times.  Pixel rows of 64 channels
// (128 bytes) hold four 32-byte segments, segment s of pixel p stored at
// s ^ (p mod 4); an 8-byte transpose read (ds_read_b64_tr_b16) takes 4
// pixels x 16 channels per 16-lane group, member m supplying pixel m / 4,
// channels 4 (m % 4) .. +3, and hands lane i channel i's 4 pixels; two reads
// make a lane's MFMA operand of 8 pixels (one patch row).  Compute wave w
// owns row tiles 9 w .. 9 w + 8 of the 36 (tap t / 4, channels 16 (t % 4) ..)
// and all 4 column tiles; the output-gradient fragments are read once per
// k-step and used by the nine row tiles.
struct TapGeom {
  int tiles_c, tiles_k, splits, pps;  // pps: patches per split
  int py_n, px_n;                     // patches down / across an image
  __host__ __device__ int n_patches(int N) const { return N * py_n * px_n; }
};

// A staged pixel row of a copy: sy, sx its offset from the patch origin
// (input rows start one pixel up and left; unused rows get an offset that no
// patch brings inside the image); off its element offset in the operand
// relative to the patch origin's pixel, channel block included.  Shared by
// the kernels and the host-side bounds checks.
struct TapSlot {
  int sy, sx, off;
};
struct WgTapArgs {
  ConvGeom g;
  TapGeom t;
  const bf16* x;
  const bf16* dy;
  float* out;  // [split][K][9 C]
};

// ------------------------------------ 3x3 / stride 1 convolution, 64 -> 64
// out[pix][o] = sum over taps (r, s) and input channels i of
// A[o][r][s][i] * in(pix + d)[i], d = (r - 1, s - 1) for the forward pass
// (A: weights [K][R][S][C], in: x) and d = (1 - r, 1 - s) for the data
// gradient (A: [C][R][S][K], in: dy).  With 64 channels on both sides the
// whole filter (64 x 576) fits in the compute waves' registers for the
// block's life: compute wave (wm, wn) of a 2 x 2 grid owns output channels
// 32 wm .. + 31 (two 16-row MFMA tiles) and patch rows 4 wn .. 4 wn + 3 (two
// 16-pixel tiles) of an 8 x 8 output patch, and holds its rows' 18 k-steps
// (9 taps x 2 halves of 32 channels) as MFMA operands (144 registers), so
// only the patches' inputs stream through LDS, in a ring of C64_NST stages:
// the patch's 10 x 10 input pixels (13 copies of 8 pixel rows, the last 4
// rows zero), pixel (ty, tx) of the tile holding 16-byte chunk u at
// u ^ ((ty + tx) mod 8), so that the 16 lanes of a read (8 consecutive
// pixels of two tile rows) hit distinct banks; then, with a residual, the
// patch's 64 residual pixels (8 copies, chunk u of pixel p at u ^ (p mod 8)).
// A fifth wave does all the copying: it never stores, so its vector-memory
// count covers copies only and it keeps up to C64_NST - 1 stages in flight
// (3 x 21 copies: the counter has 6 bits) while waiting for the oldest; the
// compute waves wait on barriers only, never on their own stores.  MFMA row
// 4 q + j of tile rt is channel 32 wm + 8 q + 4 rt + j, so a lane's
// accumulators hold 8 consecutive channels of one pixel (one 16-byte store).
// Blocks are persistent, one per CU (5 waves of at most 256 registers fill a
// CU's register file).
constexpr int C64_IN_COPIES = 13;                   // 104 input pixel rows (100 used)
constexpr int C64_RES_COPIES = 8;
constexpr int C64_ROWS = 8 * C64_IN_COPIES;
constexpr int C64_STAGE = (C64_ROWS + 64) * 128;    // input + residual bytes per stage
constexpr int C64_NST = 4;
constexpr int C64_NT = 320;                         // 4 compute waves + 1 copy wave
constexpr int C64_TARGET_BLOCKS = 256;
static_assert((C64_NST - 1) * (C64_IN_COPIES + C64_RES_COPIES) <= 63, "vector-memory counter");

struct Conv64Args {
  ConvGeom g;            // the forward convolution (C == K == 64, 3x3, stride 1, pad 1)
  const bf16* in;        // x (forward) or dy (data gradient), [N][H][W][64]
  const bf16* a;         // [64][3][3][64]
  bf16* out;             // [N][H][W][64]
  ConvEpilogue epi;      // forward: scale, shift, res, relu; data gradient: res only
  int pps, py_n, px_n;   // patches per block, patches down / across an image
};

// Copy j (0 .. 20) of the copy wave: 8 staged pixel rows (lane / 8), 16-byte
// segment lane % 8.  Input rows (j < C64_IN_COPIES): tile pixel p, image
// offset (p / 10 - 1, p % 10 - 1) from the patch origin, in range only for
// p < 100 (sy far out otherwise).  Residual rows: patch pixel p - C64_ROWS,
// offset (p / 8, p % 8).  `off` is the element offset from the patch
// origin's first channel, chunk swizzled.
__host__ __device__ inline TapSlot c64_slot(int W, int lane, int j) {
  const int pix = 8 * j + (lane >> 3);
  TapSlot t;
  int sy, sx, sw;
  if (pix < C64_ROWS) {
    sy = pix < 100 ? pix / 10 - 1 : -(1 << 24);
    sx = pix - 10 * (pix / 10) - 1;
    sw = (pix / 10 + pix % 10) & 7;
  } else {
    sy = (pix - C64_ROWS) >> 3;
    sx = (pix - C64_ROWS) & 7;
    sw = sx;
  }
  const int u = (lane & 7) ^ sw;
  t.sy = sy;
  t.sx = sx;
  t.off = sy > -(1 << 24) ? (sy * W + sx) * 64 + u * 8 : 0;
  return t;
}

// One patch out of ring slot SLOT (the slot is an immediate of every LDS
// read).  fa: the wave's filter operands; rb[v][h]: the lane's read offset
// for k-step half h when its column's tap pixel (ty, tx) has
// ty + tx = b + v mod 8 (b: the lane's own pixel, tap offset 0), chunk
// swizzle included.  The schedule keeps the reads two k-steps ahead of the
// MFMAs.
template <bool DGRAD, int SLOT>
__device__ __forceinline__ void conv64_patch(const char* smem, const uint4 (&fa)[2][18],
                                             const int (&rb)[8][2], f32x4 (&acc)[2][2]) {
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) acc[rt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < 18; ++ks) {
    const int tap = ks >> 1, r = tap / 3, s = tap % 3, h = ks & 1;
    uint4 fb[2];
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
      // tile pixel offset from the lane's own: forward (2 ct + r) rows and s
      // columns; data gradient (2 ct + 2 - r) rows and 2 - s columns
      const int d = DGRAD ? 20 * ct + 22 - 10 * r - s : 20 * ct + 10 * r + s;
      const int v = DGRAD ? (2 * ct + 4 - r - s) & 7 : (2 * ct + r + s) & 7;
      fb[ct] = *reinterpret_cast<const uint4*>(smem + SLOT * C64_STAGE + d * 128 + rb[v][h]);
    }
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) mma_unit(acc[rt][ct], fa[rt][ks], fb[ct], (bf16*)nullptr);
  }
  // scheduling groups (0x100: LDS reads, 0x008: MFMAs)
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
}

template <int L> __device__ __forceinline__ void c64_wait(int later) {
  // at most `later` (0 .. C64_NST - 2) stages of L copies still in flight
  if (later >= 2) wait_vmcnt<2 * L>();
  else if (later == 1) wait_vmcnt<L>();
  else wait_vmcnt<0>();
}

template <bool DGRAD>
__global__ __launch_bounds__(C64_NT) void conv64_kernel(Conv64Args a) {
  static_assert(C64_NST == 4, "the compute loop selects among 4 slots; c64_wait covers 2 later stages");
  __shared__ __align__(16) char smem[C64_NST * C64_STAGE];
  __shared__ __align__(16) float ss[128];  // forward: scale[64], shift[64]
  const int H = a.g.H, W = a.g.W, N = a.g.N;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int per_img = a.py_n * a.px_n;
  const int q0 = xcd_tile(blockIdx.x, gridDim.x) * a.pps;
  const int ns = max(0, min(N * per_img, q0 + a.pps) - q0);
  const bool has_res = a.epi.res != nullptr;
  auto origin = [&](int st, int& n, int& py0, int& px0) {
    const int q = q0 + st;
    n = q / per_img;
    const int rem = q - n * per_img, pyi = rem / a.px_n;
    py0 = 8 * pyi;
    px0 = 8 * (rem - pyi * a.px_n);
  };

  if (wave == 4) {
    // the copy wave: stages 0 .. C64_NST - 2 ahead, then one more per barrier
    const bf16* const res = reinterpret_cast<const bf16*>(a.epi.res);
    const void* const zero = g_zero_unit;
    auto issue = [&](int st) {
      int n, py0, px0;
      origin(st, n, py0, px0);
      const long long pbase = ((long long)n * H * W + (long long)py0 * W + px0) * 64;
      char* slot = smem + (st % C64_NST) * C64_STAGE;
#pragma unroll
      for (int j = 0; j < C64_IN_COPIES + C64_RES_COPIES; ++j) {
        if (j >= C64_IN_COPIES && !has_res) break;
        const TapSlot sl = c64_slot(W, lane, j);
        const bf16* b = (j < C64_IN_COPIES ? a.in : res) + pbase;
        const bool in = (unsigned)(py0 + sl.sy) < (unsigned)H && (unsigned)(px0 + sl.sx) < (unsigned)W;
        dma16(in ? (const void*)(b + sl.off) : zero, reinterpret_cast<uint4*>(slot + j * 1024));
      }
    };
    for (int st = 0; st < min(ns, C64_NST - 1); ++st) issue(st);
    for (int st = 0; st < ns; ++st) {
      // stage st has landed once only the later stages issued remain
      const int later = min(ns - 1 - st, C64_NST - 2);
      if (has_res) c64_wait<C64_IN_COPIES + C64_RES_COPIES>(later);
      else c64_wait<C64_IN_COPIES>(later);
      stage_barrier();
      // every compute wave is past stage st - 1: refill its slot
      if (st + C64_NST - 1 < ns) issue(st + C64_NST - 1);
    }
    return;
  }

  const int wm = wave >> 1, wn = wave & 1;
  // the wave's filter rows as MFMA operands: tile rt, row lane % 16 = 4 q + j
  // (channel 32 wm + 8 q + 4 rt + j), k-step ks = 2 tap + half: channels
  // 32 half + 8 (lane / 16) .. + 7 of tap ks / 2
  const int cq = lane & 15, cu = lane >> 4;
  uint4 fa[2][18];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int ks = 0; ks < 18; ++ks) {
      const int o = 32 * wm + 8 * (cq >> 2) + 4 * rt + (cq & 3);
      const int ch = 32 * (ks & 1) + 8 * cu;
      fa[rt][ks] = *reinterpret_cast<const uint4*>(a.a + ((long long)o * 9 + (ks >> 1)) * 64 + ch);
    }
  // the lane's column at tap offset 0: patch pixel (4 wn + (lane % 16) / 8,
  // lane % 8) = tile pixel (ty0, tx0), ip0 (forward: the tap (0, 0) pixel;
  // data gradient: two rows and columns before the tap (2, 2) pixel)
  const int ty0 = 4 * wn + (cq >> 3), tx0 = lane & 7;
  const int ip0 = ty0 * 10 + tx0;
  int rb[8][2];
#pragma unroll
  for (int v = 0; v < 8; ++v)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      rb[v][h] = ip0 * 128 + ((((4 * h + cu) ^ ((ty0 + tx0 + v) & 7))) * 16);
  // this lane's output channels: c0 .. c0 + 7
  const int c0 = 32 * wm + 8 * cu;
  const bool affine = !DGRAD && (a.epi.scale || a.epi.shift);
  if (affine && threadIdx.x < 128) {
    const int c = threadIdx.x & 63;
    const float* src = threadIdx.x < 64 ? a.epi.scale : a.epi.shift;
    ss[threadIdx.x] = src ? src[c] : (threadIdx.x < 64 ? 1.f : 0.f);
  }
  const bool relu = !DGRAD && a.epi.relu;
  // residual pixel pp = 8 ppy + ppx (ppx = lane % 8): chunk c0 / 8 at
  // (c0 / 8) ^ ppx
  const int rr = C64_ROWS * 128 + ty0 * 8 * 128 + tx0 * 128 + (((c0 >> 3) ^ tx0) * 16);

  f32x4 acc[2][2];
  for (int st = 0; st < ns; ++st) {
    stage_barrier();
    const int slot = st % C64_NST;
    switch (slot) {
      case 0: conv64_patch<DGRAD, 0>(smem, fa, rb, acc); break;
      case 1: conv64_patch<DGRAD, 1>(smem, fa, rb, acc); break;
      case 2: conv64_patch<DGRAD, 2>(smem, fa, rb, acc); break;
      default: conv64_patch<DGRAD, 3>(smem, fa, rb, acc); break;
    }
    const char* X = smem + slot * C64_STAGE;
    int n, py0, px0;
    origin(st, n, py0, px0);
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
      const int ppy = ty0 + 2 * ct, ppx = tx0;
      float v[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[j] = acc[0][ct][j];
        v[4 + j] = acc[1][ct][j];
      }
      if (affine) {
        const float4* s4 = reinterpret_cast<const float4*>(ss + c0);
        const float4* h4 = reinterpret_cast<const float4*>(ss + 64 + c0);
        const float4 sa = s4[0], sb = s4[1], ha = h4[0], hb = h4[1];
        v[0] = v[0] * sa.x + ha.x; v[1] = v[1] * sa.y + ha.y;
        v[2] = v[2] * sa.z + ha.z; v[3] = v[3] * sa.w + ha.w;
        v[4] = v[4] * sb.x + hb.x; v[5] = v[5] * sb.y + hb.y;
        v[6] = v[6] * sb.z + hb.z; v[7] = v[7] * sb.w + hb.w;
      }
      if (has_res) {
        const uint4 rv = *reinterpret_cast<const uint4*>(X + rr + ct * 16 * 128);
        const bf16x8 rbv = __builtin_bit_cast(bf16x8, rv);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] += (float)rbv[i];
      }
      if (relu) {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = relu_nan(v[i]);
      }
      const int py = py0 + ppy, px = px0 + ppx;
      if (py < H && px < W) {
        bf16x8 ob;
#pragma unroll
        for (int i = 0; i < 8; ++i) ob[i] = (bf16)v[i];
        *reinterpret_cast<uint4*>(a.out + (((long long)n * H + py) * W + px) * 64 + c0) =
            __builtin_bit_cast(uint4, ob);
      }
    }
  }
}

// ---------------------------- all-taps weight gradient, warp-specialised
// The stage layout and per-wave tiles above, with the conv64_kernel
// arrangement of the copies: a fifth wave issues every
// direct-to-LDS copy of a 4-slot ring (input rows 0-103 -- the tile's 100
// pixels and 4 zero rows, 13 copies -- then the 64 output-gradient rows, 8
// copies) and never stores, so it keeps three stages in flight (63 copies:
// the vector-memory counter's limit) while waiting for the oldest; the four
// compute waves only wait on barriers, and their transposed LDS reads run a
// tap ahead of the MFMAs.  One block per CU.
constexpr int TAPW_IN = 104;                          // staged input pixel rows
constexpr int TAPW_IN_COPIES = TAPW_IN / 8;
constexpr int TAPW_COPIES = TAPW_IN_COPIES + 8;       // 21 per stage
constexpr int TAPW_STAGE = (TAPW_IN + 64) * 128;
constexpr int TAPW_NST = 4;
constexpr int TAPW_NT = 320;
static_assert((TAPW_NST - 1) * TAPW_COPIES <= 63, "vector-memory counter");

// Copy ins (0 .. 20) of the copy wave: rows 8 ins .. + 7 of the stage, 16-byte
// segment lane % 8 (global 16-byte unit u of the pixel in segment position
// u ^ 2 (p mod 4), i.e. 32-byte segments swizzled by pixel mod 4).
__host__ __device__ inline TapSlot tapw_slot(int W, int C, int Q, int K, int c0, int k0, int lane,
                                             int ins) {
  const int sl = lane & 7;
  TapSlot t;
  if (ins < TAPW_IN_COPIES) {
    const int pix = 8 * ins + (lane >> 3);  // < TAPW_IN
    const int u = 2 * ((sl >> 1) ^ (pix & 3)) + (sl & 1);
    const int ty = pix / 10, tx = pix - 10 * (pix / 10);
    t.sy = pix < 100 ? ty - 1 : -(1 << 24);
    t.sx = tx - 1;
    t.off = pix < 100 ? (t.sy * W + t.sx) * C + c0 + u * 8 : 0;
  } else {
    const int pix = 8 * (ins - TAPW_IN_COPIES) + (lane >> 3);
    const int u = 2 * ((sl >> 1) ^ (pix & 3)) + (sl & 1);
    t.sy = pix >> 3;
    t.sx = pix & 7;
    t.off = (t.sy * Q + t.sx) * K + k0 + u * 8;
  }
  return t;
}

// One stage's MFMAs of compute wave WAVE from the ring slot at smem: the wave
// is a template parameter, so each read's pixel offset is an immediate over
// one of the lane's base offsets -- ao[v][cg]: input pixel
// base + d with d = v mod 4, channel group cg (the 32-byte unit swizzle by
// pixel mod 4 included); bo[j]: output-gradient pixel, channel group j.
template <int WAVE>
__device__ __forceinline__ void tapw_stage(const char* smem, const int (&ao)[4][4],
                                           const int (&bo)[4], f32x4 (&acc)[9][4]) {
  constexpr int S0 = 0;
#pragma unroll
  for (int kf = 0; kf < 2; ++kf) {
    uint4 fb[4];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = kf * 32 + half * 4;  // output-gradient pixel offset
        const uint2 v = lds_read_tr16(smem + S0 + TAPW_IN * 128 + d * 128 + bo[j]);
        if (half == 0) { fb[j].x = v.x; fb[j].y = v.y; } else { fb[j].z = v.x; fb[j].w = v.y; }
      }
    }
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int T = 9 * WAVE + t, tap = T >> 2, cg = T & 3;
      const int r = tap / 3, s = tap - 3 * (tap / 3);
      uint4 fa;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int d = kf * 40 + r * 10 + half * 4 + s;  // input pixel offset from the lane's
        const uint2 v = lds_read_tr16(smem + S0 + d * 128 + ao[d & 3][cg]);
        if (half == 0) { fa.x = v.x; fa.y = v.y; } else { fa.z = v.x; fa.w = v.y; }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) mma_unit(acc[t][j], fa, fb[j], (bf16*)nullptr);
    }
  }
  // scheduling groups (0x100: LDS reads, 0x008: MFMAs): each k-step's
  // output-gradient fragments and first two input fragments, then a tap's
  // MFMAs beside the reads of the tap two ahead
#pragma unroll
  for (int kf = 0; kf < 2; ++kf) {
    __builtin_amdgcn_sched_group_barrier(0x100, 12, 0);
#pragma unroll
    for (int t = 0; t < 7; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
  }
}

// Compute wave WAVE's whole loop (its accumulators live in one arm of the
// kernel's switch on the wave) and its partial sums; the stage loop is
// one barrier before each stage.
template <int WAVE>
__device__ __forceinline__ void tapw_compute(const char* smem, int ns, int lane, float* out,
                                             long long RSC, int K, int c0, int k0, int split) {
  f32x4 acc[9][4];
#pragma unroll
  for (int i = 0; i < 9; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the lane's read offsets: input pixel base gq * 10 + jr of the staged
  // 10-wide tile, output-gradient pixel gq * 8 + jr of the patch (whose
  // pixel mod 4 is jr at every offset the stage adds)
  const int gq = lane >> 4, jr = (lane & 15) >> 2, qd = lane & 3;
  const int ib = gq * 10 + jr, ob = gq * 8 + jr;
  int ao[4][4], bo[4];
#pragma unroll
  for (int v = 0; v < 4; ++v)
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) ao[v][cg] = ib * 128 + ((cg ^ ((ib + v) & 3)) * 32) + qd * 8;
#pragma unroll
  for (int j = 0; j < 4; ++j) bo[j] = ob * 128 + ((j ^ jr) * 32) + qd * 8;
  for (int st = 0; st < ns; ++st) {
    stage_barrier();
    tapw_stage<WAVE>(smem + (st % TAPW_NST) * TAPW_STAGE, ao, bo, acc);
  }
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    const int T = 9 * WAVE + t, tap = T >> 2, cg = T & 3;
    const long long row = (long long)tap * (RSC / 9) + c0 + 16 * cg + 4 * lg;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = k0 + 16 * j + lr;
      float* dst = out + ((long long)split * K + col) * RSC + row;
      *reinterpret_cast<float4*>(dst) =
          make_float4(acc[t][j][0], acc[t][j][1], acc[t][j][2], acc[t][j][3]);
    }
  }
}

__global__ __launch_bounds__(TAPW_NT) void wgrad_tapw_kernel(WgTapArgs a) {
  static_assert(TAPW_NST - 2 <= 2, "c64_wait covers at most 2 later stages");
  __shared__ __align__(16) char smem[TAPW_NST * TAPW_STAGE];
  const int H = a.g.H, W = a.g.W, C = a.g.C, K = a.g.K, P = a.g.P, Q = a.g.Q, N = a.g.N;
  const int tiles_c = a.t.tiles_c, px_n = a.t.px_n, per_img = a.t.py_n * a.t.px_n;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tiles = tiles_c * a.t.tiles_k;
  const int item = xcd_tile(blockIdx.x, tiles * a.t.splits);
  const int split = item / tiles, tile = item - split * tiles;
  const int c0 = (tile % tiles_c) * 64, k0 = (tile / tiles_c) * 64;
  const int q0 = split * a.t.pps;
  const int ns = max(0, min(N * per_img, q0 + a.t.pps) - q0);

  if (wave == 4) {
    const void* const zero = g_zero_unit;
    auto issue = [&](int st) {
      const int q = q0 + st;
      const int n = q / per_img, rem = q - n * per_img;
      const int pyi = rem / px_n;
      const int py0 = 8 * pyi, px0 = 8 * (rem - pyi * px_n);
      const bf16* xb = a.x + ((long long)n * H * W + (long long)py0 * W + px0) * C;
      const bf16* db = a.dy + ((long long)n * P * Q + (long long)py0 * Q + px0) * K;
      char* slot = smem + (st % TAPW_NST) * TAPW_STAGE;
#pragma unroll
      for (int ins = 0; ins < TAPW_COPIES; ++ins) {
        const TapSlot sl = tapw_slot(W, C, Q, K, c0, k0, lane, ins);
        const bool x = ins < TAPW_IN_COPIES;
        const bool in = x ? (unsigned)(py0 + sl.sy) < (unsigned)H && (unsigned)(px0 + sl.sx) < (unsigned)W
                          : py0 + sl.sy < P && px0 + sl.sx < Q;
        const void* src = in ? (const void*)((x ? xb : db) + sl.off) : zero;
        dma16(src, reinterpret_cast<uint4*>(slot + ins * 1024));
      }
    };
    for (int st = 0; st < min(ns, TAPW_NST - 1); ++st) issue(st);
    for (int st = 0; st < ns; ++st) {
      c64_wait<TAPW_COPIES>(min(ns - 1 - st, TAPW_NST - 2));
      stage_barrier();
      // every compute wave is past stage st - 1: refill its slot
      if (st + TAPW_NST - 1 < ns) issue(st + TAPW_NST - 1);
    }
    return;
  }

  const long long RSC = 9LL * C;
  switch (wave) {
    case 0: tapw_compute<0>(smem, ns, lane, a.out, RSC, K, c0, k0, split); break;
    case 1: tapw_compute<1>(smem, ns, lane, a.out, RSC, K, c0, k0, split); break;
    case 2: tapw_compute<2>(smem, ns, lane, a.out, RSC, K, c0, k0, split); break;
    default: tapw_compute<3>(smem, ns, lane, a.out, RSC, K, c0, k0, split); break;
  }
}

// ---------------------------------------------- weight gradient of the stem
// dw[k][r][s][c] = sum over output pixels of dy[pix][k] * x(2p + r - 3,
// 2q + s - 3)[c] for the 7x7 / stride 2 / pad 3 stem on frames stored with
// channels padded to 8 (3 real).  A block owns every output (64 k x 49 taps x
// channels 0-3, the fourth a zero pad) and reduces over 8 x 8 patches of output
// pixels.  A stage stages the patch's 22 x 22 input pixels (channels 0-3,
// 8 bytes, through registers; rows of 24 pixels) and its 64 output-gradient
// pixels (128-byte rows, direct copies -- or, with the pooled BatchNorm
// backward folded in, computed and stored by the waves -- segments swizzled as
// in the all-taps kernel).  Taps are taken in 2 x 2 blocks (r and s from 0 to 7; taps 7
// compute into discarded rows): a 16-row MFMA tile is 4 taps x 4 channels,
// its transpose read has member m supply pixel m / 4 of tap m % 4, and with
// rows of 24 pixels the 16 members' 8-byte slots differ modulo 128 bytes
// (tap offsets 0, 1, 24, 25 plus twice the pixel index), so the read meets no
// bank conflict.  Wave w owns the 4 tap blocks of filter rows 2w, 2w + 1.
constexpr int STEM_WG_ROWS = 22, STEM_WG_PITCH = 24;
constexpr int STEM_WG_X = STEM_WG_ROWS * STEM_WG_PITCH * 8;  // input bytes per stage
constexpr int STEM_WG_STAGE = STEM_WG_X + 64 * 128;

// The stem's BatchNorm + ReLU + max-pool backward, for the weight gradient to
// form its output gradient itself (POOLBWD): dy at stem pixel (h, w) is the
// pooled gradient summed over the pool windows holding (h, w) whose stored
// index names it (windows in (r, s) order, the sum rounded to bf16 as the
// separate pool backward stores it), masked by ReLU (the mask recomputed
// from z: the rounded fma((z - mean), gamma * invstd, beta) > 0), then
// dz = coef0 * g + coef1 + coef2 * (z - mean) rounded to bf16 -- the
// BatchNorm backward with coefficients from its statistics pass.
struct StemPoolBwd {
  const bf16* z;       // BatchNorm input [N][P][Q][64]
  const bf16* dyp;     // pooled gradient [N][PP][PQ][64]
  const uint8_t* arg;  // window indices (r * 3 + s), same layout
  const float *mean, *coef, *gamma, *invstd, *beta;  // coef: [3][64]
  int PP, PQ;
};

struct StemWgArgs {
  ConvGeom g;
  const bf16* x;   // [N][H][W][8]
  const bf16* dy;  // [N][P][Q][64] (unused with POOLBWD)
  float* out;      // [split][64][49][4]
  int splits, pps, py_n, px_n;
  StemPoolBwd pb;
};

__device__ __forceinline__ void bf16x8_to_f(const uint4 u, float (&v)[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __builtin_bit_cast(float, w[i] << 16);
    v[2 * i + 1] = __builtin_bit_cast(float, w[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ uint32_t bf16x2_bits(float a, float b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (bf16)a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (bf16)b) << 16);
}

// With POOLBWD, wave w forms the output gradient of the stage's pixels of
// parity class w (row parity w >> 1, column parity w & 1), then of class
// 3 - w: 1 + 4 or 2 + 2 pool windows per pixel, the same class across the
// wave.  Lane l takes channel unit l % 8 of pixel l / 8 of its half of the
// class (16 pixels, two halves); its loads for the next stage are issued
// before this stage's MFMAs.
template <bool POOLBWD>
__global__ __launch_bounds__(NT, 2) void wgrad_stem_kernel(StemWgArgs a) {
  constexpr int NST = 2;
  __shared__ __align__(16) char smem[NST * STEM_WG_STAGE];
  const int H = a.g.H, W = a.g.W, P = a.g.P, Q = a.g.Q, N = a.g.N;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int split = xcd_tile(blockIdx.x, a.splits);
  const int per_img = a.py_n * a.px_n;
  const int q0 = split * a.pps;
  const int ns = max(0, min(N * per_img, q0 + a.pps) - q0);
  const void* const zero = g_zero_unit;
  // output-gradient copy slots: instructions wave and wave + 4 of the 8
  int dsy[2], dsx[2], doff[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int pix = 8 * (wave + 4 * j) + (lane >> 3), sl = lane & 7;
    const int u = 2 * ((sl >> 1) ^ (pix & 3)) + (sl & 1);
    dsy[j] = pix >> 3;
    dsx[j] = pix & 7;
    doff[j] = (dsy[j] * Q + dsx[j]) * 64 + u * 8;
  }
  auto origin = [&](int st, int& n, int& py0, int& px0) {
    const int q = q0 + st;
    n = q / per_img;
    const int rem = q - n * per_img, pyi = rem / a.px_n;
    py0 = 8 * pyi;
    px0 = 8 * (rem - pyi * a.px_n);
  };
  // input pixels t and t + 256 of the 22 x 22 region, as registers
  uint4 xv[2];
  auto load_x = [&](int st) {
    int n, py0, px0;
    origin(st, n, py0, px0);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int t = threadIdx.x + 256 * h;
      const int ry = t / STEM_WG_ROWS, rx = t - STEM_WG_ROWS * (t / STEM_WG_ROWS);
      const int iy = 2 * py0 - 3 + ry, ix = 2 * px0 - 3 + rx;
      const bool in = t < STEM_WG_ROWS * STEM_WG_ROWS && (unsigned)iy < (unsigned)H &&
                      (unsigned)ix < (unsigned)W;
      xv[h] = in ? *reinterpret_cast<const uint4*>(a.x + (((long long)n * H + iy) * W + ix) * 8)
                 : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  auto store_x = [&](char* slot) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int t = threadIdx.x + 256 * h;
      if (t < STEM_WG_ROWS * STEM_WG_ROWS) {
        const int ry = t / STEM_WG_ROWS, rx = t - STEM_WG_ROWS * (t / STEM_WG_ROWS);
        *reinterpret_cast<uint2*>(slot + (ry * STEM_WG_PITCH + rx) * 8) = make_uint2(xv[h].x, xv[h].y);
      }
    }
  };
  auto issue_dy = [&](int st, char* slot) {
    int n, py0, px0;
    origin(st, n, py0, px0);
    const bf16* db = a.dy + ((long long)n * P * Q + (long long)py0 * Q + px0) * 64;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const bool in = py0 + dsy[j] < P && px0 + dsx[j] < Q;
      dma16(in ? (const void*)(db + doff[j]) : zero,
            reinterpret_cast<uint4*>(slot + STEM_WG_X + (wave + 4 * j) * 1024));
    }
  };

  // POOLBWD: channel unit u of the lane, its per-channel constants, and the
  // next stage's z and pool-window loads
  const int pu = lane & 7;
  float pmu[8], psc[8], pbe[8], pca[8], pcb[8], pcc[8];
  if (POOLBWD) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int c = 8 * pu + i;
      pmu[i] = a.pb.mean[c];
      psc[i] = a.pb.gamma[c] * a.pb.invstd[c];
      pbe[i] = a.pb.beta[c];
      pca[i] = a.pb.coef[c];
      pcb[i] = a.pb.coef[64 + c];
      pcc[i] = a.pb.coef[128 + c];
    }
  }
  uint4 pz[2], pg[2][4];
  uint2 pa[2][4];
  // stage pixel of half j: class cls = (j ? 3 - wave : wave), pixel k = 8 j + lane / 8 of it
  auto pix_of = [&](int j, int& dsy, int& dsx) {
    const int cls = j ? 3 - wave : wave, k = 8 * j + (lane >> 3);
    dsy = 2 * (k >> 2) + (cls >> 1);
    dsx = 2 * (k & 3) + (cls & 1);
  };
  auto pb_load = [&](int st) {
    int n, py0, px0;
    origin(st, n, py0, px0);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int cls = j ? 3 - wave : wave, hp = cls >> 1, wp = cls & 1;
      int dsy, dsx;
      pix_of(j, dsy, dsx);
      const int h = py0 + dsy, w = px0 + dsx;
      const bool in = h < P && w < Q;
      pz[j] = in ? *reinterpret_cast<const uint4*>(a.pb.z + (((long long)n * P + h) * Q + w) * 64 + 8 * pu)
                 : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
      for (int kr = 0; kr < 2; ++kr)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          if (kr > hp || ks > wp) continue;  // wave-uniform
          // odd row: window row r = 0 of pooled row h / 2 + 1, then r = 2 of h / 2;
          // odd column likewise with s; even: r (s) = 1 of h / 2 (w / 2)
          const int pr = (h >> 1) + (hp && kr == 0 ? 1 : 0);
          const int pc = wp ? (ks == 0 ? (w + 1) >> 1 : (w - 1) >> 1) : (w >> 1);
          const bool ok = in && pr < a.pb.PP && pc < a.pb.PQ;
          const long long off = (((long long)n * a.pb.PP + pr) * a.pb.PQ + pc) * 64 + 8 * pu;
          pg[j][2 * kr + ks] = ok ? *reinterpret_cast<const uint4*>(a.pb.dyp + off) : make_uint4(0u, 0u, 0u, 0u);
          pa[j][2 * kr + ks] = ok ? *reinterpret_cast<const uint2*>(a.pb.arg + off)
                                  : make_uint2(0xFFFFFFFFu, 0xFFFFFFFFu);
        }
    }
  };
  // the output gradient from the loaded values, into the stage's LDS slot
  auto pb_store = [&](char* slot) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int cls = j ? 3 - wave : wave, hp = cls >> 1, wp = cls & 1;
      int dsy, dsx;
      pix_of(j, dsy, dsx);
      float zz[8], acc8[8];
      bf16x8_to_f(pz[j], zz);
#pragma unroll
      for (int i = 0; i < 8; ++i) acc8[i] = 0.f;
#pragma unroll
      for (int kr = 0; kr < 2; ++kr)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          if (kr > hp || ks > wp) continue;  // wave-uniform
          const int r = hp ? 2 * kr : 1, sw = wp ? 2 * ks : 1, code = r * 3 + sw;
          float gv[8];
          bf16x8_to_f(pg[j][2 * kr + ks], gv);
          const uint2 av = pa[j][2 * kr + ks];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int ai = (int)(((i < 4 ? av.x : av.y) >> (8 * (i & 3))) & 0xFFu);
            if (ai == code) acc8[i] += gv[i];
          }
        }
      float o[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float g = (float)(bf16)acc8[i];
        const float t = __builtin_fmaf(zz[i] - pmu[i], psc[i], pbe[i]);
        const float gm = (float)(bf16)t > 0.f ? g : 0.f;
        o[i] = pca[i] * gm + pcb[i] + pcc[i] * (zz[i] - pmu[i]);
      }
      const int pix = dsy * 8 + dsx, pos = 2 * ((pu >> 1) ^ (pix & 3)) + (pu & 1);
      *reinterpret_cast<uint4*>(slot + STEM_WG_X + pix * 128 + pos * 16) =
          make_uint4(bf16x2_bits(o[0], o[1]), bf16x2_bits(o[2], o[3]), bf16x2_bits(o[4], o[5]),
                     bf16x2_bits(o[6], o[7]));
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (ns > 0) {
    load_x(0);
    if (POOLBWD)
      pb_load(0);
    else
      issue_dy(0, smem);
    wait_vmcnt<0>();
    store_x(smem);
    if (POOLBWD) pb_store(smem);
  }
  const int gq = lane >> 4, jr = (lane & 15) >> 2, qd = lane & 3;
  for (int st = 0; st < ns; ++st) {
    stage_barrier();  // stage st's input rows (stores) and copies are in LDS
    const bool next = st + 1 < ns;
    char* nslot = smem + ((st + 1) % NST) * STEM_WG_STAGE;
    if (next) {
      load_x(st + 1);
      if (POOLBWD)
        pb_load(st + 1);
      else
        issue_dy(st + 1, nslot);
    }
    const char* Xs = smem + (st % NST) * STEM_WG_STAGE;
    const char* Bs = Xs + STEM_WG_X;
#pragma unroll
    for (int kf = 0; kf < 2; ++kf) {
      const int py = kf * 4 + gq;
      uint4 fb[4];
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int p = py * 8 + half * 4 + jr;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint2 v = lds_read_tr16(Bs + p * 128 + ((j ^ (p & 3)) * 32) + qd * 8);
          if (half == 0) { fb[j].x = v.x; fb[j].y = v.y; } else { fb[j].z = v.x; fb[j].w = v.y; }
        }
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        // tap block (filter rows 2 wave, 2 wave + 1; columns 2t, 2t + 1); this
        // member's tap within it is qd
        const int r = 2 * wave + (qd >> 1), sc = 2 * t + (qd & 1);
        uint4 fa;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int px = half * 4 + jr;
          const uint2 v =
              lds_read_tr16(Xs + ((2 * py + r) * STEM_WG_PITCH + 2 * px + sc) * 8);
          if (half == 0) { fa.x = v.x; fa.y = v.y; } else { fa.z = v.x; fa.w = v.y; }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) mma_unit(acc[t][j], fa, fb[j], (bf16*)nullptr);
      }
    }
    if (next) {
      wait_vmcnt<0>();
      store_x(nslot);  // that slot was last read before this stage's barrier
      if (POOLBWD) pb_store(nslot);
    }
  }

  // lane rows 4 lg .. 4 lg + 3 of a tile are tap lg of the block, channels 0-3
  const int lr = lane & 15, lg = lane >> 4;
  const int r = 2 * wave + (lg >> 1);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int sc = 2 * t + (lg & 1);
    if (r < 7 && sc < 7) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int k = 16 * j + lr;
        float* dst = a.out + (((long long)split * 64 + k) * 49 + r * 7 + sc) * 4;
        *reinterpret_cast<float4*>(dst) =
            make_float4(acc[t][j][0], acc[t][j][1], acc[t][j][2], acc[t][j][3]);
      }
    }
  }
}

// Warp-specialised weight gradient for BM = 256 rows (channels of one filter
// tap, so C % 256 == 0) x BN output channels: four loader waves gather the
// stage's 64 input-pixel rows and 64 output-gradient rows (same LDS layout as
// above) NST - 1 stages ahead; the compute waves (64 x 64 each) read the
// operands with LDS transpose reads and issue the MFMAs.  A loader lane keeps
// its input pixel as (n, p, q) plus a 32-bit element offset, stepped by 64
// pixels per stage.  Barriers as in gemm_ws_kernel.
template <int BM, int BN, int NST>
__global__ __launch_bounds__((BM / 64) * (BN / 64) * 64 + WS_LOADERS * 64) void wgrad_ws_kernel(
    WgDmaArgs a) {
  constexpr int WGN = BN / 64, CW = (BM / 64) * WGN;
  constexpr int UA = BM / 8, UB = BN / 8;     // 16-byte units per pixel row
  constexpr int RA = 64 / UA, RB = 64 / UB;   // pixel rows per copy instruction
  constexpr int IA = 64 / RA, IB = 64 / RB;   // copy instructions per stage
  constexpr int LPS = (IA + IB) / 4, LA = IA / 4;
  static_assert(IA % 4 == 0 && IB % 4 == 0, "instructions split over 4 loader waves");
  static_assert(LPS * (NST - 2) < 64, "vmcnt range");
  constexpr int SA = BM / 16, SB = BN / 16;   // 32-byte segments per row
  constexpr int STAGE_BYTES = 64 * (BM + BN) * 2;
  __shared__ __align__(16) char smem[NST * STAGE_BYTES];

  const ConvGeom& g = a.g;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tiles = a.tiles_m * a.tiles_n;
  const int item = xcd_tile(blockIdx.x, tiles * a.splits);
  const int split = item / tiles, t = item - split * tiles;
  const int m0 = (t % a.tiles_m) * BM, n0 = (t / a.tiles_m) * BN;
  const int M = g.N * g.P * g.Q;
  const int mb = split * a.m_per_split;
  const int me = min(M, mb + a.m_per_split);
  const int ns = me > mb ? (me - mb + 63) / 64 : 0;

  if (wave >= CW) {
    const int lw = wave - CW;
    const void* zero = g_zero_unit;
    asm volatile("" : "+s"(zero));
    const int rs = m0 / g.C, c0 = m0 - rs * g.C;
    const int tr = rs / g.S, ts = rs - tr * g.S;
    const int PQ = g.P * g.Q;
    const int dq = 64 % g.Q, dp = (64 / g.Q) % g.P, dn = 64 / PQ;
    const int sC = g.stride * g.C, sWC = g.stride * g.W * g.C, HWC = g.H * g.W * g.C;
    int am[LA], pp[LA], qq[LA], xo[LA];
#pragma unroll
    for (int j = 0; j < LA; ++j) {
      const int pr = (lw + 4 * j) * RA + lane / UA;
      am[j] = mb + pr;
      const int m = am[j] < M ? am[j] : 0;
      const int n = m / PQ, rem = m - n * PQ;
      pp[j] = rem / g.Q;
      qq[j] = rem - pp[j] * g.Q;
      // element offset of input pixel (n, p stride - pad + tr, q stride - pad + ts), channel c0
      xo[j] = n * HWC + ((pp[j] * g.stride - g.pad + tr) * g.W + qq[j] * g.stride - g.pad + ts) * g.C + c0;
    }
    auto issue = [&](int st, char* slot) {
#pragma unroll
      for (int j = 0; j < LPS; ++j) {
        const int ins = lw + 4 * j;
        if (j < LA) {
          const int pr = ins * RA + lane / UA, sl = lane % UA;
          const int u = 2 * ((sl >> 1) ^ (pr % SA)) + (sl & 1);
          const int h = pp[j] * g.stride - g.pad + tr, w = qq[j] * g.stride - g.pad + ts;
          const bool in = am[j] < me && (unsigned)h < (unsigned)g.H && (unsigned)w < (unsigned)g.W;
          dma16(in ? (const void*)(a.x + xo[j] + u * 8) : zero,
                reinterpret_cast<uint4*>(slot + ins * 1024));
          am[j] += 64;
          qq[j] += dq;
          xo[j] += dq * sC;
          if (qq[j] >= g.Q) {
            qq[j] -= g.Q;
            ++pp[j];
            xo[j] += sWC - g.Q * sC;
          }
          pp[j] += dp;
          xo[j] += dp * sWC;
          if (pp[j] >= g.P) {
            pp[j] -= g.P;
            xo[j] += HWC - g.P * sWC;
          }
          xo[j] += dn * HWC;
        } else {
          const int ib = ins - IA;
          const int pr = ib * RB + lane / UB, sl = lane % UB;
          const int u = 2 * ((sl >> 1) ^ (pr % SB)) + (sl & 1);
          const int m = mb + st * 64 + pr;
          dma16(m < me ? (const void*)(a.dy + m * g.K + n0 + u * 8) : zero,
                reinterpret_cast<uint4*>(slot + 64 * BM * 2 + ib * 1024));
        }
      }
    };
#pragma unroll
    for (int p = 0; p < NST - 1; ++p)
      if (p < ns) issue(p, smem + p * STAGE_BYTES);
    if (NST - 2 < ns)
      wait_vmcnt<LPS * (NST - 2)>();
    else
      wait_vmcnt<0>();
    stage_barrier();
    int slot = 0;
    for (int st = 0; st < ns; ++st) {
      if (st + NST - 1 < ns) {
        const int nslot = slot == 0 ? NST - 1 : slot - 1;
        issue(st + NST - 1, smem + nslot * STAGE_BYTES);
        wait_vmcnt<LPS * (NST - 2)>();  // stage st + 1 has landed
      } else {
        wait_vmcnt<0>();
      }
      stage_barrier();
      if (++slot == NST) slot = 0;
    }
    return;
  }

  const int wm = wave / WGN, wn = wave % WGN;
  const int gq = lane >> 4, jr = (lane & 15) >> 2, qd = lane & 3;
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  stage_barrier();
  int slot = 0;
  for (int st = 0; st < ns; ++st) {
    const char* As = smem + slot * STAGE_BYTES;
    const char* Bs = As + 64 * BM * 2;
#pragma unroll
    for (int kf = 0; kf < 2; ++kf) {
      uint4 fa[4], fb[4];
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int pr = kf * 32 + gq * 8 + half * 4 + jr;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int ch = wm * 64 + i * 16 + 4 * qd;
          const uint2 v = lds_read_tr16(As + pr * (BM * 2) + (((ch >> 4) ^ (pr % SA)) * 32) +
                                        (ch & 15) * 2);
          if (half == 0) { fa[i].x = v.x; fa[i].y = v.y; } else { fa[i].z = v.x; fa[i].w = v.y; }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int ch = wn * 64 + j * 16 + 4 * qd;
          const uint2 v = lds_read_tr16(Bs + pr * (BN * 2) + (((ch >> 4) ^ (pr % SB)) * 32) +
                                        (ch & 15) * 2);
          if (half == 0) { fb[j].x = v.x; fb[j].y = v.y; } else { fb[j].z = v.x; fb[j].w = v.y; }
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) mma_unit(acc[i][j], fa[i], fb[j], (bf16*)nullptr);
    }
    stage_barrier();
    if (++slot == NST) slot = 0;
  }

  const int RSC = g.R * g.S * g.C;
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = m0 + wm * 64 + i * 16 + 4 * lg, col = n0 + wn * 64 + j * 16 + lr;
      float* dst = a.out + ((long long)split * g.K + col) * RSC + row;
      *reinterpret_cast<float4*>(dst) =
          make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
}

// ------------------------------------------------------------- image stem
// bf16 7x7 / stride 2 / pad 3 convolution of 3-channel frames (stored with
// channels padded to 8) into 64 channels, for output rows up to 112 wide.
// A block of 8 waves computes 8 output rows (one per wave) x the full row
// width x all 64 channels.  The 21 input rows it needs (8 x 2 + 5)
// are staged in LDS once, keeping channels 0..3 of each pixel (8 bytes;
// channel 3 is the zero pad), and the filter as [64][7][8 taps][4] with the
// 8th tap zero.  One MFMA k-step covers one filter row r: 8 taps x 4 channels
// = 32 products, so a lane's 16-byte operand is 2 adjacent taps x 4 channels
// -- 2 adjacent input pixels in the staged row, contiguous -- and 7 k-steps
// cover the filter (224 products per output, against 392 with 8 stored
// channels).  Global reads are batched 8 per thread before their LDS writes.
constexpr int STEM_QMAX = 112, STEM_TQ = 7, STEM_PATCH_W = 2 * STEM_TQ * 16 + 6;
constexpr int STEM_ROWS = 8, STEM_IN_ROWS = 2 * STEM_ROWS + 5;
constexpr int STEM_WROW = 232;  // 224 filter entries per channel + 8 (bank spread)

constexpr int STEM_NT = 512;

// The eval-mode stem followed by the 3x3 / stride 2 / pad 1 max pool (POOL):
// a block produces 4 pool rows (4 b .. 4 b + 3) of one image from the 9 stem
// rows 8 b - 1 .. 8 b + 7 (9 waves, one row each; rows outside the image are
// skipped).  After the epilogue each wave takes, for every pool column c,
// the maximum over stem columns 2 c - 1, 2 c, 2 c + 1 (the neighbouring
// columns come from the adjacent lanes of a 16-lane row, and for column
// 16 t - 1 from lane 15 of block t - 1, by DPP rotations), rounds it to bf16
// and writes the 56-column row to LDS, over the staged input; the block then
// takes the maximum over the 3 stem rows of each pool row.  Maxima skip NaNs
// (start from -inf and take greater values), as the separate max pool does;
// rounding is monotone, so the result equals pooling the rounded stem output.
constexpr int SP_QMAX = STEM_QMAX / 2;  // pool columns
__device__ __forceinline__ float gt_max(float m, float v) { return v > m ? v : m; }

// One wave's share of a stem output row: column blocks T0 .. T0 + TN - 1
// (16 columns each) for all 64 channels, written straight to y with the
// epilogue applied.  A row is done in two such parts so the accumulators take
// 64 registers, not 112, and two blocks fit on a CU; the first part's stores
// are in flight while the second part runs its MFMAs.
template <int T0, int TN>
__device__ __forceinline__ void stem_row_part(const bf16* wl, const uint2* prow0, int lr, int kc,
                                              int tq, int Q, bf16* yrow, const ConvEpilogue& epi) {
  if (T0 >= tq) return;  // wave-uniform
  f32x4 acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < TN; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
  for (int r = 0; r < 7; ++r) {
    uint4 fa[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      fa[i] = *reinterpret_cast<const uint4*>(wl + (i * 16 + lr) * STEM_WROW + r * 32 + kc * 8);
    const uint2* prow = prow0 + r * STEM_PATCH_W;
    uint4 fb[TN];
#pragma unroll
    for (int t = 0; t < TN; ++t)
      fb[t] = *reinterpret_cast<const uint4*>(prow + 2 * ((T0 + t) * 16 + lr) + 2 * kc);
#pragma unroll
    for (int t = 0; t < TN; ++t) {
      if (T0 + t < tq) {
#pragma unroll
        for (int i = 0; i < 4; ++i) mma_unit(acc[i][t], fa[i], fb[t], (bf16*)nullptr);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < TN; ++t) {
    const int q = (T0 + t) * 16 + lr;
    if (T0 + t >= tq || q >= Q) continue;
    bf16* dst = yrow + (long long)q * 64;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = i * 16 + 4 * kc;
      float v[4] = {acc[i][t][0], acc[i][t][1], acc[i][t][2], acc[i][t][3]};
      if (epi.scale) {
        const float4 s4 = *reinterpret_cast<const float4*>(epi.scale + k);
        v[0] *= s4.x; v[1] *= s4.y; v[2] *= s4.z; v[3] *= s4.w;
      }
      if (epi.shift) {
        const float4 b4 = *reinterpret_cast<const float4*>(epi.shift + k);
        v[0] += b4.x; v[1] += b4.y; v[2] += b4.z; v[3] += b4.w;
      }
      if (epi.relu) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = relu_nan(v[e]);
      }
      store4<bf16>(dst + k, v);
    }
  }
}

// RAW: x is [.][H][W][3] frames (image n at idx[n] when idx != null) read
// with three 2-byte loads per pixel, instead of the 8-channel padded input.
template <bool RAW, bool POOL = false>
__global__ __launch_bounds__(STEM_NT + (POOL ? 64 : 0), POOL ? 1 : 4) void stem_kernel(
    const bf16* x, const int32_t* idx, const bf16* wk, bf16* y, ConvEpilogue epi, int N, int H,
    int W, int P, int Q) {
  constexpr int ROWS = POOL ? STEM_ROWS + 1 : STEM_ROWS, NT = ROWS * 64;
  constexpr int IN_ROWS = 2 * ROWS + 5;
  constexpr int PATCH_BYTES = IN_ROWS * STEM_PATCH_W * 8, W_BYTES = 64 * STEM_WROW * 2;
  constexpr int POOL_BYTES = POOL ? ROWS * SP_QMAX * 64 * 2 : 0;
  constexpr int LDS_BYTES = PATCH_BYTES + W_BYTES > POOL_BYTES ? PATCH_BYTES + W_BYTES : POOL_BYTES;
  static_assert(PATCH_BYTES % 16 == 0, "filter alignment");
  __shared__ __align__(16) char lds[LDS_BYTES];
  uint2* patch = reinterpret_cast<uint2*>(lds);                // 4 channels per pixel
  bf16* wl = reinterpret_cast<bf16*>(lds + PATCH_BYTES);
  const int PP = (P - 1) / 2 + 1, PQ = (Q - 1) / 2 + 1;  // pool output (POOL)
  const int blocks_per_img = POOL ? cdiv(PP, 4) : cdiv(P, STEM_ROWS);
  const int n = blockIdx.x / blocks_per_img, bq = blockIdx.x % blocks_per_img;
  const int p0 = POOL ? 8 * bq - 1 : bq * STEM_ROWS;  // first stem row of the block
  const int tq = cdiv(Q, 16);
  const int pw = 2 * tq * 16 + 6;
  // filter: wk is [64][7][7][8]; keep channels 0..3, tap 7 zero
  for (int i0 = threadIdx.x; i0 < 64 * 7 * 8; i0 += 8 * NT) {
    uint2 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * NT, k = i / 56, r = (i % 56) / 8, sp = i % 8;
      v[u] = (i < 64 * 56 && sp < 7) ? *reinterpret_cast<const uint2*>(wk + ((k * 7 + r) * 7 + sp) * 8)
                                     : make_uint2(0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * NT;
      if (i < 64 * 56)
        *reinterpret_cast<uint2*>(wl + (i / 56) * STEM_WROW + ((i % 56) / 8) * 32 + (i % 8) * 4) = v[u];
    }
  }
  // input rows 2 p0 - 3 .. 2 p0 + 2 ROWS + 1, columns -3 .. pw - 4 (zero outside the frame)
  const long long img_n = (RAW && idx) ? idx[n] : n;
  const bf16* img = x + img_n * H * W * (RAW ? 3 : 8);
  // wave v stages rows v, v + ROWS, v + 2 ROWS; lane l columns l + 64 u
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  static_assert(IN_ROWS <= 3 * ROWS && STEM_PATCH_W <= 4 * 64, "staging covers the patch");
  {
    uint2 v[3][4];
#pragma unroll
    for (int rr = 0; rr < 3; ++rr)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int pr = wave + rr * ROWS, pc = lane + 64 * u;
        const int h = 2 * p0 - 3 + pr, w = pc - 3;
        const bool in = pr < IN_ROWS && pc < pw && (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
        if (RAW) {
          const unsigned short* px =
              reinterpret_cast<const unsigned short*>(img + ((long long)h * W + w) * 3);
          v[rr][u] = in ? make_uint2((unsigned)px[0] | ((unsigned)px[1] << 16), (unsigned)px[2])
                        : make_uint2(0u, 0u);
        } else {
          v[rr][u] = in ? *reinterpret_cast<const uint2*>(img + ((long long)h * W + w) * 8)
                        : make_uint2(0u, 0u);
        }
      }
#pragma unroll
    for (int rr = 0; rr < 3; ++rr)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int pr = wave + rr * ROWS, pc = lane + 64 * u;
        if (pr < IN_ROWS && pc < pw) patch[pr * STEM_PATCH_W + pc] = v[rr][u];
      }
  }
  __syncthreads();

  const int lr = lane & 15, kc = lane >> 4;
  if constexpr (!POOL) {
    const int p = p0 + wave;
    if (p >= P) return;
    bf16* yrow = y + ((long long)n * P + p) * Q * 64;
    const uint2* prow0 = patch + 2 * wave * STEM_PATCH_W;
    stem_row_part<0, 4>(wl, prow0, lr, kc, tq, Q, yrow, epi);
    stem_row_part<4, STEM_TQ - 4>(wl, prow0, lr, kc, tq, Q, yrow, epi);
    return;
  }
  {
    const int lp = wave;  // output row within the block
    const int p = p0 + lp;
    const bool row_ok = p >= 0 && p < P;
    if (!POOL && !row_ok) return;
    f32x4 acc[4][STEM_TQ];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int t = 0; t < STEM_TQ; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
    for (int r = 0; r < (row_ok ? 7 : 0); ++r) {
      uint4 fa[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        fa[i] = *reinterpret_cast<const uint4*>(wl + (i * 16 + lr) * STEM_WROW + r * 32 + kc * 8);
      const uint2* prow = patch + (2 * lp + r) * STEM_PATCH_W;
      // output column q = 16 t + lr reads input columns 2 q - 3 + 2 kc, +1; all
      // seven fragments are read first (in bounds of the staged row for every
      // t) so the LDS latency is paid once per filter row
      uint4 fb[STEM_TQ];
#pragma unroll
      for (int t = 0; t < STEM_TQ; ++t)
        fb[t] = *reinterpret_cast<const uint4*>(prow + 2 * (t * 16 + lr) + 2 * kc);
#pragma unroll
      for (int t = 0; t < STEM_TQ; ++t) {
        if (t < tq) {
#pragma unroll
          for (int i = 0; i < 4; ++i) mma_unit(acc[i][t], fa[i], fb[t], (bf16*)nullptr);
        }
      }
    }
    const int lg = lane >> 4;
    if constexpr (POOL) {
      __syncthreads();  // the staged input is dead: LDS now takes the pooled rows
      bf16* prow = reinterpret_cast<bf16*>(lds) + lp * (SP_QMAX * 64);
      float prev[4][4];  // epilogue values of column block t - 1
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) prev[i][e] = -INFINITY;
#pragma unroll
      for (int t = 0; t < STEM_TQ; ++t) {
        if (!row_ok || t >= tq) continue;  // wave-uniform
        const int q = t * 16 + lr;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = i * 16 + 4 * lg;
          float v[4] = {acc[i][t][0], acc[i][t][1], acc[i][t][2], acc[i][t][3]};
          if (epi.scale) {
            const float4 s4 = *reinterpret_cast<const float4*>(epi.scale + k);
            v[0] *= s4.x; v[1] *= s4.y; v[2] *= s4.z; v[3] *= s4.w;
          }
          if (epi.shift) {
            const float4 b4 = *reinterpret_cast<const float4*>(epi.shift + k);
            v[0] += b4.x; v[1] += b4.y; v[2] += b4.z; v[3] += b4.w;
          }
          if (epi.relu) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = relu_nan(v[e]);
          }
          float m[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            // every lane evaluates all three rotations, then selects
            const float lsame = row_ror<1>(v[e]), lprev = row_ror<1>(prev[i][e]);
            const float right = row_ror<15>(v[e]);
            const float left = lr == 0 ? lprev : lsame;
            float b = gt_max(-INFINITY, v[e]);
            if (q >= 1) b = gt_max(b, left);
            if (q + 1 < Q) b = gt_max(b, right);
            m[e] = b;
            prev[i][e] = v[e];
          }
          if ((lr & 1) == 0 && q < Q) store4<bf16>(prow + (q >> 1) * 64 + k, m);
        }
      }
      __syncthreads();
      // pool row 4 bq + m0 = max over stem rows p0 + 2 m0 .. + 2 (local rows)
      const int units = 4 * PQ * 8;
      for (int u = threadIdx.x; u < units; u += NT) {
        const int m0 = u / (PQ * 8), rem = u % (PQ * 8), c = rem / 8, cu = rem % 8;
        const int pr = 4 * bq + m0;
        if (pr >= PP) continue;
        float best[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) best[e] = -INFINITY;
#pragma unroll
        for (int d = 0; d < 3; ++d) {
          const int lrow = 2 * m0 + d, sp = p0 + lrow;
          if (sp < 0 || sp >= P) continue;
          const uint4 w4 = *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16*>(lds) +
                                                           (lrow * SP_QMAX + c) * 64 + cu * 8);
          float f0[4], f1[4];
          unpack4(make_uint2(w4.x, w4.y), f0);
          unpack4(make_uint2(w4.z, w4.w), f1);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            best[e] = gt_max(best[e], f0[e]);
            best[4 + e] = gt_max(best[4 + e], f1[e]);
          }
        }
        bf16* dst = y + (((long long)n * PP + pr) * PQ + c) * 64 + cu * 8;
        float lo4[4] = {best[0], best[1], best[2], best[3]}, hi4[4] = {best[4], best[5], best[6], best[7]};
        store4<bf16>(dst, lo4);
        store4<bf16>(dst + 4, hi4);
      }
    }
  }
}

// -------------------------------------------------------------- launching
thread_local KernelTimer* t_timer = nullptr;

template <typename T> const char* tname();
template <> const char* tname<float>() { return "f32"; }
template <> const char* tname<bf16>() { return "bf16"; }
template <template <typename, int, int, int, bool> class PolT> const char* pname();
template <> const char* pname<FwdPolicy>() { return "conv_fwd"; }
template <> const char* pname<DgradPolicy>() { return "conv_dgrad"; }
template <> const char* pname<WgradPolicy>() { return "conv_wgrad"; }

// Algorithmic cost of a conv: 2*N*P*Q*K*R*S*C0 flops; bytes = input + weights + output.
struct Cost {
  double flops, bytes;
};

Cost conv_cost(const ConvGeom& g, int C0, size_t es, bool fp32_out) {
  const double m = (double)g.N * g.P * g.Q;
  Cost c;
  c.flops = 2.0 * m * g.K * g.R * g.S * C0;
  const double x = (double)g.N * g.H * g.W * g.C, w = (double)g.K * g.R * g.S * g.C,
               y = m * g.K;
  c.bytes = (x + y) * es + w * (fp32_out ? 4.0 : (double)es);
  return c;
}

template <typename T, template <typename, int, int, int, bool> class PolT, int BM, int BN, int KU,
          bool UT>
hipError_t launch_gemm(const typename PolT<T, BM, BN, KU, UT>::Args& args, int rows, int cols,
                       int splits, hipStream_t stream, Cost cost) {
  dim3 grid(cdiv(cols, BN), cdiv(rows, BM), splits);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, PolT<T, BM, BN, KU, UT>>), grid, dim3(NT), 0, stream,
                     args);
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({std::string(pname<PolT>()) + "<" + tname<T>() + "," + std::to_string(BM) +
                           "," + std::to_string(BN) + (UT ? "" : ",gather") + ">",
                       cost.flops, cost.bytes, e0, e1});
  }
  return e;
}

// Tile and split for a rows x cols output with `ns` reduction stages: the
// largest tile that yields enough blocks for the chip, else split the
// reduction (keeping >= 4 stages per split).
struct Plan {
  int bm, bn, splits, sps;
};
constexpr long long kTargetBlocks = 512;

Plan plan_tiles(int rows, int cols, int ns, bool allow_split) {
  Plan p{64, 64, 1, ns};
  const int cand[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
  for (auto& c : cand) {
    if (c[0] == 128 && rows < 128) continue;
    const long long blocks = (long long)cdiv(cols, c[1]) * cdiv(rows, c[0]);
    if (blocks >= kTargetBlocks) {
      p.bm = c[0];
      p.bn = c[1];
      return p;
    }
  }
  // too few tiles: 128-row tiles when possible, split the reduction
  p.bm = rows >= 128 ? 128 : 64;
  p.bn = 64;
  const long long blocks = (long long)cdiv(cols, p.bn) * cdiv(rows, p.bm);
  if (allow_split) {
    int s = (int)std::min<long long>(cdivl(kTargetBlocks, blocks), std::max(1, ns / 4));
    s = std::max(1, std::min(s, 16));
    p.sps = cdiv(ns, s);
    p.splits = cdiv(ns, p.sps);
  }
  return p;
}

template <typename T, template <typename, int, int, int, bool> class PolT, int KU, bool UT>
hipError_t dispatch_tile(const typename PolT<T, 64, 64, KU, UT>::Args& args, const Plan& p,
                         int rows, int cols, hipStream_t stream, Cost cost) {
#define EKYA_TILE(BM_, BN_)                                                                    \
  if (p.bm == BM_ && p.bn == BN_)                                                              \
    return launch_gemm<T, PolT, BM_, BN_, KU, UT>(args, rows, cols, p.splits, stream, cost);
  EKYA_TILE(64, 64)
  EKYA_TILE(64, 128)
  EKYA_TILE(128, 64)
  EKYA_TILE(128, 128)
#undef EKYA_TILE
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t split_finish(const float* part, int splits, long long npix, int C, const ConvEpilogue& e,
                        void* y, hipStream_t stream) {
  const long long n4 = npix * C / 4;
  const int blocks = (int)std::min<long long>(cdivl(n4, 256), 8192);
  hipLaunchKernelGGL(split_reduce_kernel<T>, dim3(blocks), dim3(256), 0, stream, part, splits,
                     npix, C, e, (T*)y);
  return hipGetLastError();
}

// Direct-to-LDS GEMM planning: (BM, BN, blocks per CU) candidates, the first
// that fills the chip twice over without splitting, else 128-row tiles with
// the reduction split until ~400 blocks (>= 4 stages per split).
struct DmaPlan {
  int bm, bn, splits, sps;
  bool ws = false;  // warp-specialised kernel (always for bm = 256)
};

DmaPlan plan_dma(int rows, long long cols, int ns, bool allow_split) {
  // warp-specialised 128 x 256 tiles for 128 rows when they fill the chip
  // without a split and the reduction is long enough (>= 16 stages) to
  // amortise the pipeline fill
  if (rows == 128 && ns >= 16 && cdivl(cols, 256) >= 256) return {128, 256, 1, ns, true};
  if (rows % 256 == 0 && ns >= 8) {
    // warp-specialised 256 x 128 tiles, one block per CU: split the
    // reduction until the blocks about fill the chip once (>= 4 stages
    // each) -- unless there are fewer than a quarter chip of them and
    // 128 x 64 tiles already give half a chip of blocks without a split,
    // which saves the fp32 partials' round trip (measured: at 98 tiles, e.g.
    // 512 channels x 6272 pixels, two splits of 256 x 128 beat 392 unsplit
    // 128 x 64 tiles by a quarter)
    const long long tiles = (long long)(rows / 256) * cdivl(cols, 128);
    if (tiles >= 256 || !allow_split) return {256, 128, 1, ns, true};
    const long long small = (long long)(rows / 128) * cdivl(cols, 64);
    if (tiles < 64 && small >= 128) return {128, 64, 1, ns, true};
    int s = (int)std::min<long long>(256 / tiles, 16);
    s = std::max(1, std::min(s, std::max(1, ns / 4)));
    const int sps = cdiv(ns, s);
    return {256, 128, cdiv(ns, sps), sps, true};
  }
  struct Cand {
    int bm, bn, per_cu;
  };
  const Cand big[2] = {{128, 128, 2}, {128, 64, 3}};
  // 64-row GEMMs (64-channel convolutions): 64 x 128 tiles, three blocks per
  // CU, measured faster than 64 x 256 tiles two per CU at every size
  const Cand narrow[2] = {{64, 128, 3}, {64, 128, 3}};
  const Cand* c = rows <= 64 ? narrow : big;
  for (int i = 0; i < 2; ++i) {
    const long long tiles = (long long)cdiv(rows, c[i].bm) * cdivl(cols, c[i].bn);
    if (tiles >= 2LL * 256 * c[i].per_cu) return {c[i].bm, c[i].bn, 1, ns};
  }
  const long long tiles1 = (long long)cdiv(rows, c[1].bm) * cdivl(cols, c[1].bn);
  if (tiles1 >= 512 || !allow_split) return {c[1].bm, c[1].bn, 1, ns};
  const long long tiles0 = (long long)cdiv(rows, c[0].bm) * cdivl(cols, c[0].bn);
  int s = (int)std::min<long long>(cdivl(400, tiles0), std::max(1, ns / 4));
  s = std::max(1, std::min(s, 16));
  const int sps = cdiv(ns, s);
  return {c[0].bm, c[0].bn, cdiv(ns, sps), sps};
}

template <int BM, int BN, int WGM, template <int, int> class OpT>
hipError_t launch_dma(typename OpT<BM, BN>::Args a, long long cols, int rows, hipStream_t stream,
                      Cost cost, const char* name) {
  a.tiles_m = cdiv(rows, BM);
  a.tiles_n = (int)cdivl(cols, BN);
  dim3 grid(a.tiles_m * a.tiles_n * a.so.splits);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  // the BatchNorm-statistics variant exists for 128 x 128 tiles (64 pixels per wave)
  if constexpr (BM == 128 && BN == 128 && WGM == 2) {
    if (a.bn.part)
      hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, 2, OpT<BM, BN>, true>), grid, dim3(NT), 0,
                         stream, a);
    else
      hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, 2, OpT<BM, BN>>), grid, dim3(NT), 0, stream,
                         a);
  } else {
    if (a.bn.part) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, 2, OpT<BM, BN>>), grid, dim3(NT), 0, stream, a);
  }
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({std::string(name) + "<bf16," + std::to_string(BM) + "," +
                           std::to_string(BN) + ",dma>",
                       cost.flops, cost.bytes, e0, e1});
  }
  return e;
}

template <int BM, int BN, int WTM, int WTN, int NST, template <int, int> class OpT>
hipError_t launch_ws(typename OpT<BM, BN>::Args a, long long cols, int rows, hipStream_t stream,
                     Cost cost, const char* name) {
  a.tiles_m = cdiv(rows, BM);
  a.tiles_n = (int)cdivl(cols, BN);
  dim3 grid(a.tiles_m * a.tiles_n * a.so.splits);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  const dim3 block((BM / WTM) * (BN / WTN) * 64 + WS_LOADERS * 64);
  // the BatchNorm-statistics variant exists for 128 x 64 tiles (64 pixels per wave)
  if constexpr (BM == 128 && BN == 64 && WTN == 64) {
    if (a.bn.part)
      hipLaunchKernelGGL((gemm_ws_kernel<BM, BN, WTM, WTN, NST, OpT<BM, BN>, true>), grid, block,
                         0, stream, a);
    else
      hipLaunchKernelGGL((gemm_ws_kernel<BM, BN, WTM, WTN, NST, OpT<BM, BN>>), grid, block, 0,
                         stream, a);
  } else {
    if (a.bn.part) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_ws_kernel<BM, BN, WTM, WTN, NST, OpT<BM, BN>>), grid, block, 0,
                       stream, a);
  }
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({std::string(name) + "<bf16," + std::to_string(BM) + "," +
                           std::to_string(BN) + ",ws>",
                       cost.flops, cost.bytes, e0, e1});
  }
  return e;
}

template <template <int, int> class OpT, class Args>
hipError_t dispatch_dma(Args a, const DmaPlan& p, long long cols, int rows, hipStream_t stream,
                        Cost cost, const char* name) {
  if (p.bm == 256 && p.bn == 128)
    return launch_ws<256, 128, 64, 64, 3, OpT>(a, cols, rows, stream, cost, name);
  if (p.bm == 128 && p.bn == 64 && p.ws)
    return launch_ws<128, 64, 32, 64, 4, OpT>(a, cols, rows, stream, cost, name);
  if (p.bm == 128 && p.bn == 256 && p.ws)
    return launch_ws<128, 256, 64, 64, 3, OpT>(a, cols, rows, stream, cost, name);
  if (p.bm == 128 && p.bn == 128) return launch_dma<128, 128, 2, OpT>(a, cols, rows, stream, cost, name);
  if (p.bm == 128 && p.bn == 64) return launch_dma<128, 64, 2, OpT>(a, cols, rows, stream, cost, name);
  if (p.bm == 64 && p.bn == 256) return launch_dma<64, 256, 1, OpT>(a, cols, rows, stream, cost, name);
  if (p.bm == 64 && p.bn == 128) return launch_dma<64, 128, 1, OpT>(a, cols, rows, stream, cost, name);
  return hipErrorInvalidValue;
}

// Whether the kernel dispatch_dma runs for an unsplit plan has a variant that
// leaves BatchNorm chunk statistics (launch_ws / launch_dma).
bool plan_bn_epilogue(const DmaPlan& p) {
  return p.splits == 1 && p.bm == 128 && ((p.bn == 64 && p.ws) || (p.bn == 128 && !p.ws));
}

// Filter-resident path: 3x3, stride 1, pad 1, 64 -> 64 channels, bf16.
bool conv64_ok(const ConvGeom& g) {
  return g.C == 64 && g.K == 64 && g.R == 3 && g.S == 3 && g.stride == 1 && g.pad == 1 &&
         g.P == g.H && g.Q == g.W && g.N > 0 && g.H > 0 && g.W > 0 &&
         (long long)g.N * cdiv(g.H, 8) * cdiv(g.W, 8) < (1LL << 30);
}
Conv64Args plan_conv64(const ConvGeom& g) {
  Conv64Args a{};
  a.g = g;
  a.py_n = cdiv(g.H, 8);
  a.px_n = cdiv(g.W, 8);
  const long long np = (long long)g.N * a.py_n * a.px_n;
  a.pps = (int)cdivl(np, std::min<long long>(np, C64_TARGET_BLOCKS));
  return a;
}
int conv64_blocks(const Conv64Args& a) {
  return (int)cdivl((long long)a.g.N * a.py_n * a.px_n, a.pps);
}
// in: x (forward) or dy (data gradient); A: w [K][3][3][C] or wt [C][3][3][K].
hipError_t conv64(const ConvGeom& g, bool dgrad, const void* in, const void* A, void* out,
                  const ConvEpilogue& epi, hipStream_t stream) {
  Conv64Args a = plan_conv64(g);
  a.in = (const bf16*)in;
  a.a = (const bf16*)A;
  a.out = (bf16*)out;
  a.epi = epi;
  const Cost cost = conv_cost(g, 64, sizeof(bf16), false);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  const int blocks = conv64_blocks(a);
  if (dgrad)
    hipLaunchKernelGGL(conv64_kernel<true>, dim3(blocks), dim3(C64_NT), 0, stream, a);
  else
    hipLaunchKernelGGL(conv64_kernel<false>, dim3(blocks), dim3(C64_NT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({dgrad ? "conv_dgrad<bf16,c64>" : "conv_fwd<bf16,c64>", cost.flops,
                       cost.bytes, e0, e1});
  }
  return e;
}

// bf16 forward with C % 64 == 0 on the direct-to-LDS path.
hipError_t conv_fwd_dma(const ConvGeom& g, const void* x, const void* w, void* y,
                        const ConvEpilogue& epi, float* ws, size_t ws_floats, hipStream_t stream,
                        BnStatsSink* sink) {
  const int ns = g.R * g.S * g.C / 64;
  const long long npix = (long long)g.N * g.P * g.Q;
  if (conv64_ok(g) && !(sink && !sink->bwd && bn_fold_path(npix, g.K)))
    return conv64(g, false, x, w, y, epi, stream);
  DmaPlan p = plan_dma(g.K, npix, ns, ws != nullptr);
  if (p.splits > 1 && (size_t)p.splits * npix * g.K > ws_floats) p = {p.bm, p.bn, 1, ns, p.ws};
  DmaFwdArgs a{g, (const bf16*)x, (const bf16*)w, (bf16*)y, epi, SplitOut{ws, p.splits, p.sps}, 0, 0};
  const bool plain = !epi.scale && !epi.shift && !epi.res && !epi.relu;
  const bool bn_epi = sink && !sink->bwd && sink->part && plain && plan_bn_epilogue(p) &&
                      bn_fold_path(npix, g.K);
  if (bn_epi) a.bn.part = sink->part;
  hipError_t e = dispatch_dma<DmaFwdOp>(a, p, npix, g.K, stream,
                                       conv_cost(g, g.C0 ? g.C0 : g.C, sizeof(bf16), false),
                                       "conv_fwd");
  if (e == hipSuccess && bn_epi) {
    sink->done = true;
    sink->rows = 64;
  }
  if (e != hipSuccess || p.splits <= 1) return e;
  if (sink && !sink->bwd && plain && bn_fold_path(npix, g.K)) {
    sink->done = true;
    sink->rows = 128;
    return split_reduce_bn(DT_BF16, ws, p.splits, npix, g.K, nullptr, y, *sink, stream);
  }
  return split_finish<bf16>(ws, p.splits, npix, g.K, epi, y, stream);
}

// Stride-2 bf16 data gradient by parity class (DmaDgradS2Op): the GEMM plan
// is chosen for the average reduction length (a quarter of the taps); the
// split length covers the longest class.
// k2: channels of a folded shortcut (class (0, 0) only), 0 for none
DmaPlan plan_dgrad_s2(const ConvGeom& g, bool allow_split, int k2 = 0) {
  const int kc = g.K / 64;
  int ns_max = 0, ns_sum = 0;
  for (int c = 0; c < 4; ++c) {
    const S2Class k = s2_class(g, c);
    const int ns = k.nr * k.nsc * kc + (c == 0 ? k2 / 64 : 0);
    ns_max = std::max(ns_max, ns);
    ns_sum += ns;
  }
  const long long npix = (long long)g.N * g.H * g.W;
  DmaPlan p = plan_dma(g.C, npix, std::max(1, cdiv(ns_sum, 4)), allow_split);
  if (!allow_split) p.splits = 1;
  p.sps = std::max(1, cdiv(ns_max, p.splits));
  return p;
}

hipError_t conv_dgrad_s2(const ConvGeom& g, const void* dy, const void* wt, void* dx,
                         const void* res, float* ws, size_t ws_floats, hipStream_t stream,
                         const void* dy2 = nullptr, const void* wt2 = nullptr, int K2 = 0) {
  const long long npix = (long long)g.N * g.H * g.W;
  DmaPlan p = plan_dgrad_s2(g, ws != nullptr, K2);
  if (p.splits > 1 && (size_t)p.splits * npix * g.C > ws_floats) p = plan_dgrad_s2(g, false, K2);
  long long ctiles = 0;
  for (int c = 0; c < 4; ++c) {
    const S2Class k = s2_class(g, c);
    ctiles = std::max(ctiles, cdivl((long long)g.N * k.hc * k.wc, p.bn));
  }
  const long long cols = 4 * ctiles * p.bn;
  DmaDgradS2Args a{g, (const bf16*)dy, (const bf16*)wt, (bf16*)dx, (const bf16*)res,
                   SplitOut{ws, p.splits, p.sps}, 0, 0, BnEpi{}};
  Cost cost = conv_cost(g, g.C, sizeof(bf16), false);
  if (dy2) {
    a.dy2 = (const bf16*)dy2;
    a.wt2 = (const bf16*)wt2;
    a.K2 = K2;
    cost.flops += 2.0 * g.N * g.P * g.Q * (double)K2 * g.C;
    cost.bytes += ((double)g.N * g.P * g.Q * K2 + (double)K2 * g.C) * sizeof(bf16);
  }
  hipError_t e = dispatch_dma<DmaDgradS2Op>(a, p, cols, g.C, stream, cost,
                                           dy2 ? "conv_dgrad_s2+shortcut" : "conv_dgrad_s2");
  if (e != hipSuccess || p.splits <= 1) return e;
  ConvEpilogue ep;
  ep.res = res;
  return split_finish<bf16>(ws, p.splits, npix, g.C, ep, dx, stream);
}

// bf16 data gradient with K % 64 == 0 on the direct-to-LDS path.
hipError_t conv_dgrad_dma(const ConvGeom& g, const void* dy, const void* wt, void* dx,
                          const void* res, float* ws, size_t ws_floats, hipStream_t stream,
                          BnStatsSink* sink) {
  const int ns = g.R * g.S * g.K / 64;
  const long long npix = (long long)g.N * g.H * g.W;
  if (conv64_ok(g) && !(sink && sink->bwd && bn_fold_path(npix, g.C))) {
    ConvEpilogue ep;
    ep.res = res;
    return conv64(g, true, dy, wt, dx, ep, stream);
  }
  // (1x1 kernels: only one class has a tap and its reduction is too short to
  // amortise a tile's pipeline fill; the plain GEMM measured faster)
  if (g.stride == 2 && g.R * g.S > 1 && !(sink && sink->bwd && bn_fold_path(npix, g.C)))
    return conv_dgrad_s2(g, dy, wt, dx, res, ws, ws_floats, stream);
  DmaPlan p = plan_dma(g.C, npix, ns, ws != nullptr);
  if (p.splits > 1 && (size_t)p.splits * npix * g.C > ws_floats) p = {p.bm, p.bn, 1, ns, p.ws};
  DmaDgradArgs a{g, (const bf16*)dy, (const bf16*)wt, (bf16*)dx, (const bf16*)res,
                 SplitOut{ws, p.splits, p.sps}, 0, 0};
  const bool bn_epi = sink && sink->bwd && sink->part && sink->z && sink->mean &&
                      plan_bn_epilogue(p) && bn_fold_path(npix, g.C);
  if (bn_epi) {
    a.bn.part = sink->part;
    a.bn.ymask = (const bf16*)sink->ymask;
    a.bn.z = (const bf16*)sink->z;
    a.bn.mean = sink->mean;
    a.bn.bwd = 1;
  }
  hipError_t e = dispatch_dma<DmaDgradOp>(a, p, npix, g.C, stream,
                                         conv_cost(g, g.C, sizeof(bf16), false), "conv_dgrad");
  if (e == hipSuccess && bn_epi) {
    sink->done = true;
    sink->rows = 64;
  }
  if (e != hipSuccess || p.splits <= 1) return e;
  if (sink && sink->bwd && bn_fold_path(npix, g.C)) {
    sink->done = true;
    sink->rows = 128;
    return split_reduce_bn(DT_BF16, ws, p.splits, npix, g.C, res, dx, *sink, stream);
  }
  ConvEpilogue ep;
  ep.res = res;
  return split_finish<bf16>(ws, p.splits, npix, g.C, ep, dx, stream);
}

constexpr int KU_MAIN = 8;

template <typename T>
hipError_t conv_fwd_t(const ConvGeom& g, const void* x, const void* w, void* y,
                      const ConvEpilogue& epi, float* ws, size_t ws_floats, hipStream_t stream,
                      BnStatsSink* sink) {
  constexpr int E = Elt<T>::E;
  if (sizeof(T) == 2 && g.C % 64 == 0)
    return conv_fwd_dma(g, x, w, y, epi, ws, ws_floats, stream, sink);
  if (sizeof(T) == 2 && g.C == 8 && g.C0 == 3 && g.K == 64 && g.R == 7 && g.S == 7 && g.stride == 2 &&
      g.pad == 3 && g.Q <= STEM_QMAX && g.N > 0) {
    const Cost cost = conv_cost(g, 3, sizeof(bf16), false);
    KernelTimer* t = t_timer;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (t) {
      e0 = t->take();
      e1 = t->take();
      EKYA_HIP(hipEventRecord(e0, stream));
    }
    hipLaunchKernelGGL(stem_kernel<false>, dim3(g.N * cdiv(g.P, STEM_ROWS)), dim3(STEM_NT), 0,
                       stream, (const bf16*)x, (const int32_t*)nullptr, (const bf16*)w, (bf16*)y,
                       epi, g.N, g.H, g.W, g.P, g.Q);
    hipError_t e = hipGetLastError();
    if (t && e == hipSuccess) {
      EKYA_HIP(hipEventRecord(e1, stream));
      t->recs.push_back({"conv_fwd<bf16,stem7x7>", cost.flops, cost.bytes, e0, e1});
    }
    return e;
  }
  const bool ut = g.C % (KU_MAIN * E) == 0;
  const int ns = cdiv(g.R * g.S * g.C, KU_MAIN * E);
  const long long npix = (long long)g.N * g.P * g.Q;
  Plan p = plan_tiles(g.K, (int)npix, ns, ut && ws != nullptr);
  if (p.splits > 1 && (size_t)p.splits * npix * g.K > ws_floats) {
    p.splits = 1;
    p.sps = ns;
  }
  FwdArgs<T> a{g, (const T*)x, (const T*)w, (T*)y, epi, SplitOut{ws, p.splits, p.sps}};
  const Cost cost = conv_cost(g, g.C0 ? g.C0 : g.C, sizeof(T), false);
  hipError_t e;
  if (ut) {
    e = dispatch_tile<T, FwdPolicy, KU_MAIN, true>(a, p, g.K, (int)npix, stream, cost);
  } else {
    // image stem: C is one 16-byte unit; reduction elements decoded unit by unit
    const int ns4 = cdiv(g.R * g.S * g.C, 4 * E);
    a.so = SplitOut{nullptr, 1, ns4};
    if (npix / 128 >= kTargetBlocks)
      e = launch_gemm<T, FwdPolicy, 64, 128, 4, false>(a, g.K, (int)npix, 1, stream, cost);
    else
      e = launch_gemm<T, FwdPolicy, 64, 64, 4, false>(a, g.K, (int)npix, 1, stream, cost);
  }
  if (e != hipSuccess || p.splits <= 1 || !ut) return e;
  return split_finish<T>(ws, p.splits, npix, g.K, epi, y, stream);
}

template <typename T>
hipError_t conv_dgrad_t(const ConvGeom& g, const void* dy, const void* wt, void* dx,
                        const void* res, float* ws, size_t ws_floats, hipStream_t stream,
                        BnStatsSink* sink) {
  constexpr int E = Elt<T>::E;
  if (g.K % (KU_MAIN * E) != 0 || (g.stride != 1 && g.stride != 2)) return hipErrorInvalidValue;
  if (sizeof(T) == 2) return conv_dgrad_dma(g, dy, wt, dx, res, ws, ws_floats, stream, sink);
  const int ns = cdiv(g.R * g.S * g.K, KU_MAIN * E);
  const long long npix = (long long)g.N * g.H * g.W;
  Plan p = plan_tiles(g.C, (int)npix, ns, ws != nullptr);
  if (p.splits > 1 && (size_t)p.splits * npix * g.C > ws_floats) {
    p.splits = 1;
    p.sps = ns;
  }
  DgradArgs<T> a{g, (const T*)dy, (const T*)wt, (T*)dx, (const T*)res, SplitOut{ws, p.splits, p.sps}};
  hipError_t e = dispatch_tile<T, DgradPolicy, KU_MAIN, true>(a, p, g.C, (int)npix, stream,
                                                              conv_cost(g, g.C, sizeof(T), false));
  if (e != hipSuccess || p.splits <= 1) return e;
  ConvEpilogue ep;
  ep.res = res;
  return split_finish<T>(ws, p.splits, npix, g.C, ep, dx, stream);
}

int wgrad_stage_m(int dt) { return dt == DT_F32 ? 16 : 64; }

}  // namespace

hipEvent_t KernelTimer::take() {
  if (!pool.empty()) {
    hipEvent_t e = pool.back();
    pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  (void)hipEventCreateWithFlags(&e, hipEventDisableSystemFence);  // device-local timing only
  return e;
}
void set_thread_timer(KernelTimer* t) { t_timer = t; }
KernelTimer* thread_timer() { return t_timer; }

size_t conv_split_workspace_floats(int dt, const ConvGeom& g, bool dgrad) {
  const int E = dtype_vec(dt);
  if (dt == DT_BF16 && dgrad) {
    const long long npix = (long long)g.N * g.H * g.W;
    const DmaPlan p = g.stride == 2 && g.R * g.S > 1 ? plan_dgrad_s2(g, true)
                                                     : plan_dma(g.C, npix, g.R * g.S * g.K / 64, true);
    return p.splits > 1 ? (size_t)p.splits * npix * g.C : 0;
  }
  if (dt == DT_BF16 && g.C % 64 == 0) {
    const long long npix = (long long)g.N * g.P * g.Q;
    const DmaPlan p = plan_dma(g.K, npix, g.R * g.S * g.C / 64, true);
    return p.splits > 1 ? (size_t)p.splits * npix * g.K : 0;
  }
  if (dgrad) {
    const int ns = cdiv(g.R * g.S * g.K, KU_MAIN * E);
    const long long npix = (long long)g.N * g.H * g.W;
    const Plan p = plan_tiles(g.C, (int)npix, ns, true);
    return p.splits > 1 ? (size_t)p.splits * npix * g.C : 0;
  }
  if (g.C % (KU_MAIN * E) != 0) return 0;
  const int ns = cdiv(g.R * g.S * g.C, KU_MAIN * E);
  const long long npix = (long long)g.N * g.P * g.Q;
  const Plan p = plan_tiles(g.K, (int)npix, ns, true);
  return p.splits > 1 ? (size_t)p.splits * npix * g.K : 0;
}

namespace {
// Direct-to-LDS weight-gradient plan: 64 x 128 tiles (64 x 64 when K is not a
// multiple of 128), the pixel reduction split until ~576 blocks, keeping
// >= 2 stages of 64 pixels per split.
struct WgDmaPlan {
  int bm, bn, splits, mps;
  TapGeom tap;  // tap.splits > 0: the all-taps kernel (3x3, stride 1)
};
bool wgrad_dma_ok(int dt, const ConvGeom& g) { return dt == DT_BF16 && g.C % 64 == 0 && g.K % 64 == 0; }
// Blocks the all-taps weight gradient aims for: one per CU, or 96 when it
// runs beside the data-gradient chain on another stream (measured on the
// full-depth batch-128 step: 128 blocks 0.6% and 64 blocks 3% slower, 256
// slower still -- the chain on the critical path waits for the CUs and
// bandwidth the weight gradient holds, or for the weight gradient itself).
constexpr int TAP_TARGET_BLOCKS = 256;
constexpr int TAP_SHARED_BLOCKS = 96;
bool wgrad_tap_ok(const ConvGeom& g) {
  return g.R == 3 && g.S == 3 && g.stride == 1 && g.pad == 1 && g.P == g.H && g.Q == g.W &&
         g.C % 64 == 0 && g.K % 64 == 0 && (long long)g.N * g.H * g.W * g.C < (1LL << 40) &&
         (long long)g.N * g.P * g.Q * g.K < (1LL << 40);
}
TapGeom plan_wgrad_tap(const ConvGeom& g, bool shared) {
  TapGeom t;
  t.tiles_c = g.C / 64;
  t.tiles_k = g.K / 64;
  t.py_n = (g.P + 7) / 8;
  t.px_n = (g.Q + 7) / 8;
  const long long np = (long long)g.N * t.py_n * t.px_n;
  const long long tiles = (long long)t.tiles_c * t.tiles_k;
  long long s = std::max(1LL, std::min(np, cdivl(shared ? TAP_SHARED_BLOCKS : TAP_TARGET_BLOCKS, tiles)));
  t.pps = (int)cdivl(np, s);
  t.splits = (int)cdivl(np, t.pps);
  return t;
}
WgDmaPlan plan_wgrad_dma(const ConvGeom& g, bool shared = false) {
  if (wgrad_tap_ok(g)) {
    const TapGeom t = plan_wgrad_tap(g, shared);
    return {576, 64, t.splits, 0, t};
  }
  const long long M = (long long)g.N * g.P * g.Q;
  const long long stages = std::max(1LL, cdivl(M, 64));
  const long long ws_tiles = (long long)(g.R * g.S * g.C / 256) * (g.K / 128);
  if (g.C % 256 == 0 && g.K % 128 == 0 && ws_tiles >= 16 && stages >= 128 &&
      (long long)g.N * g.H * g.W * g.C < (1LL << 31) && M * g.K < (1LL << 31)) {
    // warp-specialised 256 x 128 tiles, one block per CU, for long pixel
    // reductions (shorter ones run faster as the smaller blocks below, which
    // also share CUs with the data-gradient chain): about one block per CU in
    // total, >= 4 stages per split
    long long s = std::min(std::max(1LL, 256 / ws_tiles), std::max(1LL, stages / 4));
    s = std::min(s, 64LL);
    const long long mps = cdivl(cdivl(M, s), 64) * 64;
    return {256, 128, (int)cdivl(M, mps), (int)mps, TapGeom{}};
  }
  const int bn = g.K % 128 == 0 ? 128 : 64;
  const long long tiles = (long long)(g.R * g.S * g.C / 64) * (g.K / bn);
  long long s = std::min(cdivl(576, tiles), std::max(1LL, stages / 2));
  s = std::max(1LL, std::min(s, 64LL));
  const long long mps = cdivl(cdivl(M, s), 64) * 64;
  return {64, bn, (int)cdivl(M, mps), (int)mps, TapGeom{}};
}
struct WPlan {
  int bm, bn, splits;
};

// dw == nullptr: leave the split partials (one split included) in `partials`.
hipError_t conv_wgrad_dma(const ConvGeom& g, const void* x, const void* dy, float* partials,
                          float* dw, hipStream_t stream, bool shared = false) {
  const WgDmaPlan p = plan_wgrad_dma(g, shared);
  float* out = (p.splits > 1 || !dw) ? partials : dw;
  WgDmaArgs a{g, (const bf16*)x, (const bf16*)dy, out, p.mps, 0, 0, p.splits};
  a.tiles_m = g.R * g.S * g.C / p.bm;
  a.tiles_n = g.K / p.bn;
  const Cost cost = conv_cost(g, g.C, sizeof(bf16), true);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  const dim3 grid(a.tiles_m * a.tiles_n, p.splits);
  if (p.tap.splits > 0) {
    const WgTapArgs ta{g, p.tap, (const bf16*)x, (const bf16*)dy, out};
    hipLaunchKernelGGL(wgrad_tapw_kernel, dim3(p.tap.tiles_c * p.tap.tiles_k * p.tap.splits),
                       dim3(TAPW_NT), 0, stream, ta);
  } else if (p.bm == 256)
    hipLaunchKernelGGL((wgrad_ws_kernel<256, 128, 3>), dim3(a.tiles_m * a.tiles_n * p.splits),
                       dim3(8 * 64 + WS_LOADERS * 64), 0, stream, a);
  else if (p.bn == 128)
    hipLaunchKernelGGL((wgrad_dma_kernel<64, 128>), grid, dim3(NT), 0, stream, a);
  else
    hipLaunchKernelGGL((wgrad_dma_kernel<64, 64>), grid, dim3(NT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({p.tap.splits > 0 ? std::string("conv_wgrad<bf16,taps9,64>")
                                         : std::string("conv_wgrad<bf16,") + std::to_string(p.bm) +
                                               "," + std::to_string(p.bn) +
                                               (p.bm == 256 ? ",ws>" : ",dma>"),
                       cost.flops, cost.bytes, e0, e1});
  }
  if (e != hipSuccess || p.splits == 1 || !dw) return e;
  const long long n = (long long)g.K * g.R * g.S * g.C;
  const int blocks = (int)std::min<long long>(cdivl(n, 256), 4096);
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(blocks), dim3(256), 0, stream, partials, p.splits,
                     g.K, g.R * g.S, g.C, g.C, dw);
  return hipGetLastError();
}
WPlan plan_wgrad(int dt, const ConvGeom& g) {
  // 128-row tiles, split the pixel reduction until there are ~1024 blocks
  // (>= 4 stages per split): measured faster than fewer, longer blocks.
  const long long M = (long long)g.N * g.P * g.Q;
  const int rows = g.R * g.S * g.C;
  const int bn = g.K >= 128 ? 128 : 64;
  const long long tiles = (long long)cdiv(rows, 128) * cdiv(g.K, bn);
  const long long by_work = std::max(1LL, cdivl(M, 4LL * wgrad_stage_m(dt)));
  const long long s = std::max(1LL, std::min<long long>(std::min(cdivl(1024, tiles), by_work), 1024));
  return {128, bn, (int)s};
}
}  // namespace

int conv_wgrad_splits(int dt, const ConvGeom& g) {
  return wgrad_dma_ok(dt, g) ? plan_wgrad_dma(g).splits : plan_wgrad(dt, g).splits;
}

bool conv_wgrad_partials_ok(int dt, const ConvGeom& g) {
  return wgrad_dma_ok(dt, g) && (g.C0 == 0 || g.C0 == g.C);
}

size_t conv_wgrad_partials_floats(int dt, const ConvGeom& g) {
  if (!conv_wgrad_partials_ok(dt, g)) return 0;
  const int s = plan_wgrad_dma(g).splits;
  return (size_t)(s + conv_update_groups(s)) * g.K * g.R * g.S * g.C;
}

hipError_t conv_wgrad_partials(int dt, const ConvGeom& g, const void* x, const void* dy,
                               float* partials, int* splits, hipStream_t stream, bool shared) {
  if (!conv_wgrad_partials_ok(dt, g) || !partials) return hipErrorInvalidValue;
  *splits = plan_wgrad_dma(g, shared).splits;
  return conv_wgrad_dma(g, x, dy, partials, nullptr, stream, shared);
}

namespace {
bool stem_wgrad_ok(int dt, const ConvGeom& g, int C0) {
  return dt == DT_BF16 && g.C == 8 && C0 == 3 && g.K == 64 && g.R == 7 && g.S == 7 &&
         g.stride == 2 && g.pad == 3 && g.P == (g.H - 1) / 2 + 1 && g.Q == (g.W - 1) / 2 + 1 &&
         g.P >= 1 && g.Q >= 1 && (long long)g.N * g.H * g.W * 8 < (1LL << 40);
}
// two blocks per CU: with the pooled BatchNorm backward folded in, one
// block's gradient arithmetic overlaps the other's MFMAs
constexpr int STEM_WG_BLOCKS = 512;
StemWgArgs plan_stem_wgrad(const ConvGeom& g) {
  StemWgArgs a{};
  a.g = g;
  a.py_n = (g.P + 7) / 8;
  a.px_n = (g.Q + 7) / 8;
  const long long np = (long long)g.N * a.py_n * a.px_n;
  a.pps = (int)cdivl(np, std::min<long long>(np, STEM_WG_BLOCKS));
  a.splits = (int)cdivl(np, a.pps);
  return a;
}
// stem partials [splits][64][49][4], then their group sums
size_t stem_wgrad_floats(const ConvGeom& g) {
  const int s = plan_stem_wgrad(g).splits;
  return (size_t)(s + conv_update_groups(s)) * 64 * 49 * 4;
}
hipError_t stem_wgrad(const ConvGeom& g, const void* x, const void* dy, float* partials, float* dw,
                      hipStream_t stream, const StemPoolBwd* pb = nullptr) {
  StemWgArgs a = plan_stem_wgrad(g);
  if (pb) a.pb = *pb;
  a.x = (const bf16*)x;
  a.dy = (const bf16*)dy;
  a.out = partials;
  const Cost cost = conv_cost(g, 3, sizeof(bf16), true);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  if (pb)
    hipLaunchKernelGGL(wgrad_stem_kernel<true>, dim3(a.splits), dim3(NT), 0, stream, a);
  else
    hipLaunchKernelGGL(wgrad_stem_kernel<false>, dim3(a.splits), dim3(NT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({pb ? "conv_wgrad<bf16,stem+pool_bwd>" : "conv_wgrad<bf16,stem>", cost.flops,
                       cost.bytes, e0, e1});
  }
  EKYA_HIP(e);
  const long long n = 64LL * 49 * 4;
  const float* sums = partials;
  int splits = a.splits;
  if (conv_update_groups(splits) > 0) {
    float* gs = partials + (long long)splits * n;
    EKYA_HIP(split_group_sum(partials, splits, n, gs, stream));
    sums = gs;
    splits = conv_update_groups(splits);
  }
  const long long nw = 64LL * 49 * 3;
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3((int)cdivl(nw, 256)), dim3(256), 0, stream, sums,
                     splits, 64, 49, 4, 3, dw);
  return hipGetLastError();
}
}  // namespace

size_t conv_wgrad_workspace_floats(int dt, const ConvGeom& g) {
  if (stem_wgrad_ok(dt, g, g.C0 ? g.C0 : g.C)) return stem_wgrad_floats(g);
  if (wgrad_dma_ok(dt, g)) {
    const WgDmaPlan q = plan_wgrad_dma(g);
    return q.splits > 1 ? (size_t)q.splits * g.K * g.R * g.S * g.C : 0;
  }
  const WPlan p = plan_wgrad(dt, g);
  return (size_t)p.splits * g.K * g.R * g.S * g.C;
}

bool stem_pool_ok(int dt, const ConvGeom& g) {
  return dt == DT_BF16 && g.C == 8 && (g.C0 == 0 || g.C0 == 3) && g.K == 64 && g.R == 7 &&
         g.S == 7 && g.stride == 2 && g.pad == 3 && g.Q <= STEM_QMAX && g.Q >= 1 && g.P >= 1;
}

hipError_t stem_pool_fwd(int dt, const ConvGeom& g, const void* x, bool raw, const int32_t* idx,
                         const void* w, void* y, const ConvEpilogue& epi, hipStream_t stream) {
  if (!stem_pool_ok(dt, g)) return hipErrorInvalidValue;
  if (g.N == 0) return hipSuccess;
  const int PP = (g.P - 1) / 2 + 1;
  const Cost cost = conv_cost(g, 3, sizeof(bf16), false);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  const dim3 grid(g.N * cdiv(PP, 4)), block(STEM_NT + 64);
  if (raw)
    hipLaunchKernelGGL((stem_kernel<true, true>), grid, block, 0, stream, (const bf16*)x, idx,
                       (const bf16*)w, (bf16*)y, epi, g.N, g.H, g.W, g.P, g.Q);
  else
    hipLaunchKernelGGL((stem_kernel<false, true>), grid, block, 0, stream, (const bf16*)x,
                       (const int32_t*)nullptr, (const bf16*)w, (bf16*)y, epi, g.N, g.H, g.W,
                       g.P, g.Q);
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({raw ? "conv_fwd<bf16,stem7x7+pool,frames>" : "conv_fwd<bf16,stem7x7+pool>",
                       cost.flops, cost.bytes, e0, e1});
  }
  return e;
}

bool stem_frames_ok(int dt, const ConvGeom& g) {
  return dt == DT_BF16 && g.C == 8 && (g.C0 == 0 || g.C0 == 3) && g.K == 64 && g.R == 7 &&
         g.S == 7 && g.stride == 2 && g.pad == 3 && g.Q <= STEM_QMAX && g.Q >= 1;
}

hipError_t stem_fwd_frames(int dt, const ConvGeom& g, const void* frames, const int32_t* idx,
                           const void* w, void* y, const ConvEpilogue& epi, hipStream_t stream) {
  if (!stem_frames_ok(dt, g)) return hipErrorInvalidValue;
  if (g.N == 0) return hipSuccess;
  const Cost cost = conv_cost(g, 3, sizeof(bf16), false);
  KernelTimer* t = t_timer;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t) {
    e0 = t->take();
    e1 = t->take();
    EKYA_HIP(hipEventRecord(e0, stream));
  }
  hipLaunchKernelGGL(stem_kernel<true>, dim3(g.N * cdiv(g.P, STEM_ROWS)), dim3(STEM_NT), 0, stream,
                     (const bf16*)frames, idx, (const bf16*)w, (bf16*)y, epi, g.N, g.H, g.W, g.P,
                     g.Q);
  hipError_t e = hipGetLastError();
  if (t && e == hipSuccess) {
    EKYA_HIP(hipEventRecord(e1, stream));
    t->recs.push_back({"conv_fwd<bf16,stem7x7,frames>", cost.flops, cost.bytes, e0, e1});
  }
  return e;
}

hipError_t conv_fwd(int dt, const ConvGeom& g, const void* x, const void* w, void* y,
                    const ConvEpilogue& epi, float* ws, size_t ws_floats, hipStream_t stream,
                    BnStatsSink* sink) {
  if (sink) sink->done = false;
  if (g.N * g.P * g.Q == 0) return hipSuccess;
  return dt == DT_F32 ? conv_fwd_t<float>(g, x, w, y, epi, ws, ws_floats, stream, sink)
                      : conv_fwd_t<bf16>(g, x, w, y, epi, ws, ws_floats, stream, sink);
}

bool conv_dgrad_s2_shortcut_ok(int dt, const ConvGeom& g, const ConvGeom& gs) {
  return dt == DT_BF16 && g.stride == 2 && g.R == 3 && g.S == 3 && g.pad == 1 &&
         g.K % 64 == 0 && g.C % 64 == 0 && gs.stride == 2 && gs.R == 1 && gs.S == 1 &&
         gs.pad == 0 && gs.K % 64 == 0 && gs.N == g.N && gs.H == g.H && gs.W == g.W &&
         gs.C == g.C && gs.P == g.P && gs.Q == g.Q;
}

hipError_t conv_dgrad_s2_shortcut(const ConvGeom& g, const void* dy, const void* wt,
                                  const ConvGeom& gs, const void* dy_sc, const void* wt_sc,
                                  void* dx, float* ws, size_t ws_floats, hipStream_t stream) {
  if (!conv_dgrad_s2_shortcut_ok(DT_BF16, g, gs) || !dy_sc || !wt_sc) return hipErrorInvalidValue;
  if (g.N * g.H * g.W == 0) return hipSuccess;
  return conv_dgrad_s2(g, dy, wt, dx, nullptr, ws, ws_floats, stream, dy_sc, wt_sc, gs.K);
}

hipError_t conv_dgrad(int dt, const ConvGeom& g, const void* dy, const void* wt, void* dx,
                      const void* res, float* ws, size_t ws_floats, hipStream_t stream,
                      BnStatsSink* sink) {
  if (sink) sink->done = false;
  if (g.N * g.H * g.W == 0) return hipSuccess;
  return dt == DT_F32 ? conv_dgrad_t<float>(g, dy, wt, dx, res, ws, ws_floats, stream, sink)
                      : conv_dgrad_t<bf16>(g, dy, wt, dx, res, ws, ws_floats, stream, sink);
}


bool stem_wgrad_pool_ok(int dt, const ConvGeom& g) { return stem_wgrad_ok(dt, g, 3); }

hipError_t conv_wgrad_stem_pool(const ConvGeom& g, const void* x, const void* z,
                                const void* dy_pool, const uint8_t* arg, const float* mean,
                                const float* coef, const float* gamma, const float* invstd,
                                const float* beta, float* partials, float* dw, hipStream_t stream) {
  if (!stem_wgrad_pool_ok(DT_BF16, g)) return hipErrorInvalidValue;
  if (g.N == 0) return hipSuccess;
  StemPoolBwd pb{(const bf16*)z, (const bf16*)dy_pool, arg, mean, coef, gamma, invstd, beta,
                 (g.P - 1) / 2 + 1, (g.Q - 1) / 2 + 1};
  return stem_wgrad(g, x, nullptr, partials, dw, stream, &pb);
}

hipError_t conv_wgrad(int dt, const ConvGeom& g, const void* x, const void* dy, float* partials,
                      float* dw, int C0, hipStream_t stream) {
  if (stem_wgrad_ok(dt, g, C0)) return stem_wgrad(g, x, dy, partials, dw, stream);
  if (wgrad_dma_ok(dt, g) && C0 == g.C) return conv_wgrad_dma(g, x, dy, partials, dw, stream);
  const WPlan p = plan_wgrad(dt, g);
  const long long M = (long long)g.N * g.P * g.Q;
  const int stage = wgrad_stage_m(dt);
  const int mps = (int)(cdivl(cdivl(M, p.splits), stage) * stage);
  const int rows = g.R * g.S * g.C;
  const Cost cost = conv_cost(g, C0, dtype_size(dt), true);
  // one split over unpadded channels: the tile writes dw directly
  const bool direct = p.splits == 1 && C0 == g.C;
  float* out = direct ? dw : partials;
  hipError_t e;
#define EKYA_WG(T_, KU_, BM_, BN_)                                                              \
  if (p.bm == BM_ && p.bn == BN_) {                                                            \
    WgradArgs<T_> a{g, (const T_*)x, (const T_*)dy, out, mps};                                 \
    e = launch_gemm<T_, WgradPolicy, BM_, BN_, KU_, true>(a, rows, g.K, p.splits, stream, cost); \
  }
  if (dt == DT_F32) {
    EKYA_WG(float, 4, 128, 128) else EKYA_WG(float, 4, 128, 64) else EKYA_WG(float, 4, 64, 64) else return hipErrorInvalidValue;
  } else {
    EKYA_WG(bf16, 8, 128, 128) else EKYA_WG(bf16, 8, 128, 64) else EKYA_WG(bf16, 8, 64, 64) else return hipErrorInvalidValue;
  }
#undef EKYA_WG
  if (e != hipSuccess || direct) return e;
  const long long n = (long long)g.K * g.R * g.S * C0;
  const int blocks = (int)std::min<long long>(cdivl(n, 256), 4096);
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(blocks), dim3(256), 0, stream, partials, p.splits,
                     g.K, g.R * g.S, g.C, C0, dw);
  return hipGetLastError();
}

}  // namespace ekya
