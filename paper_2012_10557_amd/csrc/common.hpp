// Shared device/host helpers of the HIP library: element types, 16-byte units,
// MFMA wrappers for gfx950, and error plumbing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace ekya {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Element traits: E elements fill one 16-byte unit.
template <typename T> struct Elt;
template <> struct Elt<float> {
  static constexpr int E = 4;
};
template <> struct Elt<bf16> {
  static constexpr int E = 8;
};

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return (bf16)v; }  // RNE

// A 16-byte unit viewed as E elements.
template <typename T> union Unit {
  uint4 u;
  T e[Elt<T>::E];
};

__device__ __forceinline__ uint4 zero_unit() { return make_uint4(0u, 0u, 0u, 0u); }

// max(v, 0) that keeps a NaN input NaN (fmaxf would return 0), so that a
// non-finite input reaches the loss and is reported.
__device__ __forceinline__ float relu_nan(float v) { return v < 0.f ? 0.f : v; }

// Four consecutive elements as float (8- or 16-byte accesses).
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


// D += A * B on one 16x16 output tile; `a` and `b` are one 16-byte unit each
// (k-contiguous).  For bf16 the unit is the whole k-chunk of one
// v_mfma_f32_16x16x32_bf16; for fp32 the four floats feed four
// v_mfma_f32_16x16x4_f32 steps (any k-to-slot assignment is valid as long as
// A and B share it).
__device__ __forceinline__ void mma_unit(f32x4& acc, uint4 a, uint4 b, bf16*) {
  bf16x8 av = __builtin_bit_cast(bf16x8, a);
  bf16x8 bv = __builtin_bit_cast(bf16x8, b);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma_unit(f32x4& acc, uint4 a, uint4 b, float*) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// Transpose an E x E block held as E units (unit i = row i) into E units
// (unit j = column j).
__device__ __forceinline__ void transpose_block(uint4 (&v)[4], float*) {
  float m[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i][0] = __uint_as_float(v[i].x);
    m[i][1] = __uint_as_float(v[i].y);
    m[i][2] = __uint_as_float(v[i].z);
    m[i][3] = __uint_as_float(v[i].w);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j)
    v[j] = make_uint4(__float_as_uint(m[0][j]), __float_as_uint(m[1][j]), __float_as_uint(m[2][j]),
                      __float_as_uint(m[3][j]));
}

__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) {  // (lo16(a), lo16(b))
  return (a & 0xFFFFu) | (b << 16);
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) {  // (hi16(a), hi16(b))
  return (a >> 16) | (b & 0xFFFF0000u);
}

__device__ __forceinline__ void transpose_block(uint4 (&v)[8], bf16*) {
  // v[i] holds row i: dword d = (x[i][2d], x[i][2d+1]).
  // out[j] dword e = (x[2e][j], x[2e+1][j]).
  uint32_t r[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    r[i][0] = v[i].x;
    r[i][1] = v[i].y;
    r[i][2] = v[i].z;
    r[i][3] = v[i].w;
  }
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    uint32_t lo[4], hi[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] = pack_lo(r[2 * e][d], r[2 * e + 1][d]);
      hi[e] = pack_hi(r[2 * e][d], r[2 * e + 1][d]);
    }
    v[2 * d] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    v[2 * d + 1] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  }
}

__host__ __device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }
__host__ __device__ __forceinline__ long long cdivl(long long a, long long b) { return (a + b - 1) / b; }

}  // namespace ekya

// Host-side HIP error propagation: returns a hipError_t from the enclosing function.
#define EKYA_HIP(expr)                     \
  do {                                     \
    hipError_t e_ = (expr);                \
    if (e_ != hipSuccess) return e_;       \
  } while (0)
