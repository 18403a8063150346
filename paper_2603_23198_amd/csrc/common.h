// Shared device/host helpers of libsfl (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sfl.h"

namespace sfl {

constexpr int kWave = 64;

typedef uint16_t bf16_t;  // raw bf16 bits
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// ---- bf16 conversions ------------------------------------------------------
// float32 -> bf16 with round-to-nearest-even on the bit pattern; subnormals are
// rounded like normals (no flush), overflow goes to infinity, NaN stays a quiet NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  uint32_t r = u + 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(r >> 16);
}
// The same rounding for a value known not to be NaN (no NaN test).
__device__ __forceinline__ bf16_t f32_to_bf16_finite(float x) {
  const uint32_t u = __float_as_uint(x);
  return (bf16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Value-type traits: element storage for the two activation dtypes.
template <typename V> struct VT;
template <> struct VT<float> {
  static __device__ __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
  static __device__ __forceinline__ float cvt(float v) { return v; }
};
template <> struct VT<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
  static __device__ __forceinline__ void store(bf16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }
  static __device__ __forceinline__ bf16_t cvt(float v) { return f32_to_bf16(v); }
};

// ---- wave primitives ---------------------------------------------------------
__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0)); }
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
// number of set bits of m in lanes below this one
__device__ __forceinline__ int mbcnt(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}
__device__ __forceinline__ int readlane_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ float readlane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

template <typename T> __device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum of a[i] for i = first, first + step, ... below n, in that order, eight loads in
// flight at a time (a load past the end re-reads a[n - 1] and zero is added in its place).
__device__ __forceinline__ float strided_sum(const float* __restrict__ a, int n, int first, int step) {
  float s = 0.f;
  for (int i0 = first; i0 < n; i0 += 8 * step) {
    float q[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) q[u] = a[min(i0 + u * step, n - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += i0 + u * step < n ? q[u] : 0.f;
  }
  return s;
}

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int u = __shfl_up(v, o, 64);
    if (l >= o) v += u;
  }
  return v;
}

__host__ __device__ constexpr int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace sfl
