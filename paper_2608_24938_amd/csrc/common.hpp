// Device helpers shared by the libexfold kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "exfold.h"

namespace exfold {

constexpr int kWave = 64;
constexpr int kMaxExperts = 256;
constexpr int kMaxTopK = 16;
constexpr int kFixedPointBits = 40;  // decode pool weight sums: rint(w * 2^40)

typedef uint16_t bf16_t;  // raw bf16 storage
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
// 16-byte staging register (a native vector: HIP's uint4 is a union-based
// struct that the optimiser cannot keep in registers when held in arrays)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Round-to-nearest-even float32 -> bf16 (NaN kept quiet).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

template <typename T> __device__ __forceinline__ float load_f32(const T *p);
template <> __device__ __forceinline__ float load_f32<float>(const float *p) { return *p; }
template <> __device__ __forceinline__ float load_f32<bf16_t>(const bf16_t *p) { return bf16_to_f32(*p); }

template <typename T> __device__ __forceinline__ T store_cvt(float v);
template <> __device__ __forceinline__ float store_cvt<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t store_cvt<bf16_t>(float v) { return f32_to_bf16(v); }

// Order-preserving map float -> uint32 (larger float -> larger key); -0 == +0.
__device__ __forceinline__ uint32_t float_key(float v) {
  if (v == 0.0f) v = 0.0f;
  uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int clamp_id(int e, int n) { return e < 0 ? 0 : (e >= n ? n - 1 : e); }

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  uint32_t lo = __shfl_xor((unsigned)(v & 0xffffffffu), mask, kWave);
  uint32_t hi = __shfl_xor((unsigned)(v >> 32), mask, kWave);
  return (uint64_t(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    uint64_t o = shfl_xor_u64(v, m);
    v = o > v ? o : v;
  }
  return v;
}

__device__ __forceinline__ double shfl_f64(double v, int src) {
  int64_t b = __double_as_longlong(v);
  int lo = __shfl((int)(b & 0xffffffff), src, kWave);
  int hi = __shfl((int)(b >> 32), src, kWave);
  return __longlong_as_double((int64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return (lane == 0) ? 0ull : (~0ull >> (64 - lane)); }

// XCD-aware remap of a workgroup id: the hardware deals consecutive workgroup
// ids round-robin over the 8 XCDs; this returns a logical id such that every
// XCD works on one contiguous range of logical ids (tiles that share operands
// then share that XCD's L2).
__device__ __forceinline__ int xcd_remap(int wg, int n_wg) {
  constexpr int kXcd = 8;
  const int q = n_wg / kXcd, r = n_wg % kXcd;
  const int xcd = wg % kXcd, local = wg / kXcd;
  return (xcd < r) ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

}  // namespace exfold
