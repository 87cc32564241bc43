// Device helpers shared by the libexfold kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <type_traits>
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

// Round-to-nearest-even float32 -> bf16 (the hardware conversion,
// v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

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

// Cross-lane helpers built on DPP (in-register, within rows of 16 lanes) and
// readlane (whole wave, uniform lane index) instead of LDS permutes, whose
// latency chains dominated the one-wave reductions.  All take full waves.
// DPP controls: quad_perm [1,0,3,2] and [2,3,0,1], row_half_mirror, row_mirror.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v, uint32_t old) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v, uint64_t old) {
  const uint32_t lo = dpp_u32<CTRL>((uint32_t)v, (uint32_t)old);
  const uint32_t hi = dpp_u32<CTRL>((uint32_t)(v >> 32), (uint32_t)(old >> 32));
  return (uint64_t(hi) << 32) | lo;
}
__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  return (uint64_t(readlane_u32((uint32_t)(v >> 32), lane)) << 32) | readlane_u32((uint32_t)v, lane);
}
__device__ __forceinline__ double readlane_f64(double v, int lane) {
  return __longlong_as_double((long long)readlane_u64((uint64_t)__double_as_longlong(v), lane));
}
__device__ __forceinline__ float readlane_f32(float v, int lane) {
  return __uint_as_float(readlane_u32(__float_as_uint(v), lane));
}

// Max (MAX) or min of a 64-bit key over the wave; every lane gets the result.
template <bool MAX>
__device__ __forceinline__ uint64_t wave_reduce_u64(uint64_t v) {
  auto pick = [](uint64_t a, uint64_t b) { return MAX ? (a > b ? a : b) : (a < b ? a : b); };
  v = pick(v, dpp_u64<0xB1>(v, v));
  v = pick(v, dpp_u64<0x4E>(v, v));
  v = pick(v, dpp_u64<0x141>(v, v));
  v = pick(v, dpp_u64<0x140>(v, v));
  return pick(pick(readlane_u64(v, 0), readlane_u64(v, 16)), pick(readlane_u64(v, 32), readlane_u64(v, 48)));
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) { return wave_reduce_u64<true>(v); }
// Max of a 32-bit value over the wave; every lane gets the result.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, dpp_u32<0xB1>(v, v));
  v = max(v, dpp_u32<0x4E>(v, v));
  v = max(v, dpp_u32<0x141>(v, v));
  v = max(v, dpp_u32<0x140>(v, v));
  return max(max(readlane_u32(v, 0), readlane_u32(v, 16)), max(readlane_u32(v, 32), readlane_u32(v, 48)));
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) { return wave_reduce_u64<false>(v); }

// Sum over the wave in a fixed association (pairs within quads, half-rows,
// rows, then the four rows in order); every lane gets the same value.
__device__ __forceinline__ double wave_sum_f64(double v) {
  auto step = [](double x, auto ctrl) {
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    return x + __longlong_as_double((long long)dpp_u64<decltype(ctrl)::value>(b, 0ull));
  };
  v = step(v, std::integral_constant<int, 0xB1>{});
  v = step(v, std::integral_constant<int, 0x4E>{});
  v = step(v, std::integral_constant<int, 0x141>{});
  v = step(v, std::integral_constant<int, 0x140>{});
  return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

// Sum of a float over the wave in the association of wave_sum_f64.
__device__ __forceinline__ float wave_sum_f32(float v) {
  v += __uint_as_float(dpp_u32<0xB1>(__float_as_uint(v), 0u));
  v += __uint_as_float(dpp_u32<0x4E>(__float_as_uint(v), 0u));
  v += __uint_as_float(dpp_u32<0x141>(__float_as_uint(v), 0u));
  v += __uint_as_float(dpp_u32<0x140>(__float_as_uint(v), 0u));
  return (readlane_f32(v, 0) + readlane_f32(v, 16)) + (readlane_f32(v, 32) + readlane_f32(v, 48));
}

// Workgroup barrier that orders LDS accesses only: global stores issued before
// it are not waited for.  For kernels whose threads exchange data through LDS
// alone and whose global outputs are read only after the kernel.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return (lane == 0) ? 0ull : (~0ull >> (64 - lane)); }

// Exclusive prefix sums of three per-thread counts over the first kW waves of
// the workgroup, thread i holding element i of each sequence: a scan inside
// each wave, then the wave totals through LDS (`part`, 3 * kW ints).  Every
// thread of the workgroup calls it (it holds one LDS barrier).  Threads of the
// first kW waves get their exclusive prefixes in ex; every thread gets the
// totals in tot.
template <int kW>
__device__ __forceinline__ void block_scan3(const int (&v)[3], int (&ex)[3], int (&tot)[3], int *part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int in[3] = {v[0], v[1], v[2]};
  if (wave < kW) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      int x[3];
#pragma unroll
      for (int q = 0; q < 3; ++q) x[q] = __shfl_up(in[q], off, 64);
      if (lane >= off) {
#pragma unroll
        for (int q = 0; q < 3; ++q) in[q] += x[q];
      }
    }
    if (lane == 63) {
#pragma unroll
      for (int q = 0; q < 3; ++q) part[q * kW + wave] = in[q];
    }
  }
  lds_barrier();
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    int pre = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kW; ++w) {
      const int sw = part[q * kW + w];
      pre += (w < wave) ? sw : 0;
      all += sw;
    }
    ex[q] = pre + in[q] - v[q];
    tot[q] = all;
  }
}

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
