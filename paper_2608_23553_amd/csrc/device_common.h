// device_common.h - small device helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace chimera {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;

// 2^22: one unit of an inner product of two grid vectors is 2^-22.
#define KEY_SCALE 4194304.0f

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Value grid: nearest multiple of max(2^-11, bf16 spacing), ties to even.
__device__ __forceinline__ uint16_t grid_bf16_bits(float x) {
  if (fabsf(x) < 0.0625f) {
    float g = rintf(x * 2048.0f) * (1.0f / 2048.0f);  // exact: |g| <= 2^-4, <= 8 significant bits
    return (uint16_t)(__float_as_uint(g) >> 16);
  }
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Order-preserving 64-bit key of (score desc, id asc): larger is better.
__device__ __forceinline__ uint64_t pack_key(int32_t score_key, uint32_t id) {
  return ((uint64_t)((uint32_t)score_key ^ 0x80000000u) << 32) | (uint64_t)(0xFFFFFFFFu - id);
}
__device__ __forceinline__ int32_t key_score(uint64_t k) { return (int32_t)((uint32_t)(k >> 32) ^ 0x80000000u); }
__device__ __forceinline__ uint32_t key_id(uint64_t k) { return 0xFFFFFFFFu - (uint32_t)k; }

// Exact conversion of a grid inner product (fp32, a multiple of 2^-22 below
// 2^2 in magnitude) to its integer key.
__device__ __forceinline__ int32_t to_key(float s) { return (int32_t)(s * KEY_SCALE); }

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

// F' of a document outside the candidate set S_Q (a real F' is never this small).
constexpr int NO_HIT = (int)0x80000000;
// Bins of the first radix pass of the refinement select (top 12 key bits).
constexpr int SEL_BINS = 4096;

// Unsigned order key of a partial score: larger F' <-> larger key.
__device__ __forceinline__ uint32_t fp_key(int32_t f) { return (uint32_t)f ^ 0x80000000u; }

// First position p in [lo, hi) of the ascending array a with a[p] >= x.
__device__ __forceinline__ int64_t lower_bound_i32(const int32_t *__restrict__ a, int64_t lo, int64_t hi, int64_t x) {
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if ((int64_t)a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

template <class T>
__device__ __forceinline__ T shfl_xor(T v, int m) {
  return __shfl_xor(v, m, 64);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = __shfl_xor(lo, m, 64);
  hi = __shfl_xor(hi, m, 64);
  return ((uint64_t)hi << 32) | lo;
}

}  // namespace chimera
