// Device-side helpers shared by the HIP kernels of libcoinf.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "schedule.hpp"

namespace coinf {

using bf16_t = uint16_t;  // bfloat16 bits

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(uint32_t(b) << 16);
}

// float32 -> bfloat16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// Per-tap actions and ring slots of one step, passed to kernels by value.
struct TapTable {
  int8_t action[CO_MAX_TAPS];
  int32_t slot[CO_MAX_TAPS];
};

// Window sources of one pool emission, passed by value.
struct PoolTaps {
  int32_t src[CO_MAX_TAPS];
};

constexpr int kBlock = 256;

inline unsigned grid_for(int64_t n, int block = kBlock) {
  return unsigned((n + block - 1) / block);
}

}  // namespace coinf
