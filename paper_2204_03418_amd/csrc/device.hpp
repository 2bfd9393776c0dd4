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

// float32 -> bfloat16, round to nearest even (the hardware conversion: one
// instruction, no branch; NaN stays a quiet NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, __bf16(f));
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

// Weight w of output channel o times that channel's scale (batch
// normalisation folded into the weights at init), rounded once to T; with no
// scale, w unchanged.
template <typename T>
__device__ __forceinline__ T scaled_weight(T w, const float* scale, int o) {
  if (!scale) return w;
  return from_f32<T>(to_f32<T>(w) * scale[o]);
}

// n / f.d for 0 <= n < 2^31 (see FastDiv).
__device__ __forceinline__ int fdiv(int n, const FastDiv& f) {
  return int((uint64_t(uint32_t(n)) * f.m) >> f.s);
}

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

// Raw buffer resource over `bytes` bytes from `base` (CDNA raw-buffer word 3:
// 32-bit data format, no swizzle).  Reads at offsets past `bytes` return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), short(0), bytes, 0x00020000);
}

// Byte offset that lies past every buffer this library builds (< 2^31), so a
// read from it returns 0: out-of-frame stencil taps load through it instead of
// branching around the load.
constexpr int kOutOfRange = 0x7ffffff0;

// Element `e` of a T buffer, or 0.0 when !in (no branch: the offset moves out
// of range and the hardware returns zero).
template <typename T>
__device__ __forceinline__ float load_or_zero(__amdgpu_buffer_rsrc_t r, int e, bool in);
template <>
__device__ __forceinline__ float load_or_zero<bf16_t>(__amdgpu_buffer_rsrc_t r, int e, bool in) {
  const int off = in ? e * 2 : kOutOfRange;
  return bf16_to_f32(bf16_t(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0)));
}
template <>
__device__ __forceinline__ float load_or_zero<float>(__amdgpu_buffer_rsrc_t r, int e, bool in) {
  const int off = in ? e * 4 : kOutOfRange;
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

// Element at byte offset voff + soff of a T buffer as float; 0.0 when the
// offset lies past the buffer (out-of-range reads return zero).
template <typename T>
__device__ __forceinline__ float load_or_zero_at(__amdgpu_buffer_rsrc_t r, int voff, int soff);
template <>
__device__ __forceinline__ float load_or_zero_at<bf16_t>(__amdgpu_buffer_rsrc_t r, int voff,
                                                         int soff) {
  return bf16_to_f32(bf16_t(__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0)));
}
template <>
__device__ __forceinline__ float load_or_zero_at<float>(__amdgpu_buffer_rsrc_t r, int voff,
                                                        int soff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// Raw bits of the T element at byte offset voff + soff (0 when the offset
// lies past the buffer): the 16-bit pattern of a bf16, the 32-bit pattern of
// an fp32.  Prefetch buffers hold raw bits and convert them when the frame is
// used: an instruction that touched a loaded value right after its load
// would make the wave wait for that load there.
template <typename T>
__device__ __forceinline__ uint32_t load_raw_at(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  if constexpr (sizeof(T) == 2)
    return uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0));
  else
    return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
}
template <typename T>
__device__ __forceinline__ float raw_to_f32(uint32_t raw) {
  if constexpr (sizeof(T) == 2)
    return __uint_as_float(raw << 16);
  else
    return __uint_as_float(raw);
}

// Store v at byte offset voff + soff of a T buffer.
__device__ __forceinline__ void store_at(__amdgpu_buffer_rsrc_t r, int voff, int soff, bf16_t v) {
  __builtin_amdgcn_raw_buffer_store_b16(v, r, voff, soff, 0);
}
__device__ __forceinline__ void store_at(__amdgpu_buffer_rsrc_t r, int voff, int soff, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, voff, soff, 0);
}

inline unsigned grid_for(int64_t n, int block = kBlock) {
  return unsigned((n + block - 1) / block);
}

}  // namespace coinf
