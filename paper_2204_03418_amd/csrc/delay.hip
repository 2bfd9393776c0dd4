// Delay line (section 3.2, co.Delay) and residual merge (section 3.1.1,
// Principle 7): the streams of parallel branches with different delays meet
// on the same frame.  The state is a ring of d input frames (slot, B, C, E)
// in the io dtype; frame n goes to slot n mod d, where it is read back d
// steps later.  Merges add in float32 and round once to the io dtype.
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

template <typename T, bool ADD>
__global__ __launch_bounds__(kBlock) void delay_step_kernel(DelayGeom g, const T* x, const T* a,
                                                            T* y, T* ring, int64_t slot,
                                                            int32_t emit, int32_t update) {
  const int64_t frame = int64_t(g.B) * g.C * g.E;
  const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= frame) return;
  const T xi = x[i];
  T old = xi;  // delay 0: the frame itself
  if (g.d > 0) {
    T* r = ring + slot * frame + i;
    old = *r;
    if (update) *r = xi;
  }
  if (emit) {
    // a and y may be the same buffer: a[i] is read before y[i] is written
    if (ADD)
      y[i] = from_f32<T>(to_f32<T>(a[i]) + to_f32<T>(old));
    else
      y[i] = old;
  }
}

// Outputs i < nout of a clip call: step t = t_first + i outputs frame
// n0 + t - d, which is clip frame t - d or, before the clip, a ring slot.
template <typename T, bool ADD>
__global__ __launch_bounds__(kBlock) void delay_steps_kernel(DelayGeom g, const T* x,
                                                             int32_t T_in, const T* a, T* y,
                                                             int32_t y_frames, const T* ring,
                                                             int64_t n0, int32_t t_first,
                                                             int32_t nout) {
  const int64_t BC = int64_t(g.B) * g.C;
  const int64_t total = BC * nout * g.E;
  const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const int64_t e = idx % g.E;
  const int64_t i = (idx / g.E) % nout;
  const int64_t bc = idx / (int64_t(g.E) * nout);
  const int64_t src = n0 + t_first + i - g.d;  // absolute frame index
  const T val = src >= n0 ? x[(bc * T_in + (src - n0)) * g.E + e]
                          : ring[((src % g.d) * BC + bc) * g.E + e];
  const int64_t o = (bc * y_frames + i) * g.E + e;
  if (ADD)
    y[o] = from_f32<T>(to_f32<T>(a[(bc * nout + i) * g.E + e]) + to_f32<T>(val));
  else
    y[o] = val;
}

// After a clip call the ring holds its last min(T, d) frames.
template <typename T>
__global__ __launch_bounds__(kBlock) void delay_ring_kernel(DelayGeom g, const T* x,
                                                            int32_t T_in, T* ring, int64_t n0,
                                                            int32_t t0) {
  const int64_t BC = int64_t(g.B) * g.C;
  const int32_t nf = T_in - t0;
  const int64_t total = BC * nf * g.E;
  const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const int64_t e = idx % g.E;
  const int64_t t = t0 + (idx / g.E) % nf;
  const int64_t bc = idx / (int64_t(g.E) * nf);
  ring[(((n0 + t) % g.d) * BC + bc) * g.E + e] = x[(bc * T_in + t) * g.E + e];
}

template <typename T>
__global__ __launch_bounds__(kBlock) void add_frames_kernel(const T* a, const T* x, T* y,
                                                            int64_t rows, int32_t E,
                                                            int32_t a_frames, int32_t x_frames,
                                                            int32_t x_offset) {
  const int64_t total = rows * a_frames * E;
  const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const int64_t e = idx % E;
  const int64_t i = (idx / E) % a_frames;
  const int64_t r = idx / (int64_t(E) * a_frames);
  y[idx] = from_f32<T>(to_f32<T>(a[idx]) + to_f32<T>(x[(r * x_frames + i + x_offset) * E + e]));
}

__global__ void delay_header_kernel(StateHeader h, StateHeader* dst) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *dst = h;
}

template <typename T>
hipError_t step_t(const DelayGeom& g, char* state, const void* x, const void* a, void* y,
                  int64_t n, bool emit, bool update, hipStream_t s) {
  T* ring = reinterpret_cast<T*>(state + g.ring_offset());
  const int64_t slot = g.d > 0 ? n % g.d : 0;
  const unsigned grid = grid_for(g.frame());
  if (a)
    hipLaunchKernelGGL((delay_step_kernel<T, true>), dim3(grid), dim3(kBlock), 0, s, g,
                       static_cast<const T*>(x), static_cast<const T*>(a), static_cast<T*>(y),
                       ring, slot, emit ? 1 : 0, update ? 1 : 0);
  else
    hipLaunchKernelGGL((delay_step_kernel<T, false>), dim3(grid), dim3(kBlock), 0, s, g,
                       static_cast<const T*>(x), nullptr, static_cast<T*>(y), ring, slot,
                       emit ? 1 : 0, update ? 1 : 0);
  return hipGetLastError();
}

template <typename T>
hipError_t steps_t(const DelayGeom& g, char* state, const void* x, int32_t T_in, const void* a,
                   void* y, int32_t y_frames, int64_t n0, int32_t t_first, int32_t nout,
                   bool update, hipStream_t s) {
  T* ring = reinterpret_cast<T*>(state + g.ring_offset());
  if (nout > 0) {
    const int64_t total = int64_t(g.B) * g.C * nout * g.E;
    if (a)
      hipLaunchKernelGGL((delay_steps_kernel<T, true>), dim3(grid_for(total)), dim3(kBlock), 0,
                         s, g, static_cast<const T*>(x), T_in, static_cast<const T*>(a),
                         static_cast<T*>(y), y_frames, ring, n0, t_first, nout);
    else
      hipLaunchKernelGGL((delay_steps_kernel<T, false>), dim3(grid_for(total)), dim3(kBlock), 0,
                         s, g, static_cast<const T*>(x), T_in, nullptr, static_cast<T*>(y),
                         y_frames, ring, n0, t_first, nout);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (update && g.d > 0 && T_in > 0) {
    // stream order: the ring is overwritten only after the outputs read it
    const int32_t t0 = T_in > g.d ? T_in - g.d : 0;
    const int64_t total = int64_t(g.B) * g.C * (T_in - t0) * g.E;
    hipLaunchKernelGGL(delay_ring_kernel<T>, dim3(grid_for(total)), dim3(kBlock), 0, s, g,
                       static_cast<const T*>(x), T_in, ring, n0, t0);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_delay_init(const DelayGeom& g, char* state, const StateHeader& hdr,
                             hipStream_t s) {
  hipLaunchKernelGGL(delay_header_kernel, dim3(1), dim3(64), 0, s, hdr,
                     reinterpret_cast<StateHeader*>(state));
  return hipGetLastError();
}

hipError_t launch_delay_step(const DelayGeom& g, char* state, const void* x, const void* a,
                             void* y, int64_t n, bool emit, bool update, hipStream_t s) {
  if (g.dtype == CO_BF16) return step_t<bf16_t>(g, state, x, a, y, n, emit, update, s);
  return step_t<float>(g, state, x, a, y, n, emit, update, s);
}

hipError_t launch_delay_steps(const DelayGeom& g, char* state, const void* x, int32_t T,
                              const void* a, void* y, int32_t y_frames, int64_t n0,
                              int32_t t_first, int32_t nout, bool update, hipStream_t s) {
  if (g.dtype == CO_BF16)
    return steps_t<bf16_t>(g, state, x, T, a, y, y_frames, n0, t_first, nout, update, s);
  return steps_t<float>(g, state, x, T, a, y, y_frames, n0, t_first, nout, update, s);
}

namespace {

// Elementwise activation: the stateless maps (nn.ReLU and the like) a
// continual network applies to each frame as it applies them to a clip.
// ReLU is exact in either dtype: max(v, 0) of a representable value.
template <typename T>
__global__ __launch_bounds__(kBlock) void act_kernel(const T* __restrict__ x, T* __restrict__ y,
                                                     int64_t n, int32_t act) {
  const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n) return;
  y[i] = act == CO_ACT_RELU ? from_f32<T>(fmaxf(to_f32<T>(x[i]), 0.f)) : x[i];
}

}  // namespace

hipError_t launch_act(const void* x, void* y, int64_t n, int32_t dtype, int32_t act,
                      hipStream_t s) {
  if (dtype == CO_BF16)
    hipLaunchKernelGGL(act_kernel<bf16_t>, dim3(grid_for(n)), dim3(kBlock), 0, s,
                       static_cast<const bf16_t*>(x), static_cast<bf16_t*>(y), n, act);
  else
    hipLaunchKernelGGL(act_kernel<float>, dim3(grid_for(n)), dim3(kBlock), 0, s,
                       static_cast<const float*>(x), static_cast<float*>(y), n, act);
  return hipGetLastError();
}

hipError_t launch_add_frames(const void* a, const void* x, void* y, int64_t rows, int32_t E,
                             int32_t a_frames, int32_t x_frames, int32_t x_offset, int32_t dtype,
                             hipStream_t s) {
  const int64_t total = rows * a_frames * E;
  if (total == 0) return hipSuccess;
  if (dtype == CO_BF16)
    hipLaunchKernelGGL(add_frames_kernel<bf16_t>, dim3(grid_for(total)), dim3(kBlock), 0, s,
                       static_cast<const bf16_t*>(a), static_cast<const bf16_t*>(x),
                       static_cast<bf16_t*>(y), rows, E, a_frames, x_frames, x_offset);
  else
    hipLaunchKernelGGL(add_frames_kernel<float>, dim3(grid_for(total)), dim3(kBlock), 0, s,
                       static_cast<const float*>(a), static_cast<const float*>(x),
                       static_cast<float*>(y), rows, E, a_frames, x_frames, x_offset);
  return hipGetLastError();
}

}  // namespace coinf
