// Depthwise continual convolution step (groups = C_in = C_out).
//
// Each output channel sees one input channel, so the per-step contraction is
// a kH x kW stencil per temporal tap: far too little arithmetic per byte for
// matrix cores.  One thread owns one output element (b, c, i, j).  It loads
// the stencil's input neighbourhood once (buffer loads; out-of-frame taps read
// an out-of-range offset, which returns zero, so no load waits behind a
// branch), issues the ring reads its add/complete taps need, evaluates every
// active tap
// from registers and updates that element's partial sums in the float32 ring
// (slot, C, B, Ho, Wo).  Consecutive threads own consecutive output pixels,
// so ring and output traffic is coalesced; the step is bound by HBM.
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

constexpr int kDwTaps = 4;  // active taps handled per pass (ring reads in flight)

// Active taps of one step, compacted: tap index, action, ring slot.
struct ActiveTaps {
  int32_t n;
  FastDiv fd_So, fd_Cout, fd_Wo;  // dividers: pixels per frame, C_out, Wo
  int32_t tap[CO_MAX_TAPS];
  int32_t act[CO_MAX_TAPS];
  int32_t slot[CO_MAX_TAPS];
};

template <typename T, int KH, int KW>
__global__ __launch_bounds__(kBlock) void conv_step_dw_kernel(
    ConvGeom g, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y, int64_t y_bc,
    const float* __restrict__ w, const float* __restrict__ bias, float* __restrict__ ring,
    int64_t ring_slot, ActiveTaps at) {
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.Cout * So;
  const int32_t idx = int32_t(blockIdx.x) * kBlock + int32_t(threadIdx.x);
  if (idx >= total) return;
  const int32_t bc = fdiv(idx, at.fd_So);
  const int32_t p = idx - bc * So;
  const int32_t bq = fdiv(bc, at.fd_Cout);
  const int32_t c = bc - bq * g.Cout;
  const int32_t i = fdiv(p, at.fd_Wo), jo = p - i * g.Wo;
  const int64_t yi = int64_t(bc) * y_bc + p;
  const int32_t ridx = (c * g.B + bq) * So + p;  // ring (slot, C, B, Ho, Wo)

  // stencil of the arriving frame: buffer loads whose out-of-frame taps
  // read zero from an out-of-range offset, so all loads issue together
  // one wave-uniform resource over everything reachable from the frame pointer
  const int x_extent = int(((int64_t(g.B) * g.Cin - 1) * x_bc + g.H * g.W) * int64_t(sizeof(T)));
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, x_extent);
  const int plane = int(int64_t(bc) * x_bc);
  float xv[KH * KW];
#pragma unroll
  for (int u = 0; u < KH; ++u) {
    const int32_t hi = i * g.sH + u * g.dH - g.pH;
#pragma unroll
    for (int v = 0; v < KW; ++v) {
      const int32_t wi = jo * g.sW + v * g.dW - g.pW;
      const bool in = hi >= 0 && hi < g.H && wi >= 0 && wi < g.W;
      xv[u * KW + v] = load_or_zero<T>(xr, plane + hi * g.W + wi, in);
    }
  }
  const float* wc = w + int64_t(c) * g.kT * (KH * KW);
  const float bo = bias[c];

  for (int32_t a0 = 0; a0 < at.n; a0 += kDwTaps) {
    // ring values of this pass's add/complete taps, requested up front
    float prev[kDwTaps];
#pragma unroll
    for (int k = 0; k < kDwTaps; ++k) {
      prev[k] = 0.f;
      const int32_t a = a0 + k;
      if (a < at.n && (at.act[a] == CO_TAP_ACC || at.act[a] == CO_TAP_EMIT))
        prev[k] = ring[int64_t(at.slot[a]) * ring_slot + ridx];
    }
#pragma unroll
    for (int k = 0; k < kDwTaps; ++k) {
      const int32_t a = a0 + k;
      if (a >= at.n) break;
      const float* wj = wc + at.tap[a] * (KH * KW);
      float acc = prev[k];
#pragma unroll
      for (int e = 0; e < KH * KW; ++e) acc = fmaf(wj[e], xv[e], acc);
      const int act = at.act[a];
      if (act == CO_TAP_START || act == CO_TAP_ACC)
        ring[int64_t(at.slot[a]) * ring_slot + ridx] = acc;
      else
        y[yi] = from_f32<T>(acc + bo);
    }
  }
}

template <typename T, int KH, int KW>
hipError_t dw_launch(const ConvGeom& g, const ConvLayout& L, char* state, const StepIO& io,
                     const co_step_plan& plan, hipStream_t s) {
  ActiveTaps at;
  at.n = 0;
  for (int j = 0; j < g.kT; ++j) {
    if (plan.action[j] == CO_TAP_NONE) continue;
    at.tap[at.n] = j;
    at.act[at.n] = plan.action[j];
    at.slot[at.n] = plan.slot[j] < 0 ? 0 : plan.slot[j];
    ++at.n;
  }
  if (at.n == 0) return hipSuccess;
  at.fd_So = make_fastdiv(uint32_t(g.So()));
  at.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  at.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  hipLaunchKernelGGL((conv_step_dw_kernel<T, KH, KW>), dim3(grid_for(g.out_frame_elems())),
                     dim3(kBlock), 0, s, g, static_cast<const T*>(io.x), io.x_bc,
                     static_cast<T*>(io.y), io.y_bc,
                     reinterpret_cast<const float*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems, at);
  return hipGetLastError();
}

template <typename T>
hipError_t dw_dispatch(const ConvGeom& g, const ConvLayout& L, char* state, const StepIO& io,
                       const co_step_plan& plan, hipStream_t s) {
  if (g.kH == 3 && g.kW == 3) return dw_launch<T, 3, 3>(g, L, state, io, plan, s);
  if (g.kH == 1 && g.kW == 1) return dw_launch<T, 1, 1>(g, L, state, io, plan, s);
  if (g.kH == 3 && g.kW == 1) return dw_launch<T, 3, 1>(g, L, state, io, plan, s);
  if (g.kH == 5 && g.kW == 5) return dw_launch<T, 5, 5>(g, L, state, io, plan, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_conv_step_depthwise(const ConvGeom& g, const ConvLayout& L, char* state,
                                      const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  if (g.dtype == CO_BF16) return dw_dispatch<bf16_t>(g, L, state, io, plan, s);
  return dw_dispatch<float>(g, L, state, io, plan, s);
}

}  // namespace coinf
