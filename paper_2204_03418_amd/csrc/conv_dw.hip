// Depthwise continual convolution step (groups = C_in = C_out).
//
// Each output channel sees one input channel, so the per-step contraction is
// a kH x kW stencil per temporal tap: far too little arithmetic per byte for
// matrix cores.  One thread owns one output element (b, c, i, j): it loads the
// stencil's input neighbourhood once into registers, evaluates every active
// tap from it, and updates that element's partial sums in the float32 ring
// (slot, C, B, Ho, Wo).  Consecutive threads own consecutive output pixels, so
// ring and output traffic is coalesced; the step is bound by HBM.
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

template <typename T, int KH, int KW>
__global__ __launch_bounds__(kBlock) void conv_step_dw_kernel(
    ConvGeom g, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y, int64_t y_bc,
    const float* __restrict__ w, const float* __restrict__ bias, float* __restrict__ ring,
    int64_t ring_slot, TapTable tt) {
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.Cout * So;
  const int32_t idx = int32_t(blockIdx.x) * kBlock + int32_t(threadIdx.x);
  if (idx >= total) return;
  const int32_t p = idx % So;
  const int32_t bc = idx / So;
  const int32_t c = bc % g.Cout;
  const int32_t i = p / g.Wo, jo = p % g.Wo;
  const T* xc = x + int64_t(bc) * x_bc;
  float xv[KH * KW];
#pragma unroll
  for (int u = 0; u < KH; ++u) {
    const int32_t hi = i * g.sH + u * g.dH - g.pH;
#pragma unroll
    for (int v = 0; v < KW; ++v) {
      const int32_t wi = jo * g.sW + v * g.dW - g.pW;
      const bool in = hi >= 0 && hi < g.H && wi >= 0 && wi < g.W;
      xv[u * KW + v] = in ? to_f32<T>(xc[hi * g.W + wi]) : 0.f;
    }
  }
  const float* wc = w + int64_t(c) * g.kT * (KH * KW);
  const int64_t yi = int64_t(bc) * y_bc + p;
  const int32_t ridx = (c * g.B + bc / g.Cout) * So + p;  // ring (slot, C, B, Ho, Wo)
  for (int32_t j = 0; j < g.kT; ++j) {
    const int act = tt.action[j];
    if (act == CO_TAP_NONE) continue;
    const float* wj = wc + j * (KH * KW);
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < KH * KW; ++e) acc = fmaf(wj[e], xv[e], acc);
    float* r = ring + int64_t(tt.slot[j] < 0 ? 0 : tt.slot[j]) * ring_slot + ridx;
    switch (act) {
      case CO_TAP_START: *r = acc; break;
      case CO_TAP_ACC: *r = *r + acc; break;
      case CO_TAP_EMIT: y[yi] = from_f32<T>(*r + acc + bias[c]); break;
      case CO_TAP_EMIT_FRESH: y[yi] = from_f32<T>(acc + bias[c]); break;
      default: break;
    }
  }
}

template <typename T, int KH, int KW>
hipError_t dw_launch(const ConvGeom& g, const ConvLayout& L, char* state, const StepIO& io,
                     const co_step_plan& plan, hipStream_t s) {
  TapTable tt;
  for (int j = 0; j < CO_MAX_TAPS; ++j) {
    tt.action[j] = plan.action[j];
    tt.slot[j] = plan.slot[j];
  }
  hipLaunchKernelGGL((conv_step_dw_kernel<T, KH, KW>), dim3(grid_for(g.out_frame_elems())),
                     dim3(kBlock), 0, s, g, static_cast<const T*>(io.x), io.x_bc,
                     static_cast<T*>(io.y), io.y_bc,
                     reinterpret_cast<const float*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems, tt);
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
