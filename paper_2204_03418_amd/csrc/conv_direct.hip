// Generic continual convolution kernels: the direct step kernel (any groups,
// stride, padding, dilation), the end-padding step, clip-mode convolution and
// the init-time packing of bias, weights and the state header.
//
// The step realises the eager evaluation the paper describes in section 3.1
// (before Principle 3): when a frame arrives, its contribution through every
// temporal tap j is computed at once and stored as a partial sum of the output
// frame that tap feeds; the output whose last tap this frame is completes and
// is emitted.  Partial sums live in a float32 ring of R output frames inside
// the caller's state buffer, laid out (slot, C_out, B, Ho, Wo).
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

// Taps handled per pass of the step kernel: their ring reads are issued
// together and one sweep over the frame's window feeds all their sums.
constexpr int kDirStepTaps = 4;

// One thread per output element (b, o, i, j).  Every temporal tap contracts
// the same window of the arriving frame, so the taps of a pass share one
// sweep over (c, u, v): each input value is loaded once for up to
// kDirStepTaps sums, and the ring partials those taps continue are requested
// before the sweep.  Each tap's sum runs over (c, u, v) in the same order as
// a tap computed alone, so the results do not depend on the pass width.
template <typename T, bool ZERO>
__global__ __launch_bounds__(kBlock) void conv_step_direct_kernel(
    ConvGeom g, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y, int64_t y_bc,
    const float* __restrict__ w, const float* __restrict__ bias, float* __restrict__ ring,
    int64_t ring_slot, TapTable tt) {
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.Cout * So;
  const int32_t idx = int32_t(blockIdx.x) * kBlock + int32_t(threadIdx.x);
  if (idx >= total) return;
  const int32_t p = idx % So;
  const int32_t bo = idx / So;
  const int32_t o = bo % g.Cout;
  const int32_t b = bo / g.Cout;
  const int32_t i = p / g.Wo, jo = p % g.Wo;
  const int32_t grp = o / g.Og;
  const T* xb = x + (int64_t(b) * g.Cin + int64_t(grp) * g.Cg) * x_bc;
  const int32_t kHW = g.kH * g.kW;
  // ring layout (slot, C_out, B, Ho, Wo): channel-major so that consecutive
  // output pixels of all streams are contiguous for every kernel family
  const int32_t ridx = (o * g.B + b) * So + p;
  const int64_t yi = int64_t(bo) * y_bc + p;
  for (int32_t j0 = 0; j0 < g.kT; j0 += kDirStepTaps) {
    int act[kDirStepTaps];
    float* r[kDirStepTaps];
    float prev[kDirStepTaps], acc[kDirStepTaps];
#pragma unroll
    for (int k = 0; k < kDirStepTaps; ++k) {
      const int32_t j = j0 + k;
      act[k] = j < g.kT ? int(tt.action[j]) : CO_TAP_NONE;
      r[k] = ring + int64_t(j < g.kT && tt.slot[j] >= 0 ? tt.slot[j] : 0) * ring_slot + ridx;
      prev[k] = (act[k] == CO_TAP_ACC || act[k] == CO_TAP_EMIT) ? *r[k] : 0.f;
      acc[k] = 0.f;
    }
    if (!ZERO) {
      for (int32_t c = 0; c < g.Cg; ++c) {
        const T* xc = xb + int64_t(c) * x_bc;
        const float* wc = w + (int64_t(o) * g.Cg + c) * g.kT * kHW + int64_t(j0) * kHW;
        for (int32_t u = 0; u < g.kH; ++u) {
          const int32_t hi = i * g.sH + u * g.dH - g.pH;
          if (hi < 0 || hi >= g.H) continue;
          for (int32_t v = 0; v < g.kW; ++v) {
            const int32_t wi = jo * g.sW + v * g.dW - g.pW;
            if (wi < 0 || wi >= g.W) continue;
            const float xv = to_f32<T>(xc[hi * g.W + wi]);
#pragma unroll
            for (int k = 0; k < kDirStepTaps; ++k)
              if (act[k] != CO_TAP_NONE) acc[k] = fmaf(wc[k * kHW + u * g.kW + v], xv, acc[k]);
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kDirStepTaps; ++k) {
      switch (act[k]) {
        case CO_TAP_START: *r[k] = acc[k]; break;
        case CO_TAP_ACC: *r[k] = prev[k] + acc[k]; break;
        case CO_TAP_EMIT: y[yi] = from_f32<T>(prev[k] + acc[k] + bias[o]); break;
        case CO_TAP_EMIT_FRESH: y[yi] = from_f32<T>(acc[k] + bias[o]); break;
        default: break;
      }
    }
  }
}

// Clip-mode regular convolution: one thread per output element.
template <typename T>
__global__ __launch_bounds__(kBlock) void conv_clip_direct_kernel(
    ConvGeom g, int32_t T_in, int32_t T_out, const T* __restrict__ x, const T* __restrict__ w,
    const T* __restrict__ bias, T* __restrict__ y) {
  const int64_t So = int64_t(g.Ho) * g.Wo;
  const int64_t total = int64_t(g.B) * g.Cout * T_out * So;
  const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const int64_t p = idx % So;
  const int64_t t = (idx / So) % T_out;
  const int64_t bo = idx / (So * T_out);
  const int32_t o = int32_t(bo % g.Cout);
  const int32_t b = int32_t(bo / g.Cout);
  const int32_t i = int32_t(p / g.Wo), jo = int32_t(p % g.Wo);
  const int32_t grp = o / g.Og;
  const int64_t S = int64_t(g.H) * g.W;
  float acc = 0.f;
  for (int32_t c = 0; c < g.Cg; ++c) {
    const T* xc = x + (int64_t(b) * g.Cin + int64_t(grp) * g.Cg + c) * T_in * S;
    for (int32_t a = 0; a < g.kT; ++a) {
      const int64_t ti = t * g.sT + int64_t(a) * g.dT - g.pT;
      if (ti < 0 || ti >= T_in) continue;
      for (int32_t u = 0; u < g.kH; ++u) {
        const int32_t hi = i * g.sH + u * g.dH - g.pH;
        if (hi < 0 || hi >= g.H) continue;
        for (int32_t v = 0; v < g.kW; ++v) {
          const int32_t wi = jo * g.sW + v * g.dW - g.pW;
          if (wi < 0 || wi >= g.W) continue;
          const float wv = to_f32<T>(w[(((int64_t(o) * g.Cg + c) * g.kT + a) * g.kH + u) * g.kW + v]);
          acc = fmaf(wv, to_f32<T>(xc[ti * S + hi * g.W + wi]), acc);
        }
      }
    }
  }
  if (g.has_bias) acc += to_f32<T>(bias[o]);
  y[idx] = from_f32<T>(acc);
}

template <typename T>
__global__ __launch_bounds__(kBlock) void pack_bias_kernel(int32_t n, int32_t has_bias,
                                                           const T* __restrict__ src,
                                                           float* __restrict__ dst) {
  const int32_t i = int32_t(blockIdx.x) * kBlock + int32_t(threadIdx.x);
  if (i < n) dst[i] = has_bias ? to_f32<T>(src[i]) : 0.f;
}

// Weights as float32 in PyTorch order; each output channel's (per_out
// consecutive values) times its scale when one is given.
template <typename T>
__global__ __launch_bounds__(kBlock) void pack_f32_kernel(int64_t n, int64_t per_out,
                                                          const T* __restrict__ src,
                                                          const float* __restrict__ wscale,
                                                          float* __restrict__ dst) {
  const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (i < n) dst[i] = wscale ? to_f32<T>(src[i]) * wscale[i / per_out] : to_f32<T>(src[i]);
}

// Batch normalisation folded into a convolution (evaluation mode): the
// per-channel scale gamma / sqrt(var + eps), written where the weight
// packing reads it, and the folded bias bias * scale + beta - mean * scale.
template <typename T>
__global__ __launch_bounds__(kBlock) void bn_fold_kernel(int32_t n, int32_t has_bias,
                                                         const T* __restrict__ bias,
                                                         const float* __restrict__ gamma,
                                                         const float* __restrict__ beta,
                                                         const float* __restrict__ mean,
                                                         const float* __restrict__ var, float eps,
                                                         float* __restrict__ scale,
                                                         float* __restrict__ bdst) {
  const int32_t o = int32_t(blockIdx.x) * kBlock + int32_t(threadIdx.x);
  if (o >= n) return;
  const float sc = gamma[o] / sqrtf(var[o] + eps);
  const float b = has_bias ? to_f32<T>(bias[o]) : 0.f;
  scale[o] = sc;
  bdst[o] = fmaf(b, sc, beta[o] - mean[o] * sc);
}

// The folded weights and bias themselves, in the io dtype: each weight
// scaled and rounded as the matrix-core packing does, the bias rounded from
// the same float32 value the state holds.
template <typename T>
__global__ __launch_bounds__(kBlock) void bn_fold_out_kernel(
    int64_t n, int64_t per_out, int32_t cout, int32_t has_bias, const T* __restrict__ w,
    const T* __restrict__ bias, const float* __restrict__ gamma, const float* __restrict__ beta,
    const float* __restrict__ mean, const float* __restrict__ var, float eps,
    T* __restrict__ w_out, T* __restrict__ b_out) {
  const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (i < n) {
    const int32_t o = int32_t(i / per_out);
    w_out[i] = from_f32<T>(to_f32<T>(w[i]) * (gamma[o] / sqrtf(var[o] + eps)));
  }
  if (i < cout) {
    const int32_t o = int32_t(i);
    const float sc = gamma[o] / sqrtf(var[o] + eps);
    const float b = has_bias ? to_f32<T>(bias[o]) : 0.f;
    b_out[o] = from_f32<T>(fmaf(b, sc, beta[o] - mean[o] * sc));
  }
}

__global__ void write_header_kernel(StateHeader h, StateHeader* dst) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *dst = h;
}

template <typename T>
hipError_t step_direct_t(const ConvGeom& g, const ConvLayout& L, char* state, const StepIO& io,
                         const co_step_plan& plan, bool zero_frame, hipStream_t s) {
  TapTable tt;
  for (int j = 0; j < CO_MAX_TAPS; ++j) {
    tt.action[j] = plan.action[j];
    tt.slot[j] = plan.slot[j];
  }
  const float* w = reinterpret_cast<const float*>(state + L.weight);
  const float* bias = reinterpret_cast<const float*>(state + L.bias);
  float* ring = reinterpret_cast<float*>(state + L.ring);
  const unsigned grid = grid_for(g.out_frame_elems());
  if (zero_frame)
    hipLaunchKernelGGL((conv_step_direct_kernel<T, true>), dim3(grid), dim3(kBlock), 0, s, g,
                       static_cast<const T*>(io.x), io.x_bc, static_cast<T*>(io.y), io.y_bc, w,
                       bias, ring, L.ring_slot_elems, tt);
  else
    hipLaunchKernelGGL((conv_step_direct_kernel<T, false>), dim3(grid), dim3(kBlock), 0, s, g,
                       static_cast<const T*>(io.x), io.x_bc, static_cast<T*>(io.y), io.y_bc, w,
                       bias, ring, L.ring_slot_elems, tt);
  return hipGetLastError();
}

// Persistent forward_steps for small direct layers (temporal stride and
// dilation 1): one thread per output element keeps its weights, the kT - 1
// partial sums it continues and the next frames' inputs in registers for the
// whole clip.  Positions e = (c, u, v) of the reduction are fixed; taps
// outside the frame read zero, which leaves the sum unchanged, so each
// temporal tap's sum runs in the step kernel's order and forward_steps
// matches repeated forward_step.
struct DirSteps {
  int32_t v0;       // virtual time of the first frame, capped at 2^29
  int32_t slot_v0;  // v0 mod R (uncapped)
  int32_t count, T, k0, update;
  int32_t x_bytes, y_bytes;
  int32_t fstride;  // bytes between consecutive frames of the clip
  FastDiv fd_So, fd_Cout, fd_Wo;
};

constexpr int kDirStepsKX = 16;  // reduction positions C_in/G * kH * kW held in registers
constexpr int kDirStepsKT = 4;   // temporal taps held in registers

// KX: reduction positions held (4, 8 or 16); PF: frames in flight (16, 8 or
// 4, so a thread holds 64 raw inputs either way).  The loop is bound by the
// latency of its frame loads, so a small layer keeps more frames in flight.
//
// PLAN (temporal stride or dilation above 1, Principle 5): which output a
// tap feeds, and whether it starts, continues or completes it, depends on
// the frame, so the loop follows the host's step plans (a PlanTable:
// explicit for a stream's first frames, periodic after) and each thread
// keeps its R partial sums in LDS, addressed by the plan's slot.  Per tap
// the arithmetic is the step kernel's: the tap's product, added to the slot
// (ACC, EMIT) or not (START, EMIT_FRESH), back to the slot or out with the
// bias.  The ring's R slots are read once and written back once, stale ones
// included.
template <typename T, int KX, int PF, bool PLAN>
__global__ __launch_bounds__(kBlock) void conv_steps_direct_kernel(
    ConvGeom g, DirSteps ds, PlanTable pt, const T* __restrict__ x, int64_t x_bc,
    T* __restrict__ y, int64_t y_bc, const float* __restrict__ w, const float* __restrict__ bias,
    float* __restrict__ ring, int64_t ring_slot) {
  constexpr int KTM = kDirStepsKT;
  constexpr uint32_t esz = sizeof(T);
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.Cout * So;
  const int32_t idx = int32_t(blockIdx.x) * kBlock + int32_t(threadIdx.x);
  if (idx >= total) return;
  const int32_t bo = fdiv(idx, ds.fd_So);
  const int32_t p = idx - bo * So;
  const int32_t b = fdiv(bo, ds.fd_Cout);
  const int32_t o = bo - b * g.Cout;
  const int32_t i = fdiv(p, ds.fd_Wo), jo = p - i * g.Wo;
  const int32_t grp = o / g.Og;
  const int32_t kHW = g.kH * g.kW;
  const int32_t kT = g.kT;
  const int32_t nk = g.Cg * kHW;
  const int32_t ridx = (o * g.B + b) * So + p;

  // byte offset of each reduction position inside frame 0 of the clip (or
  // out of range), and its weight for every temporal tap
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ds.x_bytes);
  const uint32_t plane = (uint32_t(b) * uint32_t(g.Cin) + uint32_t(grp * g.Cg)) * uint32_t(x_bc);
  int xoff[KX];
  float wr[KX][KTM];
#pragma unroll
  for (int e = 0; e < KX; ++e) {
    const int c = e / (kHW > 0 ? kHW : 1), uv = e - c * kHW;
    const int u = uv / g.kW, v = uv - u * g.kW;
    const int hi = i * g.sH + u * g.dH - g.pH, wi = jo * g.sW + v * g.dW - g.pW;
    const bool in = e < nk && hi >= 0 && hi < g.H && wi >= 0 && wi < g.W;
    xoff[e] = in ? int((plane + uint32_t(c) * uint32_t(x_bc) + uint32_t(hi * g.W + wi)) * esz)
                 : kOutOfRange;
#pragma unroll
    for (int j = 0; j < KTM; ++j)
      wr[e][j] = (e < nk && j < kT) ? w[(int64_t(o) * g.Cg + c) * kT * kHW + int64_t(j) * kHW + uv]
                                    : 0.f;
  }
  const float bo_ = bias[o];
  const int R = g.R;
  float part[KTM];
  __shared__ float pslot[PLAN ? kPlanMaxR : 1][PLAN ? kBlock : 1];
  float* const pp = &pslot[0][PLAN ? threadIdx.x : 0];  // + slot * kBlock
  if constexpr (PLAN) {
    for (int q = 0; q < R; ++q) pp[q * kBlock] = ring[int64_t(q) * ring_slot + ridx];
  } else {
#pragma unroll
    for (int j = 1; j < KTM; ++j) {
      part[j] = 0.f;
      const int tau = ds.v0 - j;
      if (j < kT && tau >= 0) part[j] = ring[int64_t((ds.slot_v0 - j + R) % R) * ring_slot + ridx];
    }
  }
  int ph = 0;  // (PLAN) phase of the next periodic frame
  int k = 0;   // (PLAN) outputs emitted so far in the call

  const int fstride = ds.fstride;
  auto load_frame = [&](int t, uint32_t (&xv)[KX]) {
    if (t < ds.T) {  // uniform; end-padding frames are zero
#pragma unroll
      for (int e = 0; e < KX; ++e) xv[e] = load_raw_at<T>(xr, xoff[e], t * fstride);
    } else {
#pragma unroll
      for (int e = 0; e < KX; ++e) xv[e] = 0u;
    }
  };
  uint32_t xq[PF][KX];  // raw bits, converted when the frame is evaluated
#pragma unroll
  for (int u = 0; u < PF; ++u) load_frame(u, xq[u]);
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, ds.y_bytes);
  const int yoff = int((uint32_t(bo) * uint32_t(y_bc) + uint32_t(p)) * esz);
  for (int t0 = 0; t0 < ds.count; t0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int t = t0 + u;
      if (t >= ds.count) break;
      const int v = ds.v0 + t;
      float cj[KTM];
#pragma unroll
      for (int j = 0; j < KTM; ++j) cj[j] = 0.f;
#pragma unroll
      for (int e = 0; e < KX; ++e)
#pragma unroll
        for (int j = 0; j < KTM; ++j) cj[j] = fmaf(wr[e][j], raw_to_f32<T>(xq[u][e]), cj[j]);
      load_frame(t + PF, xq[u]);
      if constexpr (PLAN) {
        uint64_t code;
        if (t < pt.n_start) {
          code = pt.code_start[t];
        } else {
          code = pt.code_period[ph];
          ph = ph + 1 == pt.period ? 0 : ph + 1;
        }
        float yv = 0.f;
        bool emitted = false;
#pragma unroll
        for (int j = 0; j < KTM; ++j) {
          if (j >= kT) break;  // uniform
          const int act = int(code >> (6 * j)) & 7, sl = int(code >> (6 * j + 3)) & 7;
          if (act == CO_TAP_NONE) continue;  // uniform
          const bool with = act == CO_TAP_ACC || act == CO_TAP_EMIT;
          const float a = with ? pp[sl * kBlock] + cj[j] : cj[j];
          if (act == CO_TAP_EMIT || act == CO_TAP_EMIT_FRESH) {
            yv = a;
            emitted = true;
          } else {
            pp[sl * kBlock] = a;
          }
        }
        store_at(yr, emitted ? yoff : kOutOfRange, emitted ? k * So * int32_t(esz) : 0,
                 from_f32<T>(yv + bo_));
        if (emitted) ++k;
        continue;
      }
      // fold each tap's product into its output without a branch: a missing
      // output (tau < 0) or an unused tap only selects zero, and the one
      // store is always issued, to the out-of-range offset unless tap kT - 1
      // completes an existing output (a store under a branch would make the
      // compiler wait for every frame in flight before each frame)
      float nxt[KTM];
      float yv = 0.f;
#pragma unroll
      for (int j = 0; j < KTM; ++j) {
        const int tau = v - j;
        const int first = tau >= g.pT ? 0 : g.pT - tau;
        const float a = (j == first) ? cj[j] : part[j] + cj[j];
        yv = j == kT - 1 ? a : yv;
        nxt[j] = (j < kT - 1 && tau >= 0) ? a : 0.f;
      }
      const bool emits = v - (kT - 1) >= 0;  // uniform
      store_at(yr, emits ? yoff : kOutOfRange, emits ? (ds.k0 + t) * So * int32_t(esz) : 0,
               from_f32<T>(yv + bo_));
#pragma unroll
      for (int j = KTM - 1; j >= 1; --j) part[j] = nxt[j - 1];
    }
  }
  if (PLAN && ds.update) {
    for (int q = 0; q < R; ++q) ring[int64_t(q) * ring_slot + ridx] = pp[q * kBlock];
  } else if (ds.update) {
    const int v1 = ds.v0 + ds.count;
    const int s1 = (ds.slot_v0 + ds.count) % R;
#pragma unroll
    for (int j = 1; j < KTM; ++j) {
      const int tau = v1 - j;
      if (j < kT && tau >= 0) ring[int64_t((s1 - j + R) % R) * ring_slot + ridx] = part[j];
    }
  }
}

template <typename T>
hipError_t direct_steps_t(const ConvGeom& g, const ConvLayout& L, char* state, const void* x,
                          int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                          int64_t n0, bool update, hipStream_t s) {
  DirSteps ds;
  const int64_t v0 = n0 + g.pT;
  ds.v0 = int32_t(v0 < (int64_t(1) << 29) ? v0 : (int64_t(1) << 29));
  ds.slot_v0 = int32_t(v0 % g.R);
  ds.count = count;
  ds.T = nreal;
  ds.k0 = int32_t(n0 - (n0 > g.d ? n0 : g.d));
  ds.update = update ? 1 : 0;
  const int64_t esz = sizeof(T);
  ds.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * x_bc + int64_t(nreal) * g.S()) * esz);
  ds.y_bytes = int32_t(int64_t(g.B) * g.Cout * y_bc * esz);
  ds.fstride = int32_t(g.S() * esz);
  ds.fd_So = make_fastdiv(uint32_t(g.So()));
  ds.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  ds.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  const int64_t nk = int64_t(g.Cg) * g.kH * g.kW;
  const bool plan = g.sT != 1 || g.dT != 1;
  PlanTable pt{};
  if (plan) plan_table(g, n0, count, &pt);
  // (the plan-driven frame body is larger: 16 frames in flight would not
  // unroll, and a frame register indexed at run time goes to scratch)
  auto kern = plan ? (nk <= 4   ? conv_steps_direct_kernel<T, 4, 8, true>
                      : nk <= 8 ? conv_steps_direct_kernel<T, 8, 8, true>
                                : conv_steps_direct_kernel<T, kDirStepsKX, 4, true>)
                   : (nk <= 4   ? conv_steps_direct_kernel<T, 4, 16, false>
                      : nk <= 8 ? conv_steps_direct_kernel<T, 8, 8, false>
                                : conv_steps_direct_kernel<T, kDirStepsKX, 4, false>);
  hipLaunchKernelGGL(kern, dim3(grid_for(g.out_frame_elems())),
                     dim3(kBlock), 0, s, g, ds, pt, static_cast<const T*>(x), x_bc,
                     static_cast<T*>(y), y_bc, reinterpret_cast<const float*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_step_direct(const ConvGeom& g, const ConvLayout& L, char* state,
                                   const StepIO& io, const co_step_plan& plan, bool zero_frame,
                                   hipStream_t s) {
  if (g.dtype == CO_BF16) return step_direct_t<bf16_t>(g, L, state, io, plan, zero_frame, s);
  return step_direct_t<float>(g, L, state, io, plan, zero_frame, s);
}

namespace {

int64_t round256(int64_t n) { return (n + 255) & ~int64_t(255); }

// The staged copies of one step: x (B*C_in contiguous planes) and, when the
// output lies past 32-bit reach, y (B*C_out contiguous planes).
struct StagedBytes {
  int64_t x, y;
};

StagedBytes staged_bytes(const ConvGeom& g, const StepIO& io) {
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  const int64_t yrows = int64_t(g.B) * g.Cout;
  const bool y_far = io.y && ((yrows - 1) * io.y_bc + g.So()) * esz >= (int64_t(1) << 31);
  return {int64_t(g.B) * g.Cin * g.S() * esz, y_far ? yrows * g.So() * esz : 0};
}

}  // namespace

int64_t conv_step_staging_bytes(const ConvGeom& g, const StepIO& io) {
  bool staged = false;
  switch (g.algo) {
    case CO_ALGO_GEMM: staged = gemm_step_needs_staging(g, io); break;
    case CO_ALGO_GEMM_REG: staged = reg_step_needs_staging(g, io); break;
    default: return 0;  // the direct and depthwise kernels use 64-bit offsets
  }
  if (!staged) return 0;
  const StagedBytes b = staged_bytes(g, io);
  return round256(b.x) + round256(b.y);
}

hipError_t launch_conv_step_staged(const ConvGeom& g, const ConvLayout& L, char* state,
                                   const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  const int64_t S = g.S(), So = g.So(), lim = int64_t(1) << 31;
  const int64_t xrows = int64_t(g.B) * g.Cin, yrows = int64_t(g.B) * g.Cout;
  const StagedBytes sb = staged_bytes(g, io);
  const bool y_far = sb.y > 0;
  // An input frame that is already contiguous and 16-byte aligned, with an
  // output in 32-bit reach, is what the copies below would produce: the
  // kernel has declined the geometry itself, and staging cannot help.
  const bool x_plain = io.x_bc == S && reinterpret_cast<uintptr_t>(io.x) % 16 == 0;
  if (!io.x || (x_plain && !y_far) || xrows * S * esz >= lim || yrows * So * esz >= lim)
    return hipErrorInvalidValue;
  void* xs = nullptr;
  void* ys = nullptr;
  hipError_t e = hipSuccess;
  const bool own = io.ws == nullptr;  // no workspace: stream-ordered allocations
  if (own) {
    e = hipMallocAsync(&xs, size_t(sb.x), s);
    if (e == hipSuccess && y_far) e = hipMallocAsync(&ys, size_t(sb.y), s);
  } else {
    if (round256(sb.x) + round256(sb.y) > io.ws_bytes) return hipErrorInvalidValue;
    xs = io.ws;
    if (y_far) ys = static_cast<char*>(io.ws) + round256(sb.x);
  }
  if (e == hipSuccess)
    e = hipMemcpy2DAsync(xs, size_t(S * esz), io.x, size_t(io.x_bc * esz), size_t(S * esz),
                         size_t(xrows), hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess) {
    const StepIO sio{static_cast<const char*>(xs), S, y_far ? static_cast<char*>(ys) : io.y,
                     y_far || !io.y ? So : io.y_bc};
    e = launch_conv_step(g, L, state, sio, plan, false, s);
  }
  if (e == hipSuccess && y_far)
    e = hipMemcpy2DAsync(io.y, size_t(io.y_bc * esz), ys, size_t(So * esz), size_t(So * esz),
                         size_t(yrows), hipMemcpyDeviceToDevice, s);
  if (own) {
    for (void* p : {xs, ys}) {
      if (!p) continue;
      const hipError_t f = hipFreeAsync(p, s);
      if (e == hipSuccess) e = f;
    }
  }
  return e;
}

bool direct_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames) {
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  // temporal stride or dilation: the plan-driven form (R <= 8 slots)
  return g.algo == CO_ALGO_DIRECT && ((g.sT == 1 && g.dT == 1) || plan_table_fits(g)) &&
         g.kT <= kDirStepsKT &&
         int64_t(g.Cg) * g.kH * g.kW <= kDirStepsKX &&
         int64_t(g.B) * g.Cin * x_frames * g.S() * esz < (int64_t(1) << 31) &&
         int64_t(g.B) * g.Cout * y_frames * g.So() * esz < (int64_t(1) << 31);
}

hipError_t launch_conv_steps_direct(const ConvGeom& g, const ConvLayout& L, char* state,
                                    const void* x, int64_t x_bc, int32_t nreal, int32_t count,
                                    void* y, int64_t y_bc, int64_t n0, bool update,
                                    hipStream_t s) {
  if (g.dtype == CO_BF16)
    return direct_steps_t<bf16_t>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  return direct_steps_t<float>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
}

hipError_t launch_conv_step(const ConvGeom& g, const ConvLayout& L, char* state,
                            const StepIO& io, const co_step_plan& plan, bool zero_frame,
                            hipStream_t s) {
  // An end-padding frame contributes exactly zero: every algorithm shares the
  // ring layout, so the direct kernel's no-contraction path serves them all.
  if (zero_frame) return launch_conv_step_direct(g, L, state, io, plan, true, s);
  switch (g.algo) {
    case CO_ALGO_DEPTHWISE: return launch_conv_step_depthwise(g, L, state, io, plan, s);
    case CO_ALGO_GEMM: return launch_conv_step_gemm(g, L, state, io, plan, s);
    case CO_ALGO_GEMM_REG: return launch_conv_step_reg(g, L, state, io, plan, s);
    default: return launch_conv_step_direct(g, L, state, io, plan, false, s);
  }
}

namespace {

// Weight packing of the handle's algorithm and the state header, after the
// bias went in; wscale as launch_pack_gemm.
hipError_t pack_weights_and_header(const ConvGeom& g, const ConvLayout& L, char* state,
                                   const void* weight, const float* wscale,
                                   const StateHeader& hdr, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (g.algo == CO_ALGO_GEMM) {
    e = launch_pack_gemm(g, L, state, weight, wscale, s);
    if (e == hipSuccess && L.steps_weight_bytes > 0)
      e = launch_pack_gemm_steps(g, L, state, weight, wscale, s);
  } else if (g.algo == CO_ALGO_GEMM_REG) {
    e = launch_pack_reg(g, L, state, weight, wscale, s);
  } else {
    const int64_t per_out = int64_t(g.Cg) * g.kT * g.kH * g.kW;
    const int64_t n = int64_t(g.Cout) * per_out;
    float* wdst = reinterpret_cast<float*>(state + L.weight);
    if (g.dtype == CO_BF16)
      hipLaunchKernelGGL(pack_f32_kernel<bf16_t>, dim3(grid_for(n)), dim3(kBlock), 0, s, n,
                         per_out, static_cast<const bf16_t*>(weight), wscale, wdst);
    else
      hipLaunchKernelGGL(pack_f32_kernel<float>, dim3(grid_for(n)), dim3(kBlock), 0, s, n,
                         per_out, static_cast<const float*>(weight), wscale, wdst);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(write_header_kernel, dim3(1), dim3(64), 0, s, hdr,
                     reinterpret_cast<StateHeader*>(state + L.header));
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_init(const ConvGeom& g, const ConvLayout& L, char* state,
                            const void* weight, const void* bias, const StateHeader& hdr,
                            hipStream_t s) {
  float* bdst = reinterpret_cast<float*>(state + L.bias);
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(pack_bias_kernel<bf16_t>, dim3(grid_for(g.Cout)), dim3(kBlock), 0, s,
                       g.Cout, g.has_bias, static_cast<const bf16_t*>(bias), bdst);
  else
    hipLaunchKernelGGL(pack_bias_kernel<float>, dim3(grid_for(g.Cout)), dim3(kBlock), 0, s,
                       g.Cout, g.has_bias, static_cast<const float*>(bias), bdst);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return pack_weights_and_header(g, L, state, weight, nullptr, hdr, s);
}

hipError_t launch_conv_init_bn(const ConvGeom& g, const ConvLayout& L, char* state,
                               const void* weight, const void* bias, const float* gamma,
                               const float* beta, const float* mean, const float* var, float eps,
                               const StateHeader& hdr, hipStream_t s) {
  // The scales go to the start of the ring (at least C_out floats, and not
  // read before the first step writes it), where the weight packing reads
  // them; the folded bias goes to the state's bias.
  float* bdst = reinterpret_cast<float*>(state + L.bias);
  float* scale = reinterpret_cast<float*>(state + L.ring);
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(bn_fold_kernel<bf16_t>, dim3(grid_for(g.Cout)), dim3(kBlock), 0, s,
                       g.Cout, g.has_bias, static_cast<const bf16_t*>(bias), gamma, beta, mean,
                       var, eps, scale, bdst);
  else
    hipLaunchKernelGGL(bn_fold_kernel<float>, dim3(grid_for(g.Cout)), dim3(kBlock), 0, s,
                       g.Cout, g.has_bias, static_cast<const float*>(bias), gamma, beta, mean,
                       var, eps, scale, bdst);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return pack_weights_and_header(g, L, state, weight, scale, hdr, s);
}

hipError_t launch_bn_fold(const ConvGeom& g, const void* weight, const void* bias,
                          const float* gamma, const float* beta, const float* mean,
                          const float* var, float eps, void* w_out, void* b_out, hipStream_t s) {
  const int64_t per_out = int64_t(g.Cg) * g.kT * g.kH * g.kW;
  const int64_t n = per_out * g.Cout;
  const unsigned grid = grid_for(std::max<int64_t>(n, g.Cout));
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(bn_fold_out_kernel<bf16_t>, dim3(grid), dim3(kBlock), 0, s, n, per_out,
                       g.Cout, g.has_bias, static_cast<const bf16_t*>(weight),
                       static_cast<const bf16_t*>(bias), gamma, beta, mean, var, eps,
                       static_cast<bf16_t*>(w_out), static_cast<bf16_t*>(b_out));
  else
    hipLaunchKernelGGL(bn_fold_out_kernel<float>, dim3(grid), dim3(kBlock), 0, s, n, per_out,
                       g.Cout, g.has_bias, static_cast<const float*>(weight),
                       static_cast<const float*>(bias), gamma, beta, mean, var, eps,
                       static_cast<float*>(w_out), static_cast<float*>(b_out));
  return hipGetLastError();
}

hipError_t launch_conv_clip(const ConvGeom& g, int32_t T, int32_t T_out, const void* weight,
                            const void* bias, const void* x, void* y, hipStream_t s) {
  const int64_t total = int64_t(g.B) * g.Cout * T_out * g.So();
  if (total == 0) return hipSuccess;
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(conv_clip_direct_kernel<bf16_t>, dim3(grid_for(total)), dim3(kBlock), 0,
                       s, g, T, T_out, static_cast<const bf16_t*>(x),
                       static_cast<const bf16_t*>(weight), static_cast<const bf16_t*>(bias),
                       static_cast<bf16_t*>(y));
  else
    hipLaunchKernelGGL(conv_clip_direct_kernel<float>, dim3(grid_for(total)), dim3(kBlock), 0,
                       s, g, T, T_out, static_cast<const float*>(x),
                       static_cast<const float*>(weight), static_cast<const float*>(bias),
                       static_cast<float*>(y));
  return hipGetLastError();
}

}  // namespace coinf
