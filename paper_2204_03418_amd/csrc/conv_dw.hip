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
#include <algorithm>

#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

constexpr int kDwTaps = 4;  // active taps handled per pass (ring reads in flight)

// Active taps of one step, compacted: tap index, action, ring slot.
struct ActiveTaps {
  int32_t n;
  FastDiv fd_So, fd_B, fd_Wo;  // dividers: pixels per frame, streams, Wo
  int32_t tap[CO_MAX_TAPS];
  int32_t act[CO_MAX_TAPS];
  int32_t slot[CO_MAX_TAPS];
};

// Threads per workgroup of the step kernel: one wave per workgroup measures
// fastest for these latency-bound steps.
constexpr int kDwStepBlock = 64;

template <typename T, int KH, int KW>
__global__ __launch_bounds__(kDwStepBlock) void conv_step_dw_kernel(
    ConvGeom g, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y, int64_t y_bc,
    const float* __restrict__ w, const float* __restrict__ bias, float* __restrict__ ring,
    int64_t ring_slot, ActiveTaps at) {
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.Cout * So;
  const int32_t idx = int32_t(blockIdx.x) * kDwStepBlock + int32_t(threadIdx.x);
  if (idx >= total) return;
  // threads in ring order (c, b, pixel): the ring is most of a step's bytes,
  // so its reads and writes are the ones kept contiguous across a wave
  const int32_t cb = fdiv(idx, at.fd_So);
  const int32_t p = idx - cb * So;
  const int32_t c = fdiv(cb, at.fd_B);
  const int32_t bq = cb - c * g.B;
  const int32_t bc = bq * g.Cout + c;
  const int32_t i = fdiv(p, at.fd_Wo), jo = p - i * g.Wo;
  const int64_t yi = int64_t(bc) * y_bc + p;
  const int32_t ridx = idx;  // ring (slot, C, B, Ho, Wo)

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
  at.fd_B = make_fastdiv(uint32_t(g.B));
  at.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  hipLaunchKernelGGL((conv_step_dw_kernel<T, KH, KW>),
                     dim3(grid_for(g.out_frame_elems(), kDwStepBlock)), dim3(kDwStepBlock), 0, s, g,
                     static_cast<const T*>(io.x), io.x_bc, static_cast<T*>(io.y), io.y_bc,
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

// ---- persistent forward_steps -------------------------------------------
//
// A clip of `count` frames in one launch (temporal stride 1 and dilation 1):
// the thread of output element (b, c, i, j) keeps the channel's kT stencils
// and the kT - 1 partial sums of its live outputs in registers for the whole
// clip.  The float32 ring is read once at the start and written back once at
// the end (not at all when the state is not to be updated), so per frame
// only the frame's stencil is read and the completed output written.
//
// Register acc[q] holds output tau = v - (KT - 1) + q, where v = n + pT is
// the virtual time of the arriving frame n; tap j feeds acc[KT - 1 - j].  The
// tap actions are those of the host schedule: an output's first tap on a
// real frame starts it, later taps add, tap kT - 1 completes it (section
// 3.1, Principles 3-5).
struct DwSteps {
  int32_t v0;       // virtual time n0 + pT of the first frame, capped at 2^29 (the
                    // schedule only depends on it near the start of a stream)
  int32_t slot0;    // ring slot of output v0 - (kT - 1): (n0 + pT - kT + 1) mod kT
  int32_t count;    // frames: T real, then end padding (zero frames)
  int32_t T;
  int32_t k0;       // output frame index of the call's first frame: n0 - max(n0, d)
  int32_t update;   // write the live partial sums back
  int32_t x_bytes, y_bytes;  // buffer extents from the clip pointers
  FastDiv fd_So, fd_Cout, fd_Wo, fd_W;
};

constexpr int PF = 4;  // frames in flight per thread

template <typename T, int KH, int KW, int KT>
__global__ __launch_bounds__(kBlock) void conv_steps_dw_kernel(
    ConvGeom g, DwSteps ds, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y,
    int64_t y_bc, const float* __restrict__ w, const float* __restrict__ bias,
    float* __restrict__ ring, int64_t ring_slot) {
  constexpr int NS = KH * KW;
  constexpr uint32_t esz = sizeof(T);
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.Cout * So;
  const int32_t idx = int32_t(blockIdx.x) * kBlock + int32_t(threadIdx.x);
  if (idx >= total) return;
  const int32_t bc = fdiv(idx, ds.fd_So);
  const int32_t p = idx - bc * So;
  const int32_t bq = fdiv(bc, ds.fd_Cout);
  const int32_t c = bc - bq * g.Cout;
  const int32_t i = fdiv(p, ds.fd_Wo), jo = p - i * g.Wo;
  const int32_t ridx = (c * g.B + bq) * So + p;  // ring (slot, C, B, Ho, Wo)

  float wr[KT][NS];
#pragma unroll
  for (int j = 0; j < KT; ++j)
#pragma unroll
    for (int e = 0; e < NS; ++e) wr[j][e] = w[(c * KT + j) * NS + e];
  const float bo = bias[c];

  // live partial sums at the start: outputs v0 - KT + 1 .. v0 - 1, in ring
  // slots slot0, slot0 + 1, ... (mod KT)
  float acc[KT];
#pragma unroll
  for (int q = 0; q < KT; ++q) {
    const int tau = ds.v0 - (KT - 1) + q;
    const int sl = (ds.slot0 + q) % KT;
    acc[q] = (q < KT - 1 && tau >= 0) ? ring[sl * ring_slot + ridx] : 0.f;
  }

  // stencil byte offsets inside the (b, c) plane of a frame; out-of-frame
  // taps read an out-of-range offset (zero)
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ds.x_bytes);
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, ds.y_bytes);
  const uint32_t plane = uint32_t(bc) * uint32_t(x_bc) * esz;
  int32_t soff[NS];
#pragma unroll
  for (int u = 0; u < KH; ++u) {
    const int32_t hi = i * g.sH + u * g.dH - g.pH;
#pragma unroll
    for (int v = 0; v < KW; ++v) {
      const int32_t wi = jo * g.sW + v * g.dW - g.pW;
      const bool in = hi >= 0 && hi < g.H && wi >= 0 && wi < g.W;
      soff[u * KW + v] = in ? int(plane + uint32_t(hi * g.W + wi) * esz) : kOutOfRange;
    }
  }
  const int32_t fstride = g.H * g.W * int32_t(esz);  // bytes between frames
  const int32_t yoff = int32_t((uint32_t(bc) * uint32_t(y_bc) + uint32_t(p)) * esz);

  // the stencil of frame t, zero for end-padding frames (t >= T); the frame
  // offset is wave-uniform and always inside the clip, out-of-frame taps
  // carry the out-of-range offset in their per-lane part
  auto load_frame = [&](int t, uint32_t (&xv)[NS]) {
    if (t < ds.T) {
#pragma unroll
      for (int e = 0; e < NS; ++e) xv[e] = load_raw_at<T>(xr, soff[e], t * fstride);
    } else {
#pragma unroll
      for (int e = 0; e < NS; ++e) xv[e] = 0u;
    }
  };
  // frame t's stencil sits in register set t % PF; the next PF - 1 frames'
  // are in flight while frame t is evaluated
  uint32_t xq[PF][NS];  // raw bits, converted when the frame is evaluated
#pragma unroll
  for (int u = 0; u < PF; ++u) load_frame(u, xq[u]);
  for (int t0 = 0; t0 < ds.count; t0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int t = t0 + u;
      if (t >= ds.count) break;
      const int v = ds.v0 + t;
#pragma unroll
      for (int j = KT - 1; j >= 0; --j) {
        const int q = KT - 1 - j;
        const int tau = v - j;
        // output v - j exists once tau >= 0; no branch around the arithmetic
        // (the sums of a missing output are never stored or written back)
        const bool exists = tau >= 0;
        const int first = tau >= g.pT ? 0 : g.pT - tau;  // first tap on a real frame
        float a = (j == first) ? 0.f : acc[q];  // a start overwrites the slot
#pragma unroll
        for (int e = 0; e < NS; ++e) a = fmaf(wr[j][e], raw_to_f32<T>(xq[u][e]), a);
        if (j == KT - 1)
          store_at(yr, exists ? yoff : kOutOfRange,
                   exists ? (ds.k0 + t) * So * int32_t(esz) : 0, from_f32<T>(a + bo));
        else
          acc[q] = a;
      }
      // the oldest output is complete: shift the others down one place
#pragma unroll
      for (int q = 0; q + 1 < KT; ++q) acc[q] = acc[q + 1];
      load_frame(t + PF, xq[u]);
    }
  }
  if (ds.update) {
    // live outputs after the clip: v1 - KT + 1 .. v1 - 1, slots continuing
    // from slot0 + count
    const int v1 = ds.v0 + ds.count;
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) {
      const int tau = v1 - (KT - 1) + q;
      const int sl = (ds.slot0 + ds.count + q) % KT;
      if (tau >= 0) ring[sl * ring_slot + ridx] = acc[q];
    }
  }
}

// Small planes (H * W <= 64 and Ho * Wo <= 64): one wave per (stream,
// channel) plane, one lane per input pixel and per output pixel.  Each frame
// is written, as float, into a zero-haloed tile of LDS, so every stencil tap
// is one LDS read at a lane address fixed for the whole clip plus a
// compile-time slot offset: no bounds test per tap, no address arithmetic per
// frame.  The channel's weights are wave-uniform (scalar registers).  Frames
// go in groups of U: while a group is evaluated from its U slots, the next
// group's pixels are in flight in registers.  Groups whose frames all take
// every tap on a real output (past a stream's start) skip the start and
// existence tests.  Each
// wave owns its slots, and LDS operations of a wave complete in program
// order, so only the compiler is kept from reordering them (no barrier).
// Taps, partial sums and summation order are those of the thread-per-output
// kernel above.
constexpr int kDwpWaves = 4;    // planes per workgroup (independent waves)
constexpr int kDwpSlot = 128;   // floats per frame slot: padded tile + one sink cell

struct DwpArgs {
  int32_t PW;         // padded tile width: W + 2 pW
  int32_t frame_bytes;  // input frame, bytes (frames of a plane are contiguous)
};

__device__ __forceinline__ void lds_order() { __asm__ volatile("" ::: "memory"); }

template <typename T, int KH, int KW, int KT>
__global__ __launch_bounds__(64 * kDwpWaves) void conv_steps_dwp_kernel(
    ConvGeom g, DwSteps ds, DwpArgs pa, const T* __restrict__ x, int64_t x_bc,
    T* __restrict__ y, int64_t y_bc, const float* __restrict__ w,
    const float* __restrict__ bias, float* __restrict__ ring, int64_t ring_slot) {
  constexpr int NS = KH * KW;
  constexpr int U = KT * ((4 + KT - 1) / KT);  // frames per group (acc names cycle)
  constexpr uint32_t esz = sizeof(T);
  __shared__ float lds[kDwpWaves][U][kDwpSlot];
  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int bc = int(blockIdx.x) * kDwpWaves + wave;
  if (bc >= g.B * g.Cout) return;  // whole waves; no workgroup barrier below
  const int S = g.H * g.W, So = g.Ho * g.Wo;
  const int bq = fdiv(bc, ds.fd_Cout), c = bc - bq * g.Cout;
  float(*sl)[kDwpSlot] = lds[wave];

  // zero the tiles once: halo cells are never written again
  for (int e = lane; e < U * kDwpSlot; e += 64) (&sl[0][0])[e] = 0.f;

  // input lane: pixel `lane` of the frame into its padded cell (lanes past
  // the frame load zero into the sink cell after the tile)
  const bool in_px = lane < S;
  int wpos = kDwpSlot - 1;
  if (in_px) {
    const int hp = fdiv(lane, ds.fd_W);
    wpos = (hp + g.pH) * pa.PW + (lane - hp * g.W) + g.pW;
  }
  float* const wp = &sl[0][wpos];  // + u * kDwpSlot: slot u
  const int plane = int(uint32_t(bc) * uint32_t(x_bc) * esz);
  const int xin = in_px ? plane + lane * int(esz) : kOutOfRange;
  // output lane: its stencil cells in the padded tile
  const bool pl = lane < So;
  const int p = pl ? lane : 0;
  const int i = fdiv(p, ds.fd_Wo), jo = p - i * g.Wo;
  const float* rp[NS];  // + u * kDwpSlot: slot u
#pragma unroll
  for (int u = 0; u < KH; ++u)
#pragma unroll
    for (int v = 0; v < KW; ++v)
      rp[u * KW + v] = &sl[0][(i * g.sH + u * g.dH) * pa.PW + jo * g.sW + v * g.dW];
  const int yo = pl ? int((uint32_t(bc) * uint32_t(y_bc) + uint32_t(p)) * esz) : kOutOfRange;
  const int ridx = (c * g.B + bq) * So + p;

  float wr[KT][NS];
#pragma unroll
  for (int j = 0; j < KT; ++j)
#pragma unroll
    for (int e = 0; e < NS; ++e) wr[j][e] = w[(c * KT + j) * NS + e];
  const float bo = bias[c];
  float acc[KT];
#pragma unroll
  for (int q = 0; q < KT; ++q) {
    const int tau = ds.v0 - (KT - 1) + q;
    const int slq = (ds.slot0 + q) % KT;
    acc[q] = (pl && q < KT - 1 && tau >= 0) ? ring[slq * ring_slot + ridx] : 0.f;
  }

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ds.x_bytes);
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, ds.y_bytes);
  // raw bits of this lane's pixel of frame t (zero past the clip's real frames)
  auto load = [&](int t) {
    const bool real = t < ds.T;
    return load_raw_at<T>(xr, real ? xin : kOutOfRange, real ? t * pa.frame_bytes : 0);
  };
  // evaluate the frame held in slot u: every live output takes its tap, the
  // oldest completes (STEADY: all KT outputs exist and have started)
  auto eval = [&](int t, int u, bool steady) {
    float xv[NS];
#pragma unroll
    for (int e = 0; e < NS; ++e) xv[e] = rp[e][u * kDwpSlot];
    const int v = ds.v0 + t;
#pragma unroll
    for (int j = KT - 1; j >= 0; --j) {
      const int q = KT - 1 - j;
      const int tau = v - j;
      const int first = steady ? 0 : (tau >= g.pT ? 0 : g.pT - tau);
      float a = (j == first) ? 0.f : acc[q];
#pragma unroll
      for (int e = 0; e < NS; ++e) a = fmaf(wr[j][e], xv[e], a);
      if (j == KT - 1) {
        const bool exists = steady || tau >= 0;
        store_at(yr, exists ? yo : kOutOfRange, exists ? (ds.k0 + t) * So * int(esz) : 0,
                 from_f32<T>(a + bo));
      } else {
        acc[q] = a;
      }
    }
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) acc[q] = acc[q + 1];
  };
  // groups of U frames: the group's pixels go to slots 0..U-1, the next
  // group's loads are issued, then the group is evaluated; a group is steady
  // once its first frame is (then so are the rest)
  uint32_t xa[U];
#pragma unroll
  for (int u = 0; u < U; ++u) xa[u] = load(u);
  int t = 0;
  for (; t + U <= ds.count; t += U) {
    lds_order();
#pragma unroll
    for (int u = 0; u < U; ++u) wp[u * kDwpSlot] = raw_to_f32<T>(xa[u]);
    lds_order();
#pragma unroll
    for (int u = 0; u < U; ++u) xa[u] = load(t + U + u);
    if (ds.v0 + t - (KT - 1) >= g.pT) {
#pragma unroll
      for (int u = 0; u < U; ++u) eval(t + u, u, true);
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u) eval(t + u, u, false);
    }
  }
  // ragged tail: its frames are already in registers
  lds_order();
#pragma unroll
  for (int u = 0; u < U; ++u) wp[u * kDwpSlot] = raw_to_f32<T>(xa[u]);
  lds_order();
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (t + u >= ds.count) break;
    eval(t + u, u, false);
  }

  if (ds.update && pl) {
    const int v1 = ds.v0 + ds.count;
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) {
      const int tau = v1 - (KT - 1) + q;
      const int slq = (ds.slot0 + ds.count + q) % KT;
      if (tau >= 0) ring[slq * ring_slot + ridx] = acc[q];
    }
  }
}

// Temporal stride or dilation above 1 (Principle 5): which output a tap
// feeds, and whether it starts, continues or completes it, now depends on the
// frame.  The kernel follows the host's step plans (the ones the per-frame
// step launches take, packed as a PlanTable).  Each lane keeps the R partial sums of its pixel in LDS, where a
// slot chosen at run time costs no more than a fixed one; frames go through
// zero-haloed LDS tiles as in the kernel above.  Per tap the arithmetic is
// the step kernel's: from the ring value (ACC, EMIT) or zero, the 3x3 chain,
// then back to the slot or out with the bias.
constexpr int kDwgU = 4;  // frames per group

struct DwgArgs {
  PlanTable pt;
  int32_t PW;  // padded tile width
  int32_t frame_bytes;
};

template <typename T, int KH, int KW, int KT>
__global__ __launch_bounds__(64 * kDwpWaves) void conv_steps_dwg_kernel(
    ConvGeom g, DwSteps ds, DwgArgs ga, const T* __restrict__ x, int64_t x_bc,
    T* __restrict__ y, int64_t y_bc, const float* __restrict__ w,
    const float* __restrict__ bias, float* __restrict__ ring, int64_t ring_slot) {
  constexpr int NS = KH * KW;
  constexpr int U = kDwgU;
  constexpr uint32_t esz = sizeof(T);
  __shared__ float lds[kDwpWaves][U][kDwpSlot];
  __shared__ float parts[kDwpWaves][kPlanMaxR][64];
  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int bc = int(blockIdx.x) * kDwpWaves + wave;
  if (bc >= g.B * g.Cout) return;  // whole waves; no workgroup barrier below
  const int S = g.H * g.W, So = g.Ho * g.Wo;
  const int bq = fdiv(bc, ds.fd_Cout), c = bc - bq * g.Cout;
  float(*sl)[kDwpSlot] = lds[wave];
  float* const pp = &parts[wave][0][lane];  // + slot * 64

  for (int e = lane; e < U * kDwpSlot; e += 64) (&sl[0][0])[e] = 0.f;  // halos stay zero

  const bool in_px = lane < S;
  int wpos = kDwpSlot - 1;
  if (in_px) {
    const int hp = fdiv(lane, ds.fd_W);
    wpos = (hp + g.pH) * ga.PW + (lane - hp * g.W) + g.pW;
  }
  float* const wp = &sl[0][wpos];
  const int plane = int(uint32_t(bc) * uint32_t(x_bc) * esz);
  const int xin = in_px ? plane + lane * int(esz) : kOutOfRange;
  const bool pl = lane < So;
  const int p = pl ? lane : 0;
  const int i = fdiv(p, ds.fd_Wo), jo = p - i * g.Wo;
  const float* rp[NS];
#pragma unroll
  for (int u = 0; u < KH; ++u)
#pragma unroll
    for (int v = 0; v < KW; ++v)
      rp[u * KW + v] = &sl[0][(i * g.sH + u * g.dH) * ga.PW + jo * g.sW + v * g.dW];
  const int yo = pl ? int((uint32_t(bc) * uint32_t(y_bc) + uint32_t(p)) * esz) : kOutOfRange;
  const int ridx = (c * g.B + bq) * So + p;

  float wr[KT][NS];
#pragma unroll
  for (int j = 0; j < KT; ++j)
#pragma unroll
    for (int e = 0; e < NS; ++e) wr[j][e] = w[(c * KT + j) * NS + e];
  const float bo = bias[c];
  // the ring's R slots of this pixel, live or not (stale slots go back as read)
  for (int q = 0; q < g.R; ++q) pp[q * 64] = pl ? ring[q * ring_slot + ridx] : 0.f;

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ds.x_bytes);
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, ds.y_bytes);
  auto load = [&](int t) {
    const bool real = t < ds.T;
    return load_raw_at<T>(xr, real ? xin : kOutOfRange, real ? t * ga.frame_bytes : 0);
  };
  int k = 0;          // outputs emitted so far in the call
  int ph = 0;         // phase of the next periodic frame
  auto eval = [&](int t, int u) {
    uint64_t code;
    if (t < ga.pt.n_start) {
      code = ga.pt.code_start[t];
    } else {
      code = ga.pt.code_period[ph];
      ph = ph + 1 == ga.pt.period ? 0 : ph + 1;
    }
    float xv[NS];
#pragma unroll
    for (int e = 0; e < NS; ++e) xv[e] = rp[e][u * kDwpSlot];
    bool emitted = false;
#pragma unroll
    for (int j = KT - 1; j >= 0; --j) {
      const int act = int(code >> (6 * j)) & 7, slot = int(code >> (6 * j + 3)) & 7;
      if (act == CO_TAP_NONE) continue;  // uniform
      float a = (act == CO_TAP_ACC || act == CO_TAP_EMIT) ? pp[slot * 64] : 0.f;
#pragma unroll
      for (int e = 0; e < NS; ++e) a = fmaf(wr[j][e], xv[e], a);
      if (act == CO_TAP_EMIT || act == CO_TAP_EMIT_FRESH) {
        store_at(yr, yo, k * So * int(esz), from_f32<T>(a + bo));
        emitted = true;
      } else {
        pp[slot * 64] = a;
      }
    }
    if (emitted) ++k;
  };

  uint32_t xa[U];
#pragma unroll
  for (int u = 0; u < U; ++u) xa[u] = load(u);
  for (int t = 0; t < ds.count; t += U) {
    lds_order();
#pragma unroll
    for (int u = 0; u < U; ++u) wp[u * kDwpSlot] = raw_to_f32<T>(xa[u]);
    lds_order();
#pragma unroll
    for (int u = 0; u < U; ++u) xa[u] = load(t + U + u);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (t + u >= ds.count) break;  // (the clip's last, ragged group)
      eval(t + u, u);
    }
    lds_order();
  }
  if (ds.update && pl)
    for (int q = 0; q < g.R; ++q) ring[q * ring_slot + ridx] = pp[q * 64];
}

// The small-plane kernel's conditions: one lane per input and per output
// pixel, the padded tile and its sink cell within a slot.
bool dwp_fits(const ConvGeom& g) {
  return g.S() <= 64 && g.So() <= 64 &&
         int64_t(g.H + 2 * g.pH) * (g.W + 2 * g.pW) + 1 <= kDwpSlot;
}

template <typename T, int KH, int KW, int KT>
hipError_t dw_steps_launch(const ConvGeom& g, const ConvLayout& L, char* state, const void* x,
                           int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                           int64_t n0, bool update, hipStream_t s) {
  DwSteps ds;
  const int64_t v0 = n0 + g.pT;
  ds.v0 = int32_t(v0 < (int64_t(1) << 29) ? v0 : (int64_t(1) << 29));
  ds.slot0 = int32_t(((v0 - (g.kT - 1)) % g.kT + g.kT) % g.kT);
  ds.count = count;
  ds.T = nreal;
  // output frame of step n: n - max(n0, d) (valid only for emitting steps)
  ds.k0 = int32_t(n0 - (n0 > g.d ? n0 : g.d));
  ds.update = update ? 1 : 0;
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  ds.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * x_bc + int64_t(nreal) * g.S()) * esz);
  ds.y_bytes = int32_t(((int64_t(g.B) * g.Cout - 1) * y_bc + y_bc) * esz);
  ds.fd_So = make_fastdiv(uint32_t(g.So()));
  ds.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  ds.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  ds.fd_W = make_fastdiv(uint32_t(g.W));
  const int64_t fbytes = g.S() * esz;
  if (g.sT != 1 || g.dT != 1) {
    // step plans: explicit for the call's frames in the stream's first
    // (kT - 1) dT steps, then one period of sT R steps
    DwgArgs ga{};
    plan_table(g, n0, count, &ga.pt);
    ga.PW = g.W + 2 * g.pW;
    ga.frame_bytes = int32_t(fbytes);
    hipLaunchKernelGGL((conv_steps_dwg_kernel<T, KH, KW, KT>),
                       dim3(unsigned((int64_t(g.B) * g.Cout + kDwpWaves - 1) / kDwpWaves)),
                       dim3(64 * kDwpWaves), 0, s, g, ds, ga, static_cast<const T*>(x), x_bc,
                       static_cast<T*>(y), y_bc, reinterpret_cast<const float*>(state + L.weight),
                       reinterpret_cast<const float*>(state + L.bias),
                       reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems);
    return hipGetLastError();
  }
  if (dwp_fits(g)) {
    DwpArgs pa;
    pa.PW = g.W + 2 * g.pW;
    pa.frame_bytes = int32_t(fbytes);
    const int64_t planes = int64_t(g.B) * g.Cout;
    hipLaunchKernelGGL((conv_steps_dwp_kernel<T, KH, KW, KT>),
                       dim3(unsigned((planes + kDwpWaves - 1) / kDwpWaves)), dim3(64 * kDwpWaves),
                       0, s, g, ds, pa, static_cast<const T*>(x), x_bc, static_cast<T*>(y), y_bc,
                       reinterpret_cast<const float*>(state + L.weight),
                       reinterpret_cast<const float*>(state + L.bias),
                       reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((conv_steps_dw_kernel<T, KH, KW, KT>), dim3(grid_for(g.out_frame_elems())),
                     dim3(kBlock), 0, s, g, ds, static_cast<const T*>(x), x_bc,
                     static_cast<T*>(y), y_bc, reinterpret_cast<const float*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems);
  return hipGetLastError();
}

template <typename T, int KH, int KW>
hipError_t dw_steps_kt(const ConvGeom& g, const ConvLayout& L, char* state, const void* x,
                       int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc, int64_t n0,
                       bool update, hipStream_t s) {
  switch (g.kT) {
    case 1: return dw_steps_launch<T, KH, KW, 1>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 2: return dw_steps_launch<T, KH, KW, 2>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 3: return dw_steps_launch<T, KH, KW, 3>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 4: return dw_steps_launch<T, KH, KW, 4>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 5: return dw_steps_launch<T, KH, KW, 5>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t dw_steps_dispatch(const ConvGeom& g, const ConvLayout& L, char* state, const void* x,
                             int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                             int64_t n0, bool update, hipStream_t s) {
  if (g.kH == 3 && g.kW == 3)
    return dw_steps_kt<T, 3, 3>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  if (g.kH == 1 && g.kW == 1)
    return dw_steps_kt<T, 1, 1>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_conv_step_depthwise(const ConvGeom& g, const ConvLayout& L, char* state,
                                      const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  // The stencil loads use 32-bit buffer offsets over everything reachable
  // from the frame pointer; a frame of a clip whose planes lie further apart
  // (forward_steps over a clip of 2^31 bytes or more) takes the direct
  // kernel, which shares the ring layout and the weight packing.
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  if (((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * esz >= (int64_t(1) << 31))
    return launch_conv_step_direct(g, L, state, io, plan, false, s);
  if (g.dtype == CO_BF16) return dw_dispatch<bf16_t>(g, L, state, io, plan, s);
  return dw_dispatch<float>(g, L, state, io, plan, s);
}

}  // namespace coinf

namespace coinf {

bool dw_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames) {
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  const bool fits = int64_t(g.B) * g.Cin * x_frames * g.S() * esz < (int64_t(1) << 31) &&
                    int64_t(g.B) * g.Cout * y_frames * g.So() * esz < (int64_t(1) << 31);
  // temporal stride or dilation above 1: the plan-driven small-plane kernel
  const bool strided = g.sT != 1 || g.dT != 1;
  const bool general = dwp_fits(g) && plan_table_fits(g);
  return g.algo == CO_ALGO_DEPTHWISE && (!strided || general) && g.kT >= 1 && g.kT <= 5 &&
         ((g.kH == 3 && g.kW == 3) || (g.kH == 1 && g.kW == 1)) && fits;
}

hipError_t launch_conv_steps_depthwise(const ConvGeom& g, const ConvLayout& L, char* state,
                                       const void* x, int64_t x_bc, int32_t nreal, int32_t count,
                                       void* y, int64_t y_bc, int64_t n0, bool update,
                                       hipStream_t s) {
  if (g.dtype == CO_BF16)
    return dw_steps_dispatch<bf16_t>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  return dw_steps_dispatch<float>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
}

}  // namespace coinf
