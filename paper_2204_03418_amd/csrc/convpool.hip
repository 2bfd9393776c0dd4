// Fused step of a depthwise continual convolution and the continual pool
// that consumes its output, when the pool's spatial window is the whole
// output plane (the global average / maximum pooling that closes an X3D
// bottleneck; section 3.2 defines both modules, section 3.3 their chaining).
//
// One wave per (stream, channel) plane, one lane per output pixel.  Each lane
// evaluates its pixel's active taps exactly as the depthwise step kernel does
// (same stencil values, same ring reads, same chain of multiply-adds, same
// ring writes) and rounds the completed output to the io dtype.  When the
// convolution emits, the pool steps on that frame in the same launch: lane p
// holds window element p, the wave reduces it with the pool step kernel's
// lane tree, lane 0 stores it into the pool's FIFO, and when the pool emits
// the window's frames are reduced as the pool step kernel reduces them.  The
// intermediate frame never goes to memory, and the results equal the two
// separate steps bit for bit.
#include <math.h>

#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

constexpr int kCpWaves = 4;  // planes per workgroup

struct CpTaps {  // the convolution step's active taps, compacted
  int32_t n;
  int32_t tap[CO_MAX_TAPS];
  int32_t act[CO_MAX_TAPS];
  int32_t slot[CO_MAX_TAPS];
};

struct CpPool {  // the pool step's plan
  int32_t step;   // the pool steps (the convolution emitted)
  int32_t update;
  int32_t emit;
  int32_t write_slot;
  int32_t src[CO_MAX_TAPS];
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}

template <typename T, int KH, int KW>
__global__ __launch_bounds__(64 * kCpWaves) void convpool_step_kernel(
    ConvGeom g, const T* __restrict__ x, int64_t x_bc, const float* __restrict__ w,
    const float* __restrict__ bias, float* __restrict__ ring, int64_t ring_slot, CpTaps at,
    PoolGeom pg, T* __restrict__ z, int64_t z_bc, float* __restrict__ fifo, int64_t fifo_slot,
    float* __restrict__ valid, CpPool pp, FastDiv fd_Cout, FastDiv fd_Wo) {
  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  const int BC = g.B * g.Cout;
  const int bc = int(blockIdx.x) * kCpWaves + wave;
  if (bc >= BC) return;  // whole waves; no barrier follows
  const int So = g.Ho * g.Wo;
  const bool pl = lane < So;
  const int p = pl ? lane : 0;
  const int bq = fdiv(bc, fd_Cout), c = bc - bq * g.Cout;
  const int i = fdiv(p, fd_Wo), jo = p - i * g.Wo;
  const int ridx = (c * g.B + bq) * So + p;

  // the depthwise step (see conv_step_dw_kernel)
  // frame planes are x_bc elements apart (S for a single frame, T * S when
  // the frame is read in place from a clip)
  const int x_extent = int(((int64_t(g.B) * g.Cin - 1) * x_bc + g.H * g.W) * int64_t(sizeof(T)));
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, x_extent);
  const int plane = int(int64_t(bc) * x_bc);
  float xv[KH * KW];
#pragma unroll
  for (int u = 0; u < KH; ++u) {
    const int hi = i * g.sH + u * g.dH - g.pH;
#pragma unroll
    for (int v = 0; v < KW; ++v) {
      const int wi = jo * g.sW + v * g.dW - g.pW;
      const bool in = pl && hi >= 0 && hi < g.H && wi >= 0 && wi < g.W;
      xv[u * KW + v] = load_or_zero<T>(xr, plane + hi * g.W + wi, in);
    }
  }
  const float* wc = w + int64_t(c) * g.kT * (KH * KW);
  const float bo = bias[c];
  T yv = from_f32<T>(0.f);
  for (int a = 0; a < at.n; ++a) {
    const int act = at.act[a];
    float acc = 0.f;
    if (pl && (act == CO_TAP_ACC || act == CO_TAP_EMIT))
      acc = ring[int64_t(at.slot[a]) * ring_slot + ridx];
    const float* wj = wc + at.tap[a] * (KH * KW);
#pragma unroll
    for (int e = 0; e < KH * KW; ++e) acc = fmaf(wj[e], xv[e], acc);
    if (act == CO_TAP_START || act == CO_TAP_ACC) {
      if (pl) ring[int64_t(at.slot[a]) * ring_slot + ridx] = acc;
    } else {
      yv = from_f32<T>(acc + bo);
    }
  }
  if (!pp.step) return;

  // the pool step on the frame just completed (see pool_step_kernel): lane p
  // holds window element p of output (b, c)
  const bool is_max = pg.kind == CO_POOL_MAX;
  float val = is_max ? -INFINITY : 0.f;
  if (pl) val = is_max ? fmaxf(val, to_f32<T>(yv)) : val + to_f32<T>(yv);
  val = is_max ? wave_max(val) : wave_sum(val);
  if (pp.update && lane == 0) {
    fifo[int64_t(pp.write_slot) * fifo_slot + bc] = val;
    if (bc == 0) valid[pp.write_slot] = 1.f;
  }
  if (!pp.emit) return;
  float acc = is_max ? -INFINITY : 0.f;
  float tcount = 0.f;
  if (lane < pg.kT) {
    const int s = pp.src[lane];
    if (s != -1) {
      float ev, ok;
      if (s == -2) {
        ev = val;
        ok = 1.f;
      } else {
        ev = fifo[int64_t(s) * fifo_slot + bc];
        ok = valid[s];
      }
      acc = is_max ? fmaxf(acc, ev) : acc + ev;
      tcount += ok;
    }
  }
  if (is_max) {
    acc = wave_max(acc);
  } else {
    acc = wave_sum(acc);
    tcount = wave_sum(tcount);
  }
  if (lane != 0) return;
  float out;
  if (is_max) {
    out = acc;
  } else {
    const float div = pg.count_include_pad ? float(pg.kT * pg.kH * pg.kW)
                                           : tcount * float(pg.kH * pg.kW);
    out = div > 0.f ? acc / div : 0.f;
  }
  z[int64_t(bc) * z_bc] = from_f32<T>(out);
}

template <typename T, int KH, int KW>
hipError_t cp_launch(const ConvGeom& g, const ConvLayout& L, char* cstate, const PoolGeom& pg,
                     const PoolLayout& PL, char* pstate, const void* x, int64_t x_bc, void* z,
                     int64_t z_bc, const co_step_plan& cplan, const co_pool_plan* pplan,
                     bool update, hipStream_t s) {
  CpTaps at;
  at.n = 0;
  for (int j = 0; j < g.kT; ++j) {
    if (cplan.action[j] == CO_TAP_NONE) continue;
    at.tap[at.n] = j;
    at.act[at.n] = cplan.action[j];
    at.slot[at.n] = cplan.slot[j] < 0 ? 0 : cplan.slot[j];
    ++at.n;
  }
  CpPool pp{};
  pp.step = pplan ? 1 : 0;
  if (pplan) {
    pp.update = update ? 1 : 0;
    pp.emit = pplan->emit;
    pp.write_slot = pplan->write_slot;
    for (int t = 0; t < CO_MAX_TAPS; ++t) pp.src[t] = pplan->src[t];
  }
  if (at.n == 0 && !pp.step) return hipSuccess;
  const int64_t planes = int64_t(g.B) * g.Cout;
  hipLaunchKernelGGL((convpool_step_kernel<T, KH, KW>),
                     dim3(unsigned((planes + kCpWaves - 1) / kCpWaves)), dim3(64 * kCpWaves), 0,
                     s, g, static_cast<const T*>(x), x_bc,
                     reinterpret_cast<const float*>(cstate + L.weight),
                     reinterpret_cast<const float*>(cstate + L.bias),
                     reinterpret_cast<float*>(cstate + L.ring), L.ring_slot_elems, at, pg,
                     static_cast<T*>(z), z_bc, reinterpret_cast<float*>(pstate + PL.fifo),
                     PL.fifo_slot_elems, reinterpret_cast<float*>(pstate + PL.valid), pp,
                     make_fastdiv(uint32_t(g.Cout)), make_fastdiv(uint32_t(g.Wo)));
  return hipGetLastError();
}

template <typename T>
hipError_t cp_dispatch(const ConvGeom& g, const ConvLayout& L, char* cstate, const PoolGeom& pg,
                       const PoolLayout& PL, char* pstate, const void* x, int64_t x_bc, void* z,
                       int64_t z_bc, const co_step_plan& cplan, const co_pool_plan* pplan,
                       bool update, hipStream_t s) {
  if (g.kH == 3 && g.kW == 3)
    return cp_launch<T, 3, 3>(g, L, cstate, pg, PL, pstate, x, x_bc, z, z_bc, cplan, pplan,
                              update, s);
  if (g.kH == 1 && g.kW == 1)
    return cp_launch<T, 1, 1>(g, L, cstate, pg, PL, pstate, x, x_bc, z, z_bc, cplan, pplan,
                              update, s);
  return hipErrorInvalidValue;
}

}  // namespace

bool convpool_supported(const ConvGeom& g, const PoolGeom& pg) {
  const bool taps = (g.kH == 3 && g.kW == 3) || (g.kH == 1 && g.kW == 1);
  return g.algo == CO_ALGO_DEPTHWISE && taps && g.dtype == pg.dtype && g.B == pg.B &&
         g.Cout == pg.C && pg.H == g.Ho && pg.W == g.Wo && g.So() <= 64 && pg.kH == g.Ho &&
         pg.kW == g.Wo && pg.pH == 0 && pg.pW == 0 && pg.dH == 1 && pg.dW == 1 &&
         pg.Ho == 1 && pg.Wo == 1 && pg.kT <= 64 &&
         g.S() > 0;
}

hipError_t launch_convpool_step(const ConvGeom& g, const ConvLayout& L, char* cstate,
                                const PoolGeom& pg, const PoolLayout& PL, char* pstate,
                                const void* x, int64_t x_bc, void* z, int64_t z_bc,
                                const co_step_plan& cplan, const co_pool_plan* pplan, bool update,
                                hipStream_t s) {
  if (g.dtype == CO_BF16)
    return cp_dispatch<bf16_t>(g, L, cstate, pg, PL, pstate, x, x_bc, z, z_bc, cplan, pplan,
                               update, s);
  return cp_dispatch<float>(g, L, cstate, pg, PL, pstate, x, x_bc, z, z_bc, cplan, pplan, update,
                            s);
}

}  // namespace coinf
