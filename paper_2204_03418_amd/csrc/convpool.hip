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

// Planes per workgroup.  One wave per workgroup measures fastest (the
// X3D-style step 1.80 M -> 1.99 M stream-frames/s, the clip 7.20 M -> 7.46 M):
// each plane's wave is dispatched and retired on its own.
constexpr int kCpWaves = 1;

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

// The depthwise step of one lane (output pixel p of plane (stream, channel
// c), flat plane index bc, ring index ridx) from its stencil values xv, then
// the pool step on the completed frame (see the kernels below): shared by
// the fused kernels so that they give the separate steps' bits.
template <typename T, int KH, int KW>
__device__ __forceinline__ void dw_pool_tail(
    const float (&xv)[KH * KW], bool pl, int lane, int c, int bc, int ridx, const ConvGeom& g,
    const float* __restrict__ w, const float* __restrict__ bias, float* __restrict__ ring,
    int64_t ring_slot, const CpTaps& at, int act2, const PoolGeom& pg, T* __restrict__ z,
    int64_t z_bc, float* __restrict__ fifo, int64_t fifo_slot, float* __restrict__ valid,
    const CpPool& pp) {
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
  // an activation between the convolution and the pool applies to the
  // emitted (rounded) frame, as a separate elementwise step would
  if (act2 == CO_ACT_RELU) yv = from_f32<T>(fmaxf(to_f32<T>(yv), 0.f));
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
  dw_pool_tail<T, KH, KW>(xv, pl, lane, c, bc, ridx, g, w, bias, ring, ring_slot, at, CO_ACT_NONE,
                          pg, z, z_bc, fifo, fifo_slot, valid, pp);
}

// Fused step of an X3D-style bottleneck (sections 3.2-3.3: a pointwise
// convolution, batch normalisation and activation, a depthwise continual
// convolution, batch normalisation and activation, and the pool over the
// plane; the normalisations are folded into the convolutions' weights at
// init).  A workgroup owns kBnWaves channel planes of one stream.  The
// stream's input frame (C_in x H x W, at most 64 pixels per plane) is staged
// into LDS once; each wave computes its channel's pointwise output at every
// pixel (lane = pixel) exactly as the pointwise (1x1x1) direct step kernel
// does -- products accumulated over the input channels in order with fmaf
// from zero, the bias added, the result rounded to the io dtype and the
// activation applied -- and writes it into its own zero-haloed plane in LDS.
// The depthwise stencil then reads that plane instead of memory, and the
// depthwise and pool steps follow as in convpool_step_kernel.  The
// intermediate frames never leave the CU; the results equal the separate
// steps bit for bit.
constexpr int kBnWaves = 4;

template <typename T, int KH, int KW>
__global__ __launch_bounds__(64 * kBnWaves) void bneck_step_kernel(
    int32_t Ci, const T* __restrict__ x, int64_t x_bc, const float* __restrict__ w1,
    const float* __restrict__ b1, int32_t act1, ConvGeom g, const float* __restrict__ w,
    const float* __restrict__ bias, float* __restrict__ ring, int64_t ring_slot, CpTaps at,
    int32_t act2, PoolGeom pg, T* __restrict__ z, int64_t z_bc, float* __restrict__ fifo,
    int64_t fifo_slot, float* __restrict__ valid, CpPool pp, int32_t cblocks, FastDiv fd_S,
    FastDiv fd_W, FastDiv fd_Wo) {
  extern __shared__ float lds[];
  const int tid = int(threadIdx.x);
  const int lane = tid & 63, wave = tid >> 6;
  const int S = g.H * g.W;
  const int Hp = g.H + 2 * g.pH, Wp = g.W + 2 * g.pW;
  const int bq = int(blockIdx.x) / cblocks;
  const int cb = int(blockIdx.x) - bq * cblocks;
  float* xs = lds;                 // the stream's input frame, [C_in][S]
  float* zs = lds + Ci * S;        // kBnWaves zero-haloed planes of Hp x Wp
  float* zw = zs + wave * Hp * Wp;
  for (int e = tid; e < kBnWaves * Hp * Wp; e += 64 * kBnWaves) zs[e] = 0.f;
  for (int e = tid; e < Ci * S; e += 64 * kBnWaves) {
    const int ci = fdiv(e, fd_S), q = e - ci * S;
    xs[e] = to_f32<T>(x[(int64_t(bq) * Ci + ci) * x_bc + q]);
  }
  __syncthreads();
  const int c = cb * kBnWaves + wave;
  const bool cvalid = c < g.Cout;
  if (cvalid && lane < S) {
    const float* wr = w1 + int64_t(c) * Ci;
    float acc = 0.f;
    for (int ci = 0; ci < Ci; ++ci) acc = fmaf(wr[ci], xs[ci * S + lane], acc);
    T z1 = from_f32<T>(acc + b1[c]);
    if (act1 == CO_ACT_RELU) z1 = from_f32<T>(fmaxf(to_f32<T>(z1), 0.f));
    const int qi = fdiv(lane, fd_W), qj = lane - qi * g.W;
    zw[(qi + g.pH) * Wp + qj + g.pW] = to_f32<T>(z1);
  }
  __syncthreads();
  if (!cvalid) return;  // after the last barrier
  const int So = g.Ho * g.Wo;
  const bool pl = lane < So;
  const int p = pl ? lane : 0;
  const int i = fdiv(p, fd_Wo), jo = p - i * g.Wo;
  float xv[KH * KW];
#pragma unroll
  for (int u = 0; u < KH; ++u)
#pragma unroll
    for (int v = 0; v < KW; ++v)
      xv[u * KW + v] = pl ? zw[(i * g.sH + u * g.dH) * Wp + jo * g.sW + v * g.dW] : 0.f;
  const int bc = bq * g.Cout + c;
  const int ridx = (c * g.B + bq) * So + p;
  dw_pool_tail<T, KH, KW>(xv, pl, lane, c, bc, ridx, g, w, bias, ring, ring_slot, at, act2, pg,
                          z, z_bc, fifo, fifo_slot, valid, pp);
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

// A clip of `count` frames in one launch (temporal stride and dilation 1 in
// both modules).  One wave per (stream, channel) plane, as in the step kernel
// above, for the whole clip: the convolution's kT - 1 partial sums and the
// pool's last kT reduced frames stay in registers, so only the clip, the
// pooled outputs and the two states move through memory.
//
// The plane's frames are staged through LDS in blocks of kCpsF frames,
// widened to fp32 once and laid out as a zero-haloed padded plane with the
// block's frames of one position side by side: a stencil tap is then one
// 8-byte LDS read per two frames at an address fixed for the lane, with no
// bounds test and no conversion per use.  Block k + 1 is written to the
// other buffer while block k is evaluated, and block k + 2 is already in
// registers.  Arithmetic per frame is the step kernels': the same
// multiply-add chain per tap, the same rounding of the output, the same lane
// tree for the spatial window and the pool step's tap tree for the temporal
// one, so a clip gives the bits of stepping frame by frame.
constexpr int kCpsWaves = 1;  // planes per workgroup (as above)
constexpr int kCpsF = 8;           // frames per staged block
constexpr int kCpsG = 2;           // frames per LDS read of a tap
constexpr int kCpsMaxPadded = 128;  // padded plane, elements

struct CpSteps {
  int32_t v0;       // virtual time of the first frame: n0 + pT (clamped)
  int32_t slot0;    // ring slot of output v0 - (kT - 1)
  int32_t count;    // frames in the call
  int32_t update;
  int32_t x_bytes;  // bytes of the clip reachable from x
  int32_t fstride;  // bytes between consecutive frames of a plane
  int32_t Hp, Wp;   // padded input plane
  int32_t nblk;     // staged blocks: ceil(count / kCpsF)
  int32_t tfirst;   // first frame of the call whose convolution step emits
  int64_t n0p;      // pool steps before the call
  int64_t emit0p;   // first pool step of the call that emits: max(n0p, pool delay)
  FastDiv fd_Cout, fd_Wo, fd_W;
};

template <typename T, int KH, int KW, int KT, int PKT>
__global__ __launch_bounds__(64 * kCpsWaves) void convpool_steps_kernel(
    ConvGeom g, CpSteps cs, const T* __restrict__ x, int64_t x_bc, const float* __restrict__ w,
    const float* __restrict__ bias, float* __restrict__ ring, int64_t ring_slot, PoolGeom pg,
    T* __restrict__ z, int64_t z_bc, float* __restrict__ fifo, int64_t fifo_slot,
    const float* __restrict__ valid) {
  constexpr int NS = KH * KW;
  constexpr int F = kCpsF;
  constexpr uint32_t esz = sizeof(T);
  extern __shared__ float cps_lds[];  // [wave][buffer][padded position][frame]
  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int BC = g.B * g.Cout;
  const int bc_raw = int(blockIdx.x) * kCpsWaves + wave;
  const bool wlive = bc_raw < BC;  // whole waves; idle ones still meet the barriers
  const int bc = wlive ? bc_raw : 0;
  const int So = g.Ho * g.Wo;
  const bool pl = wlive && lane < So;
  const int p = lane < So ? lane : 0;
  const int bq = fdiv(bc, cs.fd_Cout), c = bc - bq * g.Cout;
  const int i = fdiv(p, cs.fd_Wo), jo = p - i * g.Wo;
  const int ridx = (c * g.B + bq) * So + p;
  const int buf_elems = cs.Hp * cs.Wp * F;
  float* wl = cps_lds + wave * 2 * buf_elems;
  for (int e = lane; e < 2 * buf_elems; e += 64) wl[e] = 0.f;  // the halo stays zero

  float wr[KT][NS];
#pragma unroll
  for (int j = 0; j < KT; ++j)
#pragma unroll
    for (int e = 0; e < NS; ++e) wr[j][e] = w[(c * KT + j) * NS + e];
  const float bo = bias[c];
  float acc[KT];
#pragma unroll
  for (int q = 0; q < KT; ++q) {
    const int tau = cs.v0 - (KT - 1) + q;
    const int sl = (cs.slot0 + q) % KT;
    acc[q] = (pl && q < KT - 1 && tau >= 0) ? ring[sl * ring_slot + ridx] : 0.f;
  }
  // stencil taps: padded positions of this lane's output pixel, times F
  int toff[NS];
#pragma unroll
  for (int u = 0; u < KH; ++u)
#pragma unroll
    for (int v = 0; v < KW; ++v)
      toff[u * KW + v] = ((i * g.sH + u * g.dH) * cs.Wp + (jo * g.sW + v * g.dW)) * F;

  // pool: reduced value and validity of pool frame m - (PKT - 1) + q before
  // the pool's step m; frames before the stream began are start padding
  const bool is_max = pg.kind == CO_POOL_MAX;
  const float neutral = is_max ? -INFINITY : 0.f;
  const int kHW = pg.kH * pg.kW;
  float fv[PKT], fok[PKT];
#pragma unroll
  for (int q = 0; q + 1 < PKT; ++q) {
    const int64_t rf = cs.n0p - (PKT - 1) + q;
    const bool have = wlive && rf >= 0;
    fv[q] = have ? fifo[(rf % PKT) * fifo_slot + bc] : neutral;
    fok[q] = have ? valid[rf % PKT] : 0.f;
  }

  // staging: lane e holds input element e of the plane (H * W <= 64)
  const int h_in = fdiv(lane, cs.fd_W), w_in = lane - h_in * g.W;
  const int spos = (wlive && lane < g.H * g.W) ? ((h_in + g.pH) * cs.Wp + w_in + g.pW) * F : -1;
  const int sbyte = int((uint32_t(bc) * uint32_t(x_bc) + uint32_t(lane)) * esz);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, cs.x_bytes);
  uint32_t raw[F];
  auto fetch = [&](int blk) {
#pragma unroll
    for (int f = 0; f < F; ++f) {
      const int t = blk * F + f;
      raw[f] = 0u;
      if (spos >= 0 && t < cs.count) raw[f] = load_raw_at<T>(xr, sbyte, t * cs.fstride);
    }
  };
  auto stash = [&](int buf) {
    if (spos < 0) return;
    float4* dst = reinterpret_cast<float4*>(wl + buf * buf_elems + spos);
#pragma unroll
    for (int f4 = 0; f4 < F / 4; ++f4)
      dst[f4] = make_float4(raw_to_f32<T>(raw[4 * f4]), raw_to_f32<T>(raw[4 * f4 + 1]),
                            raw_to_f32<T>(raw[4 * f4 + 2]), raw_to_f32<T>(raw[4 * f4 + 3]));
  };

  __syncthreads();  // the zero fill before the first block lands
  fetch(0);
  stash(0);
  if (cs.nblk > 1) fetch(1);
  __syncthreads();
  for (int k = 0; k < cs.nblk; ++k) {
    const float* fb = wl + (k & 1) * buf_elems;
#pragma unroll
    for (int h2 = 0; h2 < F / kCpsG; ++h2) {
      if (k * F + kCpsG * h2 >= cs.count) break;  // uniform
      float2 xq[NS];
#pragma unroll
      for (int e = 0; e < NS; ++e)
        xq[e] = *reinterpret_cast<const float2*>(fb + toff[e] + kCpsG * h2);
#pragma unroll
      for (int ff = 0; ff < kCpsG; ++ff) {
        const int t = k * F + kCpsG * h2 + ff;
        if (t >= cs.count) break;  // uniform
        float xv[NS];
#pragma unroll
        for (int e = 0; e < NS; ++e) xv[e] = ff == 0 ? xq[e].x : xq[e].y;
        const int v = cs.v0 + t;
#pragma unroll
        for (int j = KT - 1; j >= 0; --j) {
          const int q = KT - 1 - j;
          const int tau = v - j;
          if (tau < 0) continue;
          const int first = tau >= g.pT ? 0 : g.pT - tau;
          float a = (j == first) ? 0.f : acc[q];
#pragma unroll
          for (int e = 0; e < NS; ++e) a = fmaf(wr[j][e], xv[e], a);
          if (j != KT - 1) {
            acc[q] = a;
            continue;
          }
          // the convolution emits: the pool steps on the rounded frame
          const T yv = from_f32<T>(a + bo);
          float val = neutral;
          if (pl) val = is_max ? fmaxf(val, to_f32<T>(yv)) : val + to_f32<T>(yv);
#pragma unroll
          for (int m = 32; m > 0; m >>= 1) {
            const float o = __shfl_xor(val, m, 64);
            val = is_max ? fmaxf(val, o) : val + o;
          }
          val = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(val), 0));
          fv[PKT - 1] = val;
          fok[PKT - 1] = 1.f;
          const int64_t m = cs.n0p + (t - cs.tfirst);
          if (m >= pg.d) {
            float tv[8], tc[8];
#pragma unroll
            for (int l = 0; l < 8; ++l) {
              const bool in = l < PKT && m - (PKT - 1) + l >= 0;
              tv[l] = in ? fv[l < PKT ? l : 0] : neutral;
              tc[l] = in ? fok[l < PKT ? l : 0] : 0.f;
            }
#pragma unroll
            for (int mm = 4; mm > 0; mm >>= 1) {
              float nv[8], nc[8];
#pragma unroll
              for (int l = 0; l < 8; ++l) {
                nv[l] = is_max ? fmaxf(tv[l], tv[l ^ mm]) : tv[l] + tv[l ^ mm];
                nc[l] = tc[l] + tc[l ^ mm];
              }
#pragma unroll
              for (int l = 0; l < 8; ++l) {
                tv[l] = nv[l];
                tc[l] = nc[l];
              }
            }
            float out;
            if (is_max) {
              out = tv[0];
            } else {
              const float div = pg.count_include_pad ? float(PKT * kHW) : tc[0] * float(kHW);
              out = div > 0.f ? tv[0] / div : 0.f;
            }
            if (wlive && lane == 0) z[int64_t(bc) * z_bc + (m - cs.emit0p)] = from_f32<T>(out);
          }
#pragma unroll
          for (int q2 = 0; q2 + 1 < PKT; ++q2) {
            fv[q2] = fv[q2 + 1];
            fok[q2] = fok[q2 + 1];
          }
        }
#pragma unroll
        for (int q = 0; q + 1 < KT; ++q) acc[q] = acc[q + 1];
      }
    }
    if (k + 1 < cs.nblk) {
      // block k + 1 into the buffer block k - 1 used (every wave left it at
      // the last barrier), then block k + 2 into registers
      stash((k + 1) & 1);
      if (k + 2 < cs.nblk) fetch(k + 2);
    }
    __syncthreads();
  }
  if (!cs.update) return;
  if (pl) {
    const int v1 = cs.v0 + cs.count;
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) {
      const int tau = v1 - (KT - 1) + q;
      const int sl = (cs.slot0 + cs.count + q) % KT;
      if (tau >= 0) ring[sl * ring_slot + ridx] = acc[q];
    }
  }
  if (wlive && lane == 0) {
    const int64_t n1p = cs.n0p + (cs.count > cs.tfirst ? cs.count - cs.tfirst : 0);
#pragma unroll
    for (int q = 0; q + 1 < PKT; ++q) {
      const int64_t rf = n1p - (PKT - 1) + q;
      if (rf >= 0) fifo[(rf % PKT) * fifo_slot + bc] = fv[q];
    }
  }
}

template <typename T, int KH, int KW, int KT, int PKT>
hipError_t cps_launch(const ConvGeom& g, const ConvLayout& L, char* cstate, const PoolGeom& pg,
                      const PoolLayout& PL, char* pstate, const void* x, int32_t T_in, void* z,
                      int64_t z_cap, int64_t n0c, int64_t n0p, bool update, hipStream_t s) {
  CpSteps cs;
  const int64_t v0 = n0c + g.pT;
  cs.v0 = int32_t(v0 < (int64_t(1) << 29) ? v0 : (int64_t(1) << 29));
  cs.slot0 = int32_t(((v0 - (g.kT - 1)) % g.kT + g.kT) % g.kT);
  cs.count = T_in;
  cs.update = update ? 1 : 0;
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  const int64_t x_bc = int64_t(T_in) * g.S();
  cs.x_bytes = int32_t(int64_t(g.B) * g.Cin * x_bc * esz);
  cs.fstride = int32_t(g.S() * esz);
  cs.Hp = g.H + 2 * g.pH;
  cs.Wp = g.W + 2 * g.pW;
  cs.nblk = (T_in + kCpsF - 1) / kCpsF;
  const int64_t tf = int64_t(g.kT - 1) - v0;
  cs.tfirst = int32_t(tf > 0 ? tf : 0);
  cs.n0p = n0p;
  cs.emit0p = n0p > pg.d ? n0p : pg.d;
  cs.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  cs.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  cs.fd_W = make_fastdiv(uint32_t(g.W));
  const int64_t planes = int64_t(g.B) * g.Cout;
  const size_t lds = size_t(kCpsWaves) * 2 * cs.Hp * cs.Wp * kCpsF * sizeof(float);
  float* valid = reinterpret_cast<float*>(pstate + PL.valid);
  hipLaunchKernelGGL((convpool_steps_kernel<T, KH, KW, KT, PKT>),
                     dim3(unsigned((planes + kCpsWaves - 1) / kCpsWaves)), dim3(64 * kCpsWaves),
                     lds, s, g, cs, static_cast<const T*>(x), x_bc,
                     reinterpret_cast<const float*>(cstate + L.weight),
                     reinterpret_cast<const float*>(cstate + L.bias),
                     reinterpret_cast<float*>(cstate + L.ring), L.ring_slot_elems, pg,
                     static_cast<T*>(z), z_cap, reinterpret_cast<float*>(pstate + PL.fifo),
                     PL.fifo_slot_elems, valid);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !update) return e;
  const int32_t n_pool = T_in > cs.tfirst ? T_in - cs.tfirst : 0;
  return launch_pool_valid(valid, pg.R, n0p, n_pool, n_pool, s);
}

template <typename T, int KH, int KW, int KT>
hipError_t cps_pkt(const ConvGeom& g, const ConvLayout& L, char* cstate, const PoolGeom& pg,
                   const PoolLayout& PL, char* pstate, const void* x, int32_t T_in, void* z,
                   int64_t z_cap, int64_t n0c, int64_t n0p, bool update, hipStream_t s) {
  switch (pg.kT) {
#define CO_CPS_CASE(P)                                                                        \
    case P:                                                                                   \
      return cps_launch<T, KH, KW, KT, P>(g, L, cstate, pg, PL, pstate, x, T_in, z, z_cap,    \
                                          n0c, n0p, update, s);
    CO_CPS_CASE(1) CO_CPS_CASE(2) CO_CPS_CASE(3) CO_CPS_CASE(4) CO_CPS_CASE(5)
#undef CO_CPS_CASE
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int KH, int KW>
hipError_t cps_kt(const ConvGeom& g, const ConvLayout& L, char* cstate, const PoolGeom& pg,
                  const PoolLayout& PL, char* pstate, const void* x, int32_t T_in, void* z,
                  int64_t z_cap, int64_t n0c, int64_t n0p, bool update, hipStream_t s) {
  switch (g.kT) {
#define CO_CPS_CASE(K)                                                                        \
    case K:                                                                                   \
      return cps_pkt<T, KH, KW, K>(g, L, cstate, pg, PL, pstate, x, T_in, z, z_cap, n0c, n0p, \
                                   update, s);
    CO_CPS_CASE(1) CO_CPS_CASE(2) CO_CPS_CASE(3) CO_CPS_CASE(4) CO_CPS_CASE(5)
#undef CO_CPS_CASE
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t cps_dispatch(const ConvGeom& g, const ConvLayout& L, char* cstate, const PoolGeom& pg,
                        const PoolLayout& PL, char* pstate, const void* x, int32_t T_in, void* z,
                        int64_t z_cap, int64_t n0c, int64_t n0p, bool update, hipStream_t s) {
  if (g.kH == 3 && g.kW == 3)
    return cps_kt<T, 3, 3>(g, L, cstate, pg, PL, pstate, x, T_in, z, z_cap, n0c, n0p, update, s);
  if (g.kH == 1 && g.kW == 1)
    return cps_kt<T, 1, 1>(g, L, cstate, pg, PL, pstate, x, T_in, z, z_cap, n0c, n0p, update, s);
  return hipErrorInvalidValue;
}

}  // namespace

namespace {

// The plans of one fused step, as cp_launch builds them.
void cp_plans(const ConvGeom& g, const co_step_plan& cplan, const co_pool_plan* pplan,
              bool update, CpTaps* at, CpPool* pp) {
  at->n = 0;
  for (int j = 0; j < g.kT; ++j) {
    if (cplan.action[j] == CO_TAP_NONE) continue;
    at->tap[at->n] = j;
    at->act[at->n] = cplan.action[j];
    at->slot[at->n] = cplan.slot[j] < 0 ? 0 : cplan.slot[j];
    ++at->n;
  }
  *pp = CpPool{};
  pp->step = pplan ? 1 : 0;
  if (pplan) {
    pp->update = update ? 1 : 0;
    pp->emit = pplan->emit;
    pp->write_slot = pplan->write_slot;
    for (int t = 0; t < CO_MAX_TAPS; ++t) pp->src[t] = pplan->src[t];
  }
}

template <typename T, int KH, int KW>
hipError_t bn_launch(const ConvGeom& pw, const ConvLayout& PWL, char* pwstate, int32_t act1,
                     const ConvGeom& g, const ConvLayout& L, char* cstate, int32_t act2,
                     const PoolGeom& pg, const PoolLayout& PL, char* pstate, const void* x,
                     int64_t x_bc, void* z, int64_t z_bc, const co_step_plan& cplan,
                     const co_pool_plan* pplan, bool update, hipStream_t s) {
  CpTaps at;
  CpPool pp;
  cp_plans(g, cplan, pplan, update, &at, &pp);
  if (at.n == 0 && !pp.step) return hipSuccess;
  const int32_t cblocks = int32_t((g.Cout + kBnWaves - 1) / kBnWaves);
  const int S = g.H * g.W;
  const size_t lds = size_t(pw.Cin * S + kBnWaves * (g.H + 2 * g.pH) * (g.W + 2 * g.pW)) * 4;
  hipLaunchKernelGGL((bneck_step_kernel<T, KH, KW>), dim3(unsigned(g.B * cblocks)),
                     dim3(64 * kBnWaves), lds, s, pw.Cin, static_cast<const T*>(x), x_bc,
                     reinterpret_cast<const float*>(pwstate + PWL.weight),
                     reinterpret_cast<const float*>(pwstate + PWL.bias), act1, g,
                     reinterpret_cast<const float*>(cstate + L.weight),
                     reinterpret_cast<const float*>(cstate + L.bias),
                     reinterpret_cast<float*>(cstate + L.ring), L.ring_slot_elems, at, act2, pg,
                     static_cast<T*>(z), z_bc, reinterpret_cast<float*>(pstate + PL.fifo),
                     PL.fifo_slot_elems, reinterpret_cast<float*>(pstate + PL.valid), pp, cblocks,
                     make_fastdiv(uint32_t(S)), make_fastdiv(uint32_t(g.W)),
                     make_fastdiv(uint32_t(g.Wo)));
  return hipGetLastError();
}

}  // namespace

bool bneck_supported(const ConvGeom& pw, const ConvGeom& g, const PoolGeom& pg) {
  const int64_t S = int64_t(g.H) * g.W;
  return convpool_supported(g, pg) && pw.algo == CO_ALGO_DIRECT && pw.G == 1 && pw.kT == 1 &&
         pw.kH == 1 && pw.kW == 1 && pw.sT == 1 && pw.sH == 1 && pw.sW == 1 && pw.pT == 0 &&
         pw.pH == 0 && pw.pW == 0 && pw.dtype == g.dtype && pw.B == g.B && pw.Cout == g.Cin &&
         pw.H == g.H && pw.W == g.W && S <= 64 && int64_t(pw.Cin) * S <= kBnMaxStage &&
         int64_t(pw.B) * pw.Cin * S * (pw.dtype == CO_BF16 ? 2 : 4) < (int64_t(1) << 31);
}

hipError_t launch_bneck_step(const ConvGeom& pw, const ConvLayout& PWL, char* pwstate,
                             int32_t act1, const ConvGeom& g, const ConvLayout& L, char* cstate,
                             int32_t act2, const PoolGeom& pg, const PoolLayout& PL, char* pstate,
                             const void* x, int64_t x_bc, void* z, int64_t z_bc,
                             const co_step_plan& cplan, const co_pool_plan* pplan, bool update,
                             hipStream_t s) {
  if (g.dtype == CO_BF16) {
    if (g.kH == 3 && g.kW == 3)
      return bn_launch<bf16_t, 3, 3>(pw, PWL, pwstate, act1, g, L, cstate, act2, pg, PL, pstate,
                                     x, x_bc, z, z_bc, cplan, pplan, update, s);
    if (g.kH == 1 && g.kW == 1)
      return bn_launch<bf16_t, 1, 1>(pw, PWL, pwstate, act1, g, L, cstate, act2, pg, PL, pstate,
                                     x, x_bc, z, z_bc, cplan, pplan, update, s);
  } else {
    if (g.kH == 3 && g.kW == 3)
      return bn_launch<float, 3, 3>(pw, PWL, pwstate, act1, g, L, cstate, act2, pg, PL, pstate, x,
                                    x_bc, z, z_bc, cplan, pplan, update, s);
    if (g.kH == 1 && g.kW == 1)
      return bn_launch<float, 1, 1>(pw, PWL, pwstate, act1, g, L, cstate, act2, pg, PL, pstate, x,
                                    x_bc, z, z_bc, cplan, pplan, update, s);
  }
  return hipErrorInvalidValue;
}

bool convpool_supported(const ConvGeom& g, const PoolGeom& pg) {
  const bool taps = (g.kH == 3 && g.kW == 3) || (g.kH == 1 && g.kW == 1);
  return g.algo == CO_ALGO_DEPTHWISE && taps && g.dtype == pg.dtype && g.B == pg.B &&
         g.Cout == pg.C && pg.H == g.Ho && pg.W == g.Wo && g.So() <= 64 && pg.kH == g.Ho &&
         pg.kW == g.Wo && pg.pH == 0 && pg.pW == 0 && pg.dH == 1 && pg.dW == 1 &&
         pg.Ho == 1 && pg.Wo == 1 && pg.kT <= 64 && g.S() > 0 &&
         // the step kernel addresses a frame with 32-bit buffer offsets
         int64_t(g.B) * g.Cin * g.S() * (g.dtype == CO_BF16 ? 2 : 4) < (int64_t(1) << 31);
}

bool convpool_steps_supported(const ConvGeom& g, const PoolGeom& pg, int64_t T) {
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  const int64_t Hp = g.H + 2 * g.pH, Wp = g.W + 2 * g.pW;
  return convpool_supported(g, pg) && g.sT == 1 && g.dT == 1 && g.kT >= 1 && g.kT <= 5 &&
         pg.sT == 1 && pg.dT == 1 && pg.kT >= 1 && pg.kT <= 5 && pg.R == pg.kT &&
         g.R == g.kT && Hp * Wp <= kCpsMaxPadded && int64_t(g.H) * g.W <= 64 &&
         int64_t(g.B) * g.Cin * T * g.S() * esz < (int64_t(1) << 31);
}

hipError_t launch_convpool_steps(const ConvGeom& g, const ConvLayout& L, char* cstate,
                                 const PoolGeom& pg, const PoolLayout& PL, char* pstate,
                                 const void* x, int32_t T, void* z, int64_t z_cap, int64_t n0c,
                                 int64_t n0p, bool update, hipStream_t s) {
  if (!convpool_steps_supported(g, pg, T) || T <= 0) return hipErrorInvalidValue;
  if (g.dtype == CO_BF16)
    return cps_dispatch<bf16_t>(g, L, cstate, pg, PL, pstate, x, T, z, z_cap, n0c, n0p, update,
                                s);
  return cps_dispatch<float>(g, L, cstate, pg, PL, pstate, x, T, z, z_cap, n0c, n0p, update, s);
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
