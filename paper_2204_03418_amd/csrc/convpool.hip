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
  int32_t pk[CO_MAX_TAPS];  // tap | action << 8 | ring slot << 16
  __host__ __device__ int tap(int a) const { return pk[a] & 0xff; }
  __host__ __device__ int act(int a) const { return (pk[a] >> 8) & 0xff; }
  __host__ __device__ int slot(int a) const { return pk[a] >> 16; }
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

constexpr int kCpMaxTaps = 8;  // temporal taps of a fused depthwise convolution

// What one lane of a fused step reads from the states, all of it known
// before the step's arithmetic: the ring partial sums of the taps that
// continue one (ACC, EMIT) and, when the pool emits, the pooled frame and
// valid flag of window element `lane` from the FIFO.  Loading them at the
// start of the kernel overlaps their round trips with the rest.
struct CpPrefetch {
  float prev[kCpMaxTaps];
  float fev, fok;
};

__device__ __forceinline__ void dw_pool_prefetch(bool pl, int lane, int bc, int ridx,
                                                 const float* __restrict__ ring,
                                                 int64_t ring_slot, const CpTaps& at,
                                                 const PoolGeom& pg,
                                                 const float* __restrict__ fifo,
                                                 int64_t fifo_slot,
                                                 const float* __restrict__ valid,
                                                 const CpPool& pp, CpPrefetch* f) {
#pragma unroll
  for (int a = 0; a < kCpMaxTaps; ++a) {
    f->prev[a] = 0.f;
    if (a < at.n) {
      const int act = at.act(a);
      if (pl && (act == CO_TAP_ACC || act == CO_TAP_EMIT))
        f->prev[a] = ring[int64_t(at.slot(a)) * ring_slot + ridx];
    }
  }
  f->fev = 0.f;
  f->fok = 0.f;
  // the FIFO slots read here are never the one this step writes (the
  // window's other frames are older than the arriving one)
  if (pp.step && pp.emit && lane < pg.kT) {
    const int s = pp.src[lane];
    if (s >= 0) {
      f->fev = fifo[int64_t(s) * fifo_slot + bc];
      f->fok = valid[s];
    }
  }
}

// The depthwise step of one lane (output pixel p of a plane with flat index
// bc, ring index ridx, the channel's weights wc (kT x KH x KW) and bias bo)
// from its stencil values xv and the prefetched state values, then the pool
// step on the completed frame (see the kernels below): shared by the fused
// kernels so that they give the separate steps' bits.
template <typename T, int KH, int KW>
__device__ __forceinline__ void dw_pool_tail(
    const float (&xv)[KH * KW], const CpPrefetch& f, bool pl, int lane, int bc, int ridx,
    const float* wc, float bo, float* __restrict__ ring, int64_t ring_slot, const CpTaps& at,
    int act2, const PoolGeom& pg, T* __restrict__ z, int64_t z_bc, float* __restrict__ fifo,
    int64_t fifo_slot, float* __restrict__ valid, const CpPool& pp) {
  T yv = from_f32<T>(0.f);
#pragma unroll
  for (int a = 0; a < kCpMaxTaps; ++a) {
    if (a >= at.n) break;
    const int act = at.act(a);
    float acc = f.prev[a];
    const float* wj = wc + at.tap(a) * (KH * KW);
#pragma unroll
    for (int e = 0; e < KH * KW; ++e) acc = fmaf(wj[e], xv[e], acc);
    if (act == CO_TAP_START || act == CO_TAP_ACC) {
      if (pl) ring[int64_t(at.slot(a)) * ring_slot + ridx] = acc;
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
      const float ev = s == -2 ? val : f.fev;
      acc = is_max ? fmaxf(acc, ev) : acc + ev;
      tcount += s == -2 ? 1.f : f.fok;
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
  CpPrefetch pf;
  dw_pool_prefetch(pl, lane, bc, ridx, ring, ring_slot, at, pg, fifo, fifo_slot, valid, pp, &pf);
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
  dw_pool_tail<T, KH, KW>(xv, pf, pl, lane, bc, ridx, w + int64_t(c) * g.kT * (KH * KW), bias[c],
                          ring, ring_slot, at, CO_ACT_NONE, pg, z, z_bc, fifo, fifo_slot, valid,
                          pp);
}

// Fused step of an X3D-style bottleneck (sections 3.2-3.3: a pointwise
// convolution, batch normalisation and activation, a depthwise continual
// convolution, batch normalisation and activation, and the pool over the
// plane; the normalisations are folded into the convolutions' weights at
// init).  A workgroup owns one 16-channel fragment of the pointwise output
// for one stream (at most 64 pixels per plane).  Wave w computes pixels
// 16w..16w+15 of the fragment on the matrix cores exactly as the register
// GEMM step kernel computes a pointwise layer: the same packed weights, the
// same operand lanes (eight channels per lane and k-step for bf16, one for
// fp32), the k-steps in the same order from zero, the same epilogue (the zero
// partial sum and the bias added, rounded to the io dtype), then the
// activation as the elementwise step applies it.  The results go into 16
// zero-haloed planes in LDS; after one barrier each of the 8 waves runs the
// depthwise and pool steps of two channels from there, as in
// convpool_step_kernel, with every state read issued at the kernel's start.  The intermediate frames never leave the CU, and the
// results equal the separate steps bit for bit.
constexpr int kBnWaves = 4;  // pixel fragments of the plane (64 pixels)
constexpr int kBnCh = 16;    // channels per workgroup: one 16-column fragment
constexpr int kBnTail = 16;  // waves per workgroup; each steps kBnCh / kBnTail channels
constexpr int kBnPer = kBnCh / kBnTail;
// k-steps whose operand loads issue together (bf16: eight 2-byte loads per
// lane and k-step; fp32: one)
constexpr int kBnKB = 2;
constexpr int kBnKF = 8;

typedef float bn_v4f __attribute__((ext_vector_type(4)));
typedef __bf16 bn_v8bf __attribute__((ext_vector_type(8)));

template <typename T, int KH, int KW>
__global__ __launch_bounds__(64 * kBnTail, 8) void bneck_step_kernel(
    int32_t Ci, int32_t CS, int32_t CSU, const T* __restrict__ x, int64_t x_bc, int32_t x_bytes,
    const uint4* __restrict__ w1, int32_t w1_bytes, const float* __restrict__ b1, int32_t act1,
    ConvGeom g, const float* __restrict__ w, const float* __restrict__ bias,
    float* __restrict__ ring, int64_t ring_slot, CpTaps at, int32_t act2, PoolGeom pg,
    T* __restrict__ z, int64_t z_bc, float* __restrict__ fifo, int64_t fifo_slot,
    float* __restrict__ valid, CpPool pp, int32_t cblocks, FastDiv fd_W, FastDiv fd_Wo) {
  // LDS: the workgroup's depthwise weights (kBnCh x kT x KH x KW) and biases
  // (kBnCh), then kBnCh zero-haloed planes of Hp x Wp
  extern __shared__ float lds[];
  constexpr bool kBF = sizeof(T) == 2;
  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int S = g.H * g.W;
  const int Hp = g.H + 2 * g.pH, Wp = g.W + 2 * g.pW, HWp = Hp * Wp;
  const int bq = int(blockIdx.x) / cblocks;
  const int nf = int(blockIdx.x) - bq * cblocks;  // channel fragment
  const int kTW = g.kT * KH * KW;
  float* ws = lds;
  float* zs = lds + kBnCh * (kTW + 1);
  // the fragment's channels are consecutive, so their weights are one run
  {
    const int nch = min(kBnCh, g.Cout - nf * kBnCh);
    for (int e = tid; e < nch * kTW; e += 64 * kBnTail) ws[e] = w[int64_t(nf) * kBnCh * kTW + e];
    if (tid < nch) ws[kBnCh * kTW + tid] = bias[nf * kBnCh + tid];
  }
  // this wave's depthwise channels (wave + kBnTail k of the fragment) and
  // output pixel: their state reads first
  const int So = g.Ho * g.Wo;
  const bool pl = lane < So;
  const int p = pl ? lane : 0;
  int cl[kBnPer], bc[kBnPer], ridx[kBnPer];
  bool cv[kBnPer];
#pragma unroll
  for (int k = 0; k < kBnPer; ++k) {
    cl[k] = wave + kBnTail * k;
    const int c = nf * kBnCh + cl[k];
    cv[k] = c < g.Cout;
    bc[k] = bq * g.Cout + c;
    ridx[k] = (c * g.B + bq) * So + p;
  }
  CpPrefetch pf[kBnPer];
  const bool pw_wave = wave < kBnWaves;
#pragma unroll
  for (int k = 0; k < kBnPer; ++k)
    dw_pool_prefetch(pl & cv[k], cv[k] ? lane : 64, bc[k], ridx[k], ring, ring_slot, at, pg, fifo,
                     fifo_slot, valid, pp, &pf[k]);
  // zero the planes' halo; the interior is written by the pointwise phase
  // below (every pixel of every plane in use), so the two never touch the
  // same element before the barrier
  for (int e = tid; e < kBnCh * HWp; e += 64 * kBnTail) {
    const int q = e % HWp;
    const int r = q / Wp, col = q - r * Wp;
    if (r < g.pH || r >= g.pH + g.H || col < g.pW || col >= g.pW + g.W) zs[e] = 0.f;
  }

  // ---- pointwise convolution on the matrix cores (waves 0-3) -------------
  // lane (lrow, lgrp) supplies pixel P = 16 * wave + lrow; pixels past the
  // plane and channels past C_in read an out-of-range offset (zero)
  if (pw_wave) {
    const int oc = nf * 16 + lrow;  // the output channel this lane holds
    const bool ov = oc < g.Cin;
    const float bo = ov ? b1[oc] : 0.f;
    const int P = wave * 16 + lrow;
    const bool pv = P < S;
    constexpr uint32_t esz = sizeof(T);
    const uint32_t plane_b = uint32_t(x_bc) * esz;
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, x_bytes);
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(w1, w1_bytes);
    // k-steps in groups of kBnKB whose loads issue together; k-steps past the
    // layer's read zeros (as the step kernel's k-steps past C_in do)
    bn_v4f acc = bn_v4f{0.f, 0.f, 0.f, 0.f};
    if constexpr (kBF) {
      const int lane_c = lgrp * 8;
      const uint32_t base = (uint32_t(bq) * uint32_t(Ci) + uint32_t(lane_c)) * plane_b +
                            uint32_t(pv ? P : 0) * esz;
      for (int c0 = 0; c0 < CS; c0 += kBnKB) {
        uint4 a[kBnKB], b[kBnKB];
#pragma unroll
        for (int k = 0; k < kBnKB; ++k) {
          const int cb = c0 + k;
          const bool live = cb < CS;
          uint32_t r[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const bool ok = live & pv & (cb * 32 + lane_c + e < Ci);
            r[e] = __builtin_amdgcn_raw_buffer_load_b16(
                xr, ok ? int(base + uint32_t(cb * 32 + e) * plane_b) : kOutOfRange, 0, 0);
          }
          a[k] = make_uint4(r[0] | (r[1] << 16), r[2] | (r[3] << 16), r[4] | (r[5] << 16),
                            r[6] | (r[7] << 16));
          const auto b4 = __builtin_amdgcn_raw_buffer_load_b128(
              wr, live ? ((nf * CSU + cb) << 10) + lane * 16 : kOutOfRange, 0, 0);
          b[k] = make_uint4(b4[0], b4[1], b4[2], b4[3]);
        }
        // keep the group's loads one batch ahead of its matrix work
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < kBnKB; ++k)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bn_v8bf, a[k]),
                                                        __builtin_bit_cast(bn_v8bf, b[k]), acc, 0,
                                                        0, 0);
      }
    } else {
      // one channel per lane and k-step; a weight unit holds four k-steps
      const uint32_t base = (uint32_t(bq) * uint32_t(Ci) + uint32_t(lgrp)) * plane_b +
                            uint32_t(pv ? P : 0) * esz;
      for (int c0 = 0; c0 < CS; c0 += kBnKF) {
        float a[kBnKF];
        uint4 b[kBnKF / 4];
#pragma unroll
        for (int k = 0; k < kBnKF; ++k) {
          const int cb = c0 + k;
          const bool ok = (cb < CS) & pv & (cb * 4 + lgrp < Ci);
          a[k] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
              xr, ok ? int(base + uint32_t(cb * 4) * plane_b) : kOutOfRange, 0, 0));
        }
#pragma unroll
        for (int q = 0; q < kBnKF / 4; ++q) {
          const int cq = c0 / 4 + q;
          const auto b4 = __builtin_amdgcn_raw_buffer_load_b128(
              wr, cq < CSU ? ((nf * CSU + cq) << 10) + lane * 16 : kOutOfRange, 0, 0);
          b[q] = make_uint4(b4[0], b4[1], b4[2], b4[3]);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < kBnKF; ++k) {
          const uint4 u = b[k / 4];
          const uint32_t bw = (k & 3) == 0 ? u.x : (k & 3) == 1 ? u.y : (k & 3) == 2 ? u.z : u.w;
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[k], __uint_as_float(bw), acc, 0, 0, 0);
        }
      }
    }
    // lane (lrow, lgrp) holds channel oc at pixels 16*wave + 4*lgrp + r
    float* zc = zs + lrow * HWp;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int p = wave * 16 + 4 * lgrp + r;
      const float val = acc[r] + bo;  // (the step kernel's chain starts from a zero partial sum)
      T z1;
      if constexpr (kBF)
        z1 = __builtin_bit_cast(uint16_t, __bf16(val));
      else
        z1 = val;
      if (act1 == CO_ACT_RELU) z1 = from_f32<T>(fmaxf(to_f32<T>(z1), 0.f));
      if (ov & (p < S)) {
        const int qi = fdiv(p, fd_W), qj = p - qi * g.W;
        zc[(qi + g.pH) * Wp + qj + g.pW] = to_f32<T>(z1);
      }
    }
  }  // pointwise waves
  __syncthreads();

  // ---- depthwise convolution and pool, kBnPer channels per wave -----------
  const int i = fdiv(p, fd_Wo), jo = p - i * g.Wo;
#pragma unroll
  for (int k = 0; k < kBnPer; ++k) {
    if (!cv[k]) return;  // wave-uniform, after the last barrier
    const float* zw = zs + cl[k] * HWp;
    float xv[KH * KW];
#pragma unroll
    for (int u = 0; u < KH; ++u)
#pragma unroll
      for (int v = 0; v < KW; ++v)
        xv[u * KW + v] = pl ? zw[(i * g.sH + u * g.dH) * Wp + jo * g.sW + v * g.dW] : 0.f;
    dw_pool_tail<T, KH, KW>(xv, pf[k], pl, lane, bc[k], ridx[k], ws + cl[k] * kTW,
                            ws[kBnCh * kTW + cl[k]], ring, ring_slot, at, act2, pg, z, z_bc,
                            fifo, fifo_slot, valid, pp);
  }
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
    at.pk[at.n] =
        j | (int32_t(cplan.action[j]) << 8) | ((cplan.slot[j] < 0 ? 0 : cplan.slot[j]) << 16);
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
// both modules).  One wave per (stream, channel) plane for the whole clip,
// one lane per input and per output pixel: the convolution's kT - 1 partial
// sums stay in registers, so only the clip, the pooled outputs and the two
// states move through memory.
//
// Convolution: each frame is written, as float, into a zero-haloed tile of
// LDS, so a stencil tap is one LDS read at a lane address fixed for the clip
// plus a compile-time slot offset; the channel's weights are wave-uniform;
// frames go in groups of U, the next group's pixels in flight while a group
// is evaluated (the depthwise forward_steps kernel's scheme).  Pool: lane p
// turns its completed, rounded output into window leaf p as the pool step
// kernel does (the neutral value combined with the element; lanes past the
// plane hold the neutral value) and writes it to the frame's row of 64 leaves
// in LDS.  Every NB frames the lanes switch to frames: lane r reduces row r
// in the pool step kernel's shuffle-tree order, takes the window's frames
// from the lanes below (the previous block's, or the FIFO's, across the
// block's start) and combines them in that kernel's temporal tree.  So a clip
// gives the bits of stepping frame by frame, and the spatial tree, temporal
// tree and division cost one lane per frame, not a wave.
constexpr int kCpsSlot = 128;       // floats per frame slot: padded tile + sink cell
constexpr int kCpsMaxPadded = 128;  // padded plane, elements (the bottleneck kernel's bound)

struct CpSteps {
  int32_t v0;       // virtual time of the first frame: n0 + pT (clamped)
  int32_t slot0;    // ring slot of output v0 - (kT - 1)
  int32_t count;    // frames in the call
  int32_t update;
  int32_t x_bytes;  // bytes of the clip reachable from x
  int32_t fstride;  // bytes between consecutive frames of a plane
  int32_t PW;       // padded tile width: W + 2 pW
  int32_t tfirst;   // first frame of the call whose convolution step emits
  int64_t n0p;      // pool steps before the call
  int64_t emit0p;   // first pool step of the call that emits: max(n0p, pool delay)
  FastDiv fd_Cout, fd_Wo, fd_W;
};

__device__ __forceinline__ void cps_lds_order() { __asm__ volatile("" ::: "memory"); }

template <typename T, int KH, int KW, int KT, int PKT, bool IS_MAX>
__global__ __launch_bounds__(64) void convpool_steps_kernel(
    ConvGeom g, CpSteps cs, const T* __restrict__ x, int64_t x_bc, const float* __restrict__ w,
    const float* __restrict__ bias, float* __restrict__ ring, int64_t ring_slot, PoolGeom pg,
    T* __restrict__ z, int64_t z_bc, float* __restrict__ fifo, int64_t fifo_slot,
    const float* __restrict__ valid) {
  constexpr int NS = KH * KW;
  constexpr int U = KT * ((4 + KT - 1) / KT);  // frames per group (acc names cycle)
  constexpr uint32_t esz = sizeof(T);
  // frames per pool block: whole groups, about 2.3 KB of leaf rows
  constexpr int NB = U * ((2304 / (64 * int(esz))) / U > 0 ? (2304 / (64 * int(esz))) / U : 1);
  static_assert(NB <= 64, "one lane per row");
  constexpr bool is_max = IS_MAX;
  __shared__ float slot[U][kCpsSlot];
  constexpr int RS = 64 + 16 / int(esz);  // row stride: rows 16 bytes apart in bank order
  __shared__ T rows[NB][RS];
  const float neutral = is_max ? -INFINITY : 0.f;
  const int lane = int(threadIdx.x);
  const int bc = int(blockIdx.x);  // one wave per plane
  const int S = g.H * g.W, So = g.Ho * g.Wo;
  const int bq = fdiv(bc, cs.fd_Cout), c = bc - bq * g.Cout;

  for (int e = lane; e < U * kCpsSlot; e += 64) (&slot[0][0])[e] = 0.f;  // halos stay zero

  // input lane: pixel `lane` of the frame into its padded cell (lanes past
  // the frame load zero into the sink cell after the tile)
  int wpos = kCpsSlot - 1;
  if (lane < S) {
    const int hp = fdiv(lane, cs.fd_W);
    wpos = (hp + g.pH) * cs.PW + (lane - hp * g.W) + g.pW;
  }
  float* const wp = &slot[0][wpos];  // + u * kCpsSlot: slot u
  const int xin = lane < S ? int((uint32_t(bc) * uint32_t(x_bc) + uint32_t(lane)) * esz)
                           : kOutOfRange;
  // output lane: its stencil cells in the padded tile
  const bool pl = lane < So;
  const int p = pl ? lane : 0;
  const int i = fdiv(p, cs.fd_Wo), jo = p - i * g.Wo;
  const float* rp[NS];  // + u * kCpsSlot: slot u
#pragma unroll
  for (int u = 0; u < KH; ++u)
#pragma unroll
    for (int v = 0; v < KW; ++v)
      rp[u * KW + v] = &slot[0][(i * g.sH + u * g.dH) * cs.PW + jo * g.sW + v * g.dW];
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
    const int tau = cs.v0 - (KT - 1) + q;
    const int slq = (cs.slot0 + q) % KT;
    acc[q] = (pl && q < KT - 1 && tau >= 0) ? ring[slq * ring_slot + ridx] : 0.f;
  }

  // pool: the previous block's reduced frames and validity by lane; before
  // the first block, lanes NB - (PKT - 1) + q hold the FIFO's pool frame
  // n0p - (PKT - 1) + q (frames before the stream began are start padding)
  float prev = neutral, prevok = 0.f;
  {
    const int q = lane - (NB - (PKT - 1));
    const int64_t rf = cs.n0p - (PKT - 1) + q;
    if (q >= 0 && lane < NB && rf >= 0) {
      prev = fifo[(rf % PKT) * fifo_slot + bc];
      prevok = valid[rf % PKT];
    }
  }

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, cs.x_bytes);
  auto load = [&](int t) {
    const bool real = t < cs.count;
    return load_raw_at<T>(xr, real ? xin : kOutOfRange, real ? t * cs.fstride : 0);
  };
  // evaluate the frame in slot u (row r of the pool block): every live
  // output takes its tap, the oldest completes and becomes this lane's leaf
  auto eval = [&](int t, int u, T* row, bool steady) {
    float xv[NS];
#pragma unroll
    for (int e = 0; e < NS; ++e) xv[e] = rp[e][u * kCpsSlot];
    const int v = cs.v0 + t;
#pragma unroll
    for (int j = KT - 1; j >= 0; --j) {
      const int q = KT - 1 - j;
      const int tau = v - j;
      const int first = steady ? 0 : (tau >= g.pT ? 0 : g.pT - tau);
      float a = (j == first) ? 0.f : acc[q];
#pragma unroll
      for (int e = 0; e < NS; ++e) a = fmaf(wr[j][e], xv[e], a);
      if (j == KT - 1) {
        const float yv = to_f32<T>(from_f32<T>(a + bo));
        const float lf = is_max ? fmaxf(neutral, yv) : neutral + yv;
        row[lane] = from_f32<T>(pl ? lf : neutral);
      } else {
        acc[q] = a;
      }
    }
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) acc[q] = acc[q + 1];
  };
  auto comb = [&](float a, float b2) { return is_max ? fmaxf(a, b2) : a + b2; };

  uint32_t xa[U];
#pragma unroll
  for (int u = 0; u < U; ++u) xa[u] = load(u);
  for (int sb0 = 0; sb0 < cs.count; sb0 += NB) {
    // the block's frames through the convolution, in groups of U
    for (int gi = 0; gi < NB / U; ++gi) {
      const int t = sb0 + gi * U;
      if (t >= cs.count) break;  // uniform
      cps_lds_order();
#pragma unroll
      for (int u = 0; u < U; ++u) wp[u * kCpsSlot] = raw_to_f32<T>(xa[u]);
      cps_lds_order();
#pragma unroll
      for (int u = 0; u < U; ++u) xa[u] = load(t + U + u);
      T* row0 = &rows[gi * U][0];
      if (t + U <= cs.count && cs.v0 + t - (KT - 1) >= g.pT) {
#pragma unroll
        for (int u = 0; u < U; ++u) eval(t + u, u, row0 + u * RS, true);
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (t + u >= cs.count) break;  // (the clip's last, ragged group)
          eval(t + u, u, row0 + u * RS, false);
        }
      }
    }
    cps_lds_order();

    // lanes = frames: lane r reduces frame sb0 + r of the block
    const int t = sb0 + lane;
    const bool pooled = lane < NB && t < cs.count && t >= cs.tfirst;  // the pool steps
    const T* row = &rows[lane < NB ? lane : 0][0];
    float tr[32];
#pragma unroll
    for (int l = 0; l < 32; ++l) tr[l] = comb(to_f32<T>(row[l]), to_f32<T>(row[l + 32]));
#pragma unroll
    for (int m = 16; m > 0; m >>= 1)
#pragma unroll
      for (int l = 0; l < m; ++l) tr[l] = comb(tr[l], tr[l + m]);
    cps_lds_order();
    const float cur = pooled ? tr[0] : neutral;
    const float curok = pooled ? 1.f : 0.f;
    // the window of pool step m: pool frames m - (PKT - 1) + q, q = 0..PKT-1
    const int64_t m = cs.n0p + (t - cs.tfirst);
    float fv[PKT], fok[PKT];
    fv[PKT - 1] = cur;
    fok[PKT - 1] = curok;
#pragma unroll
    for (int q = 0; q + 1 < PKT; ++q) {
      const int k = PKT - 1 - q;
      const int src = ((lane - k) & 63) << 2, psrc = ((NB + lane - k) & 63) << 2;
      const float a1 = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(cur)));
      const float b1 = __int_as_float(__builtin_amdgcn_ds_bpermute(psrc, __float_as_int(prev)));
      const float a2 = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(curok)));
      const float b2 = __int_as_float(__builtin_amdgcn_ds_bpermute(psrc, __float_as_int(prevok)));
      fv[q] = lane >= k ? a1 : b1;
      fok[q] = lane >= k ? a2 : b2;
    }
    float tv[8];
#pragma unroll
    for (int l = 0; l < 8; ++l) {
      const bool in = l < PKT && m - (PKT - 1) + l >= 0;
      tv[l] = in ? fv[l < PKT ? l : 0] : neutral;
    }
#pragma unroll
    for (int mm = 4; mm > 0; mm >>= 1) {
      float nv[8];
#pragma unroll
      for (int l = 0; l < 8; ++l) nv[l] = comb(tv[l], tv[l ^ mm]);
#pragma unroll
      for (int l = 0; l < 8; ++l) tv[l] = nv[l];
    }
    float out = tv[0];
    if (!is_max) {
      float div = float(PKT * So);
      if (!pg.count_include_pad) {
        float tc[8];
#pragma unroll
        for (int l = 0; l < 8; ++l) {
          const bool in = l < PKT && m - (PKT - 1) + l >= 0;
          tc[l] = in ? fok[l < PKT ? l : 0] : 0.f;
        }
#pragma unroll
        for (int mm = 4; mm > 0; mm >>= 1) {
          float nc[8];
#pragma unroll
          for (int l = 0; l < 8; ++l) nc[l] = tc[l] + tc[l ^ mm];
#pragma unroll
          for (int l = 0; l < 8; ++l) tc[l] = nc[l];
        }
        div = tc[0] * float(So);
      }
      out = div > 0.f ? out / div : 0.f;
    }
    if (pooled && m >= pg.d) z[int64_t(bc) * z_bc + (m - cs.emit0p)] = from_f32<T>(out);
    // the call's last PKT - 1 pool frames go to their FIFO slots
    if (cs.update && pooled && t >= cs.count - (PKT - 1)) fifo[(m % PKT) * fifo_slot + bc] = cur;
    prev = cur;
    prevok = curok;
  }

  if (cs.update && pl) {
    const int v1 = cs.v0 + cs.count;
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) {
      const int tau = v1 - (KT - 1) + q;
      const int slq = (cs.slot0 + cs.count + q) % KT;
      if (tau >= 0) ring[slq * ring_slot + ridx] = acc[q];
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
  cs.PW = g.W + 2 * g.pW;
  const int64_t tf = int64_t(g.kT - 1) - v0;
  cs.tfirst = int32_t(tf > 0 ? tf : 0);
  cs.n0p = n0p;
  cs.emit0p = n0p > pg.d ? n0p : pg.d;
  cs.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  cs.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  cs.fd_W = make_fastdiv(uint32_t(g.W));
  const int64_t planes = int64_t(g.B) * g.Cout;
  float* valid = reinterpret_cast<float*>(pstate + PL.valid);
  auto kern = pg.kind == CO_POOL_MAX ? convpool_steps_kernel<T, KH, KW, KT, PKT, true>
                                      : convpool_steps_kernel<T, KH, KW, KT, PKT, false>;
  hipLaunchKernelGGL(kern, dim3(unsigned(planes)), dim3(64), 0, s, g, cs,
                     static_cast<const T*>(x), x_bc,
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
    at->pk[at->n] =
        j | (int32_t(cplan.action[j]) << 8) | ((cplan.slot[j] < 0 ? 0 : cplan.slot[j]) << 16);
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
  RegConfig rc;
  if (!reg_config(pw, pw.cfg, &rc)) return hipErrorInvalidValue;
  const int32_t cblocks = int32_t((g.Cin + kBnCh - 1) / kBnCh);
  const int64_t S = int64_t(g.H) * g.W;
  const int64_t x_bytes = ((int64_t(pw.B) * pw.Cin - 1) * x_bc + S) * int64_t(sizeof(T));
  const int64_t w_bytes = int64_t(rc.n_frags) * rc.U * 64 * 16;
  if (x_bytes >= (int64_t(1) << 31) || w_bytes >= (int64_t(1) << 31))
    return hipErrorInvalidValue;
  const size_t lds =
      size_t(kBnCh) * ((g.H + 2 * g.pH) * (g.W + 2 * g.pW) + g.kT * KH * KW + 1) * 4;
  hipLaunchKernelGGL((bneck_step_kernel<T, KH, KW>), dim3(unsigned(g.B * cblocks)),
                     dim3(64 * kBnTail), lds, s, pw.Cin, rc.CS, rc.CSU,
                     static_cast<const T*>(x), x_bc, int32_t(x_bytes),
                     reinterpret_cast<const uint4*>(pwstate + PWL.weight), int32_t(w_bytes),
                     reinterpret_cast<const float*>(pwstate + PWL.bias), act1, g,
                     reinterpret_cast<const float*>(cstate + L.weight),
                     reinterpret_cast<const float*>(cstate + L.bias),
                     reinterpret_cast<float*>(cstate + L.ring), L.ring_slot_elems, at, act2, pg,
                     static_cast<T*>(z), z_bc, reinterpret_cast<float*>(pstate + PL.fifo),
                     PL.fifo_slot_elems, reinterpret_cast<float*>(pstate + PL.valid), pp, cblocks,
                     make_fastdiv(uint32_t(g.W)), make_fastdiv(uint32_t(g.Wo)));
  return hipGetLastError();
}

}  // namespace

bool bneck_supported(const ConvGeom& pw, const ConvGeom& g, const PoolGeom& pg) {
  const int64_t S = int64_t(g.H) * g.W;
  const int64_t Hp = g.H + 2 * g.pH, Wp = g.W + 2 * g.pW;
  RegConfig rc;
  return convpool_supported(g, pg) && pw.algo == CO_ALGO_GEMM_REG &&
         reg_config(pw, pw.cfg, &rc) && pw.G == 1 && pw.kT == 1 && pw.kH == 1 && pw.kW == 1 &&
         pw.sT == 1 && pw.sH == 1 && pw.sW == 1 && pw.pT == 0 && pw.pH == 0 && pw.pW == 0 &&
         pw.dtype == g.dtype && pw.B == g.B && pw.Cout == g.Cin && pw.H == g.H && pw.W == g.W &&
         S <= 16 * kBnWaves && Hp * Wp <= kCpsMaxPadded &&
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
  return g.algo == CO_ALGO_DEPTHWISE && taps && g.kT <= kCpMaxTaps && g.R < 32768 &&
         g.dtype == pg.dtype &&
         g.B == pg.B &&
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
         g.R == g.kT && Hp * Wp + 1 <= kCpsSlot && int64_t(g.H) * g.W <= 64 &&
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
