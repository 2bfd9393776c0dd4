// Continual average / maximum pooling kernels.
//
// A pooling window factorises into a spatial reduction of each frame and a
// temporal reduction over the window's frames.  The state keeps the spatially
// reduced frames of the last f input frames in a FIFO of float32 frames
// (slot, B, C, Ho, Wo) plus one validity flag per slot (0 for end-padding
// frames).  Each step reduces the arriving frame once -- the intermediate
// result future outputs need, computed eagerly as section 3.1 describes
// before Principle 3 -- and, when the schedule emits, reduces the window's
// kT slots into the output.  Average pooling stores window sums (pads add 0)
// and divides once at emission; maximum pooling stores window maxima (pads
// are -inf).  Groups of lanes share each output element (see
// pool_step_kernel), so a window of 49 positions is loaded in one round.
#include <math.h>

#include <algorithm>

#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

// Reduction of v over the G lanes of a lane group (G a power of two <= 64).
template <int G>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int m = G / 2; m > 0; m >>= 1) v += __shfl_xor(v, m, G);
  return v;
}
template <int G>
__device__ __forceinline__ float group_max(float v) {
#pragma unroll
  for (int m = G / 2; m > 0; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, G));
  return v;
}

// One pool step.  G lanes share one output element (b, c, i, j): they load
// the spatial window together (lane r takes window elements r, r + G, ...,
// with clamped addresses so all loads are in flight at once) and reduce it
// with cross-lane shuffles; the FIFO slot is written by lane 0; when the
// schedule emits, lane j of the group fetches temporal tap j and the group
// reduces again.  No thread ever waits on a chain of dependent loads.
template <typename T, int G>
__global__ __launch_bounds__(kBlock) void pool_step_kernel(
    PoolGeom g, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y, int64_t y_bc,
    float* __restrict__ fifo, int64_t fifo_slot, float* __restrict__ valid, int32_t write_slot,
    int32_t update, int32_t emit, int32_t pad_frame, PoolTaps taps, FastDiv fd_So, FastDiv fd_Wo,
    FastDiv fd_kW) {
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.C * So;
  const int64_t gid = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  const int32_t idx = int32_t(gid / G);  // output element of this lane's group
  const int32_t r = int32_t(gid % G);    // lane within the group
  const bool live = idx < total;         // whole groups are live or not
  const int32_t e_idx = live ? idx : 0;
  const int32_t bc = fdiv(e_idx, fd_So);
  const int32_t p = e_idx - bc * So;
  const int32_t i = fdiv(p, fd_Wo), jo = p - i * g.Wo;
  const bool is_max = g.kind == CO_POOL_MAX;
  const int32_t kHW = g.kH * g.kW;

  // spatial reduction of the arriving frame (out-of-frame positions read an
  // out-of-range buffer offset: zero, no branch around the load)
  float val = is_max ? -INFINITY : 0.f;
  const int x_extent =
      pad_frame ? 0 : int(((int64_t(g.B) * g.C - 1) * x_bc + g.H * g.W) * int64_t(sizeof(T)));
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, x_extent);
  const int plane = int(int64_t(bc) * x_bc);
  for (int32_t e = r; e < kHW; e += G) {
    const int32_t u = fdiv(e, fd_kW), v = e - u * g.kW;
    const int32_t hi = i * g.sH + u * g.dH - g.pH;
    const int32_t wi = jo * g.sW + v * g.dW - g.pW;
    const bool in = hi >= 0 && hi < g.H && wi >= 0 && wi < g.W && !pad_frame;
    const float xv = load_or_zero<T>(xr, plane + hi * g.W + wi, in);
    if (in) val = is_max ? fmaxf(val, xv) : val + xv;
  }
  val = is_max ? group_max<G>(val) : group_sum<G>(val);
  if (!live) return;

  if (update && r == 0) {
    fifo[int64_t(write_slot) * fifo_slot + idx] = val;
    if (idx == 0) valid[write_slot] = pad_frame ? 0.f : 1.f;
  }
  if (!emit) return;

  // temporal reduction over the window's kT frames, spread over the group
  float acc = is_max ? -INFINITY : 0.f;
  float tcount = 0.f;
  for (int32_t t = r; t < g.kT; t += G) {
    const int32_t s = taps.src[t];
    if (s == -1) continue;  // start padding: ignored by max, adds 0 to a sum
    float ev, ok;
    if (s == -2) {          // the arriving frame
      ev = val;
      ok = pad_frame ? 0.f : 1.f;
    } else {
      ev = fifo[int64_t(s) * fifo_slot + idx];
      ok = valid[s];
    }
    acc = is_max ? fmaxf(acc, ev) : acc + ev;
    tcount += ok;
  }
  if (is_max) {
    acc = group_max<G>(acc);
  } else {
    acc = group_sum<G>(acc);
    tcount = group_sum<G>(tcount);
  }
  if (r != 0) return;
  float out;
  if (is_max) {
    out = acc;
  } else {
    // spatial positions inside the frame (count_include_pad = 0 divisor)
    int32_t vh = 0, vw = 0;
    for (int32_t u = 0; u < g.kH; ++u) {
      const int32_t hi = i * g.sH + u * g.dH - g.pH;
      vh += (hi >= 0 && hi < g.H) ? 1 : 0;
    }
    for (int32_t v = 0; v < g.kW; ++v) {
      const int32_t wi = jo * g.sW + v * g.dW - g.pW;
      vw += (wi >= 0 && wi < g.W) ? 1 : 0;
    }
    const float div = g.count_include_pad ? float(g.kT * kHW) : tcount * float(vh * vw);
    out = div > 0.f ? acc / div : 0.f;
  }
  y[int64_t(bc) * y_bc + p] = from_f32<T>(out);
}

template <typename T>
__global__ __launch_bounds__(kBlock) void pool_clip_kernel(PoolGeom g, int32_t T_in,
                                                           int32_t T_out,
                                                           const T* __restrict__ x,
                                                           T* __restrict__ y) {
  const int64_t So = int64_t(g.Ho) * g.Wo;
  const int64_t total = int64_t(g.B) * g.C * T_out * So;
  const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const int64_t p = idx % So;
  const int64_t t = (idx / So) % T_out;
  const int64_t bc = idx / (So * T_out);
  const int32_t i = int32_t(p / g.Wo), jo = int32_t(p % g.Wo);
  const int64_t S = int64_t(g.H) * g.W;
  const bool is_max = g.kind == CO_POOL_MAX;
  float acc = is_max ? -INFINITY : 0.f;
  int32_t count = 0;
  for (int32_t a = 0; a < g.kT; ++a) {
    const int64_t ti = t * g.sT + int64_t(a) * g.dT - g.pT;
    if (ti < 0 || ti >= T_in) continue;
    for (int32_t u = 0; u < g.kH; ++u) {
      const int32_t hi = i * g.sH + u * g.dH - g.pH;
      if (hi < 0 || hi >= g.H) continue;
      for (int32_t v = 0; v < g.kW; ++v) {
        const int32_t wi = jo * g.sW + v * g.dW - g.pW;
        if (wi < 0 || wi >= g.W) continue;
        const float e = to_f32<T>(x[(bc * T_in + ti) * S + hi * g.W + wi]);
        acc = is_max ? fmaxf(acc, e) : acc + e;
        ++count;
      }
    }
  }
  float out;
  if (is_max) {
    out = acc;
  } else {
    const int32_t div = g.count_include_pad ? g.kT * g.kH * g.kW : count;
    out = div > 0 ? acc / float(div) : 0.f;
  }
  y[idx] = from_f32<T>(out);
}

// ---- persistent forward_steps -------------------------------------------
//
// A clip of `count` frames in one launch (temporal stride 1 and dilation 1,
// a spatial window of at most G positions): the G lanes of output element
// (b, c, i, j) reduce each frame's window (one load per lane, the next
// frame's requested before the current one is reduced) and keep the last kT
// reduced frames and their validity in registers; when the schedule emits
// they reduce the window's frames into the output.  The FIFO is read at the
// start and written back at the end; the validity flags of the call's
// frames are written by the host afterwards.
struct PoolSteps {
  int64_t n0;     // step counter before the first frame
  int32_t count;  // frames: T real, then end padding
  int32_t T;
  int64_t emit0;  // first emitting step of the call: max(n0, d)
  int32_t sT;     // temporal stride: steps from n = d on emit every sT
  int32_t t_e0;   // first emitting frame of the call (count if none)
  int32_t update;
  int32_t x_bytes;  // bytes of the clip reachable from x
  int32_t y_bytes;  // bytes of the output clip
  int32_t fstride;  // bytes between consecutive frames
  FastDiv fd_So, fd_Wo, fd_kW;
};

template <typename T, int G, int KT, bool IS_MAX>
__global__ __launch_bounds__(kBlock) void pool_steps_kernel(
    PoolGeom g, PoolSteps ps, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y,
    int64_t y_bc, float* __restrict__ fifo, int64_t fifo_slot, const float* __restrict__ valid) {
  const int32_t So = g.Ho * g.Wo;
  const int32_t total = g.B * g.C * So;
  const int64_t gid = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  const int32_t idx = int32_t(gid / G);  // output element of this lane's group
  const int32_t r = int32_t(gid % G);    // lane within the group
  const bool live = idx < total;         // whole groups are live or not
  if (!live) return;                     // (no barrier follows)
  const int32_t bc = fdiv(idx, ps.fd_So);
  const int32_t p = idx - bc * So;
  const int32_t i = fdiv(p, ps.fd_Wo), jo = p - i * g.Wo;
  constexpr bool is_max = IS_MAX;  // (compile-time: no select per operation)
  const float neutral = is_max ? -INFINITY : 0.f;
  const int32_t kHW = g.kH * g.kW;

  // this lane's window position (at most one: kH*kW <= G)
  int32_t soff = -1;
  if (r < kHW) {
    const int32_t u = fdiv(r, ps.fd_kW), v = r - u * g.kW;
    const int32_t hi = i * g.sH + u * g.dH - g.pH;
    const int32_t wi = jo * g.sW + v * g.dW - g.pW;
    if (hi >= 0 && hi < g.H && wi >= 0 && wi < g.W) soff = hi * g.W + wi;
  }
  // divisor of an average with count_include_pad = 0: spatial positions in the frame
  int32_t vh = 0, vw = 0;
  for (int32_t u = 0; u < g.kH; ++u) {
    const int32_t hi = i * g.sH + u * g.dH - g.pH;
    vh += (hi >= 0 && hi < g.H) ? 1 : 0;
  }
  for (int32_t v = 0; v < g.kW; ++v) {
    const int32_t wi = jo * g.sW + v * g.dW - g.pW;
    vw += (wi >= 0 && wi < g.W) ? 1 : 0;
  }

  // fv[q], fok[q]: reduced value and validity of real frame n - (KT - 1) + q
  // at frame n; frames before the stream began are start padding
  float fv[KT], fok[KT];
#pragma unroll
  for (int q = 0; q + 1 < KT; ++q) {
    const int64_t rf = ps.n0 - (KT - 1) + q;
    const bool have = rf >= 0;
    fv[q] = have ? fifo[(rf % KT) * fifo_slot + idx] : neutral;
    fok[q] = have ? valid[rf % KT] : 0.f;
  }
  // the emitted value goes out through a buffer store that every lane issues
  // every frame, to the out-of-range offset unless lane 0 of a group emits:
  // a store under a branch would make the compiler wait for every frame in
  // flight before each frame
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, ps.y_bytes);
  const int yoff = int((uint32_t(bc) * uint32_t(y_bc) + uint32_t(p)) * sizeof(T));
  // raw bits of this lane's window element of frame t (converted when the
  // frame is reduced, so the loads stay in flight); positions outside the
  // frame read the out-of-range offset and become the neutral value at use
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ps.x_bytes);
  const int loff = soff >= 0 ? int((uint32_t(bc) * uint32_t(x_bc) + uint32_t(soff)) * sizeof(T))
                             : kOutOfRange;
  // every frame issues its load (frames past the clip at the out-of-range
  // offset), so the compiler's count of loads in flight stays exact around
  // the frame loop
  auto load = [&](int t) -> uint32_t {
    const bool real = t < ps.T;  // uniform
    return load_raw_at<T>(xr, real ? loff : kOutOfRange, real ? t * ps.fstride : 0);
  };
  auto value = [&](int t, uint32_t raw) {
    return (t < ps.T && soff >= 0) ? raw_to_f32<T>(raw) : neutral;
  };
  // frame t's window element sits in xq[t % PF]; the next PF - 1 frames'
  // are in flight while frame t is reduced (one register per frame, so the
  // loop keeps many: it is bound by the latency of these loads)
  constexpr int PF = 16;
  uint32_t xq[PF];
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    xq[u] = load(u);
    __builtin_amdgcn_sched_barrier(0);  // in frame order
  }
  // whole groups of PF frames with no exit inside: frames past the call
  // (the last group's tail) store nothing and leave the window as it is.
  // With a temporal stride the window is still the last kT frames; only
  // every sT-th step from the first emitting one emits (ep: its phase, ko:
  // the outputs so far).
  int ep = 0, ko = 0;
  for (int t0 = 0; t0 < ps.count; t0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int t = t0 + u;
      const bool dead = t >= ps.count;  // uniform
      const float xv = value(t, xq[u]);
      const float val = is_max ? group_max<G>(xv) : group_sum<G>(xv);
      xq[u] = load(t + PF);
      fv[KT - 1] = val;
      fok[KT - 1] = t < ps.T ? 1.f : 0.f;
      const int64_t n = ps.n0 + t;
      {
        // the window's frames as the per-step kernel combines them (tap q in
        // lane q of a lane group, then an xor-shuffle tree), so both paths
        // give the same bits; start padding contributes nothing
        float tv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const bool in = q < KT && n - (KT - 1) + q >= 0;
          tv[q] = in ? fv[q < KT ? q : 0] : neutral;
        }
#pragma unroll
        for (int m = 4; m > 0; m >>= 1) {
          float nv[8];
#pragma unroll
          for (int l = 0; l < 8; ++l) nv[l] = is_max ? fmaxf(tv[l], tv[l ^ m]) : tv[l] + tv[l ^ m];
#pragma unroll
          for (int l = 0; l < 8; ++l) tv[l] = nv[l];
        }
        const float acc = tv[0];
        // the count of real frames, only for an average without the pads
        // (uniform branch, no memory operation inside)
        float tcount = 0.f;
        if (!is_max && !g.count_include_pad) {
          float tc[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const bool in = q < KT && n - (KT - 1) + q >= 0;
            tc[q] = in ? fok[q < KT ? q : 0] : 0.f;
          }
#pragma unroll
          for (int m = 4; m > 0; m >>= 1) {
            float nc[8];
#pragma unroll
            for (int l = 0; l < 8; ++l) nc[l] = tc[l] + tc[l ^ m];
#pragma unroll
            for (int l = 0; l < 8; ++l) tc[l] = nc[l];
          }
          tcount = tc[0];
        }
        float out;
        if (is_max) {
          out = acc;
        } else {
          const float div = g.count_include_pad ? float(KT * kHW) : tcount * float(vh * vw);
          out = div > 0.f ? acc / div : 0.f;
        }
        const bool on = (t >= ps.t_e0) & !dead;  // uniform
        const bool emits = on & (ep == 0);
        store_at(yr, (emits && r == 0) ? yoff : kOutOfRange,
                 emits ? int(int64_t(ko) * So * int64_t(sizeof(T))) : 0, from_f32<T>(out));
        ko += emits ? 1 : 0;
        ep = on ? (ep + 1 == ps.sT ? 0 : ep + 1) : ep;
      }
      // (a dead frame's value went into the last place only, which the next
      // frame overwrites; the call ends after the group anyway)
#pragma unroll
      for (int q = 0; q + 1 < KT; ++q) {
        fv[q] = dead ? fv[q] : fv[q + 1];
        fok[q] = dead ? fok[q] : fok[q + 1];
      }
      __builtin_amdgcn_sched_barrier(0);  // frames in order
    }
  }
  if (ps.update && r == 0) {
    const int64_t n1 = ps.n0 + ps.count;
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) {
      const int64_t rf = n1 - (KT - 1) + q;
      if (rf >= 0) fifo[(rf % KT) * fifo_slot + idx] = fv[q];
    }
  }
}

// Global spatial pooling (the window covers the whole frame: kH = H, kW = W,
// no spatial padding or dilation, one output per plane and frame), as in a
// network head.  Lanes hold frames instead of window positions: one wave per
// (stream, channel) plane stages a block of kPgFrames of its frames -- they
// lie contiguously in the clip -- into LDS with 16-byte loads (the next
// block's loads in flight while a block is reduced), and lane t reduces
// frame t of the block alone, in the order of the per-step kernel's shuffle
// tree over 64 window lanes (element r in leaf r, the rest neutral), so both
// paths give the same bits.  The window's frames then come from the lanes
// below (from the previous block, or the FIFO, across the block's start) and
// combine in that kernel's temporal tree.  The per-step kernel spends a
// shuffle tree, a temporal tree and a division on each frame for one value;
// here each costs one lane.
constexpr int kPgFrames = 32;  // frames per block, lanes 0..31

struct PoolGlobalArgs {
  int32_t nblk;       // blocks of the call: ceil(count / kPgFrames)
  int32_t lds_bytes;  // per wave: a block, its alignment and 64 elements of over-read
  int32_t F;          // window span f = (kT - 1) dT + 1: FIFO slots
  int64_t tau0;       // output index of the call's first emission
};

// Value of `cur` in lane (lane - k) of this block, or of `prev` in the
// previous block's lane kPgFrames + lane - k.
__device__ __forceinline__ float lane_back(float cur, float prev, int lane, int k) {
  const float a = __int_as_float(__builtin_amdgcn_ds_bpermute(((lane - k) & 63) << 2,
                                                              __float_as_int(cur)));
  const float b = __int_as_float(__builtin_amdgcn_ds_bpermute(
      ((kPgFrames + lane - k) & 63) << 2, __float_as_int(prev)));
  return lane >= k ? a : b;
}

template <typename T, int KT, bool IS_MAX>
__global__ __launch_bounds__(64) void pool_steps_global_kernel(
    PoolGeom g, PoolSteps ps, PoolGlobalArgs pa, const T* __restrict__ x, int64_t x_bc,
    T* __restrict__ y, int64_t y_bc, float* __restrict__ fifo, int64_t fifo_slot,
    const float* __restrict__ valid) {
  extern __shared__ uint4 pg_lds[];
  constexpr uint32_t esz = sizeof(T);
  constexpr int NU = esz == 2 ? 5 : 9;  // 16-byte units per lane and block
  constexpr bool is_max = IS_MAX;
  const float neutral = is_max ? -INFINITY : 0.f;
  const int lane = int(threadIdx.x);
  const int bc = int(blockIdx.x);  // one wave per plane
  const int S = g.H * g.W;
  const int plane = int(uint32_t(bc) * uint32_t(x_bc) * esz);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ps.x_bytes);
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, ps.y_bytes);
  const int yplane = int(uint32_t(bc) * uint32_t(y_bc) * esz);

  // the previous block's reduced frames and validity by lane; before the
  // first block, lanes kPgFrames - (F - 1) + q hold the FIFO's frame
  // n0 - (F - 1) + q (the window spans F = (kT - 1) dT + 1 frames)
  const int F = pa.F;
  float prev = neutral, prevok = 0.f;
  {
    const int q = lane - (kPgFrames - (F - 1));
    const int64_t rf = ps.n0 - (F - 1) + q;
    if (q >= 0 && lane < kPgFrames && rf >= 0) {
      prev = fifo[(rf % F) * fifo_slot + bc];
      prevok = valid[rf % F];
    }
  }

  // block b's real frames from the 16-byte boundary at or below their first
  // byte; units past them read the out-of-range offset, and the one unit
  // that runs past the clip's end is read element by element
  struct Block {
    int s0, a0, units;
  };
  auto block = [&](int b) {
    Block k;
    const int t0 = b * kPgFrames;
    const int nr = min(max(ps.T - t0, 0), kPgFrames);
    k.s0 = plane + t0 * ps.fstride;
    k.a0 = k.s0 & ~15;
    k.units = nr > 0 ? (k.s0 + nr * ps.fstride - k.a0 + 15) >> 4 : 0;
    return k;
  };
  auto fetch = [&](const Block& k, uint4 (&v)[NU]) {
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      const int u = j * 64 + lane;
      const int off = k.a0 + u * 16;
      const bool whole = u < k.units && off + 16 <= ps.x_bytes;
      const auto v4 = __builtin_amdgcn_raw_buffer_load_b128(xr, whole ? off : kOutOfRange, 0, 0);
      v[j] = make_uint4(v4[0], v4[1], v4[2], v4[3]);
      if (u < k.units && off + 16 > ps.x_bytes) {
        uint32_t h[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if constexpr (esz == 2) {
            const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(
                xr, off + 4 * e + 2 <= ps.x_bytes ? off + 4 * e : kOutOfRange, 0, 0);
            const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(
                xr, off + 4 * e + 4 <= ps.x_bytes ? off + 4 * e + 2 : kOutOfRange, 0, 0);
            h[e] = lo | (hi << 16);
          } else {
            h[e] = __builtin_amdgcn_raw_buffer_load_b32(
                xr, off + 4 * e + 4 <= ps.x_bytes ? off + 4 * e : kOutOfRange, 0, 0);
          }
        }
        v[j] = make_uint4(h[0], h[1], h[2], h[3]);
      }
    }
  };

  uint4 v[NU];
  Block cb = block(0);
  fetch(cb, v);
  for (int b = 0; b < pa.nblk; ++b) {
#pragma unroll
    for (int j = 0; j < NU; ++j)
      if (j * 64 + lane < cb.units) pg_lds[j * 64 + lane] = v[j];
    __syncthreads();  // (one wave: its LDS writes land before the reads)
    const int shift = cb.s0 - cb.a0;
    if (b + 1 < pa.nblk) {
      cb = block(b + 1);
      fetch(cb, v);
    }

    // lane t: frame t0 + t, its S elements in leaves 0..S-1.  The leaf
    // masks are built from a vector copy of S made here, in the loop: as
    // loop invariants the compiler would hoist all 64 of them, as scalar
    // lane masks, out of the loop and spill them
    int Sv;
    __asm__ volatile("v_mov_b32 %0, %1" : "=v"(Sv) : "s"(S));
    const uint32_t nb = __float_as_uint(neutral);
    const int t = b * kPgFrames + lane;
    const bool live = lane < kPgFrames;
    const char* fb =
        reinterpret_cast<const char*>(pg_lds) + shift + (live ? lane : 0) * ps.fstride;
    auto leaf = [&](int r) {
      float xv;
      if constexpr (esz == 2)
        xv = __uint_as_float(uint32_t(*reinterpret_cast<const uint16_t*>(fb + 2 * r)) << 16);
      else
        xv = *reinterpret_cast<const float*>(fb + 4 * r);
      // as the per-step kernel: the neutral value, combined with the element
      const float lv = is_max ? fmaxf(neutral, xv) : neutral + xv;
      const uint32_t keep = uint32_t((r - Sv) >> 31);  // all ones when r < S
      return __uint_as_float((__float_as_uint(lv) & keep) | (nb & ~keep));
    };
    auto comb = [&](float a, float c) { return is_max ? fmaxf(a, c) : a + c; };
    float tr[32];
#pragma unroll
    for (int l = 0; l < 32; ++l) tr[l] = comb(leaf(l), leaf(l + 32));
#pragma unroll
    for (int m = 16; m > 0; m >>= 1)
#pragma unroll
      for (int l = 0; l < m; ++l) tr[l] = comb(tr[l], tr[l + m]);
    const bool real = live && t < ps.T;
    const float cur = real ? tr[0] : neutral;
    const float curok = real ? 1.f : 0.f;
    __syncthreads();  // the reads are done before the next block's writes

    // the window of step n = n0 + t: frames n - (KT - 1 - q) dT, q = 0..KT-1
    // (the temporal stride only decides which steps emit)
    const int64_t n = ps.n0 + t;
    float fv[KT], fok[KT];
    fv[KT - 1] = cur;
    fok[KT - 1] = curok;
#pragma unroll
    for (int q = 0; q + 1 < KT; ++q) {
      fv[q] = lane_back(cur, prev, lane, (KT - 1 - q) * g.dT);
      fok[q] = lane_back(curok, prevok, lane, (KT - 1 - q) * g.dT);
    }
    float tv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const bool in = q < KT && n - int64_t(KT - 1 - q) * g.dT >= 0;
      tv[q] = in ? fv[q < KT ? q : 0] : neutral;
    }
#pragma unroll
    for (int m = 4; m > 0; m >>= 1) {
      float nv[8];
#pragma unroll
      for (int l = 0; l < 8; ++l) nv[l] = is_max ? fmaxf(tv[l], tv[l ^ m]) : tv[l] + tv[l ^ m];
#pragma unroll
      for (int l = 0; l < 8; ++l) tv[l] = nv[l];
    }
    float out = tv[0];
    if (!is_max) {
      float div = float(KT * S);
      if (!g.count_include_pad) {
        float tc[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const bool in = q < KT && n - int64_t(KT - 1 - q) * g.dT >= 0;
          tc[q] = in ? fok[q < KT ? q : 0] : 0.f;
        }
#pragma unroll
        for (int m = 4; m > 0; m >>= 1) {
          float nc[8];
#pragma unroll
          for (int l = 0; l < 8; ++l) nc[l] = tc[l] + tc[l ^ m];
#pragma unroll
          for (int l = 0; l < 8; ++l) tc[l] = nc[l];
        }
        div = tc[0] * float(S);
      }
      out = div > 0.f ? out / div : 0.f;
    }
    const bool emits = live && t < ps.count && n >= g.d && (n - g.d) % g.sT == 0;
    const int64_t k = emits ? (n - g.d) / g.sT - pa.tau0 : 0;  // the call's k-th output
    store_at(yr, emits ? yplane : kOutOfRange, emits ? int(k * int64_t(esz)) : 0,
             from_f32<T>(out));
    // the call's last F - 1 frames go to their FIFO slots
    if (ps.update && live && t < ps.count && t >= ps.count - (F - 1))
      fifo[(n % F) * fifo_slot + bc] = cur;
    prev = cur;
    prevok = curok;
  }
}

// Validity flags of the FIFO slots the call's frames went to (one thread).
__global__ void pool_valid_kernel(float* valid, int32_t R, int64_t n0, int32_t count, int32_t T) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int32_t first = count > R ? count - R : 0;
  for (int32_t t = first; t < count; ++t) valid[(n0 + t) % R] = t < T ? 1.f : 0.f;
}

__global__ void pool_header_kernel(StateHeader h, StateHeader* dst) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *dst = h;
}

template <typename T, int G>
hipError_t pool_step_g(const PoolGeom& g, const PoolLayout& L, char* state, const StepIO& io,
                       const co_pool_plan& plan, bool update, bool pad, hipStream_t s) {
  PoolTaps taps;
  for (int j = 0; j < CO_MAX_TAPS; ++j) taps.src[j] = plan.src[j];
  float* fifo = reinterpret_cast<float*>(state + L.fifo);
  float* valid = reinterpret_cast<float*>(state + L.valid);
  hipLaunchKernelGGL((pool_step_kernel<T, G>), dim3(grid_for(g.out_frame_elems() * G)),
                     dim3(kBlock), 0, s, g, static_cast<const T*>(io.x), io.x_bc,
                     static_cast<T*>(io.y), io.y_bc, fifo, L.fifo_slot_elems, valid,
                     plan.write_slot, update ? 1 : 0, plan.emit, pad ? 1 : 0, taps,
                     make_fastdiv(uint32_t(g.So())), make_fastdiv(uint32_t(g.Wo)),
                     make_fastdiv(uint32_t(g.kW)));
  return hipGetLastError();
}

// Lanes per output element: enough to cover the spatial window (and the
// temporal taps) in about one load each.
template <typename T>
hipError_t pool_step_t(const PoolGeom& g, const PoolLayout& L, char* state, const StepIO& io,
                       const co_pool_plan& plan, bool update, bool pad, hipStream_t s) {
  const int work = std::max(g.kH * g.kW, g.kT);
  if (work > 16) return pool_step_g<T, 64>(g, L, state, io, plan, update, pad, s);
  if (work > 4) return pool_step_g<T, 16>(g, L, state, io, plan, update, pad, s);
  return pool_step_g<T, 4>(g, L, state, io, plan, update, pad, s);
}

}  // namespace

hipError_t launch_pool_step(const PoolGeom& g, const PoolLayout& L, char* state,
                            const StepIO& io, const co_pool_plan& plan, bool update_state,
                            bool pad_frame, hipStream_t s) {
  if (g.dtype == CO_BF16) return pool_step_t<bf16_t>(g, L, state, io, plan, update_state, pad_frame, s);
  return pool_step_t<float>(g, L, state, io, plan, update_state, pad_frame, s);
}

hipError_t launch_pool_init(const PoolGeom& g, const PoolLayout& L, char* state,
                            const StateHeader& hdr, hipStream_t s) {
  hipLaunchKernelGGL(pool_header_kernel, dim3(1), dim3(64), 0, s, hdr,
                     reinterpret_cast<StateHeader*>(state + L.header));
  return hipGetLastError();
}

hipError_t launch_pool_clip(const PoolGeom& g, int32_t T, int32_t T_out, const void* x, void* y,
                            hipStream_t s) {
  const int64_t total = int64_t(g.B) * g.C * T_out * g.So();
  if (total == 0) return hipSuccess;
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(pool_clip_kernel<bf16_t>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, T,
                       T_out, static_cast<const bf16_t*>(x), static_cast<bf16_t*>(y));
  else
    hipLaunchKernelGGL(pool_clip_kernel<float>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, T,
                       T_out, static_cast<const float*>(x), static_cast<float*>(y));
  return hipGetLastError();
}

namespace {

template <typename T, int KT>
hipError_t pool_global_launch(const PoolGeom& g, const PoolLayout& L, char* state, const void* x,
                              int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                              int64_t n0, bool update, hipStream_t s);
bool pool_global_fits(const PoolGeom& g);

template <typename T, int G, int KT>
hipError_t pool_steps_launch(const PoolGeom& g, const PoolLayout& L, char* state, const void* x,
                             int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                             int64_t n0, bool update, hipStream_t s) {
  if (pool_global_fits(g))
    return pool_global_launch<T, KT>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  PoolSteps ps;
  ps.n0 = n0;
  ps.count = count;
  ps.T = nreal;
  ps.emit0 = n0 > g.d ? n0 : g.d;
  ps.sT = g.sT;
  {
    const int64_t te = n0 >= g.d ? (g.sT - (n0 - g.d) % g.sT) % g.sT : g.d - n0;
    ps.t_e0 = int32_t(std::min<int64_t>(te, count));
  }
  ps.update = update ? 1 : 0;
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  ps.x_bytes = int32_t(((int64_t(g.B) * g.C - 1) * x_bc + int64_t(nreal) * g.S()) * esz);
  ps.y_bytes = int32_t(int64_t(g.B) * g.C * y_bc * esz);
  ps.fstride = int32_t(g.S() * esz);
  ps.fd_So = make_fastdiv(uint32_t(g.So()));
  ps.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  ps.fd_kW = make_fastdiv(uint32_t(g.kW));
  float* fifo = reinterpret_cast<float*>(state + L.fifo);
  float* valid = reinterpret_cast<float*>(state + L.valid);
  auto kern = g.kind == CO_POOL_MAX ? pool_steps_kernel<T, G, KT, true>
                                     : pool_steps_kernel<T, G, KT, false>;
  hipLaunchKernelGGL(kern, dim3(grid_for(g.out_frame_elems() * G)), dim3(kBlock), 0, s, g, ps,
                     static_cast<const T*>(x), x_bc, static_cast<T*>(y), y_bc, fifo,
                     L.fifo_slot_elems, valid);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !update) return e;
  hipLaunchKernelGGL(pool_valid_kernel, dim3(1), dim3(64), 0, s, valid, g.R, n0, count, nreal);
  return hipGetLastError();
}

// Global spatial pooling over small frames with the per-step kernel's
// 64-lane window groups (16 < H*W <= 64): the frames-in-lanes kernel.
bool pool_global_fits(const PoolGeom& g) {
  const int kHW = g.kH * g.kW;
  return g.kH == g.H && g.kW == g.W && g.pH == 0 && g.pW == 0 && g.dH == 1 && g.dW == 1 &&
         g.Ho == 1 && g.Wo == 1 && kHW > 16 && kHW <= 64;
}

template <typename T, int KT>
hipError_t pool_global_launch(const PoolGeom& g, const PoolLayout& L, char* state, const void* x,
                              int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                              int64_t n0, bool update, hipStream_t s) {
  PoolSteps ps{};  // (the emission fields go in pa)
  ps.n0 = n0;
  ps.count = count;
  ps.T = nreal;
  ps.emit0 = n0 > g.d ? n0 : g.d;
  ps.sT = g.sT;
  ps.update = update ? 1 : 0;
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  ps.x_bytes = int32_t(((int64_t(g.B) * g.C - 1) * x_bc + int64_t(nreal) * g.S()) * esz);
  ps.y_bytes = int32_t(int64_t(g.B) * g.C * y_bc * esz);
  ps.fstride = int32_t(g.S() * esz);
  PoolGlobalArgs pa;
  pa.nblk = int32_t((int64_t(count) + kPgFrames - 1) / kPgFrames);
  pa.F = g.R;  // the FIFO holds the window's span
  const int64_t lo = n0 > g.d ? n0 : g.d;
  pa.tau0 = (lo - g.d + g.sT - 1) / g.sT;
  // the block, its alignment shift and the 64-element over-read of the last lane
  pa.lds_bytes = int32_t(((kPgFrames * g.S() + 64) * esz + 16 + 15) / 16 * 16);
  if (pa.lds_bytes > 64 * 16 * (esz == 2 ? 5 : 9)) return hipErrorInvalidValue;  // NU units
  float* fifo = reinterpret_cast<float*>(state + L.fifo);
  float* valid = reinterpret_cast<float*>(state + L.valid);
  auto kern = g.kind == CO_POOL_MAX ? pool_steps_global_kernel<T, KT, true>
                                     : pool_steps_global_kernel<T, KT, false>;
  hipLaunchKernelGGL(kern, dim3(unsigned(int64_t(g.B) * g.C)), dim3(64), pa.lds_bytes, s, g, ps,
                     pa, static_cast<const T*>(x), x_bc, static_cast<T*>(y), y_bc, fifo,
                     L.fifo_slot_elems, valid);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !update) return e;
  hipLaunchKernelGGL(pool_valid_kernel, dim3(1), dim3(64), 0, s, valid, g.R, n0, count, nreal);
  return hipGetLastError();
}

template <typename T, int G>
hipError_t pool_steps_kt(const PoolGeom& g, const PoolLayout& L, char* state, const void* x,
                         int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                         int64_t n0, bool update, hipStream_t s) {
  switch (g.kT) {
    case 1: return pool_steps_launch<T, G, 1>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 2: return pool_steps_launch<T, G, 2>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 3: return pool_steps_launch<T, G, 3>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 4: return pool_steps_launch<T, G, 4>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    case 5: return pool_steps_launch<T, G, 5>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t pool_steps_t(const PoolGeom& g, const PoolLayout& L, char* state, const void* x,
                        int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                        int64_t n0, bool update, hipStream_t s) {
  const int kHW = g.kH * g.kW;
  if (kHW > 16) return pool_steps_kt<T, 64>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  if (kHW > 4) return pool_steps_kt<T, 16>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  return pool_steps_kt<T, 4>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
}

}  // namespace

hipError_t launch_pool_valid(float* valid, int32_t R, int64_t n0, int32_t count, int32_t T,
                             hipStream_t s) {
  hipLaunchKernelGGL(pool_valid_kernel, dim3(1), dim3(64), 0, s, valid, R, n0, count, T);
  return hipGetLastError();
}

bool pool_steps_supported(const PoolGeom& g, int64_t x_frames, int64_t y_frames) {
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  // temporal stride or dilation above 1: the frames-in-lanes global pool,
  // whose window reaches (kT - 1) dT lanes back across one block; the lane
  // group kernel, whose window is the last kT frames, takes a stride alone
  const bool strided = g.sT != 1 || g.dT != 1;
  const bool general = pool_global_fits(g) ? int64_t(g.kT - 1) * g.dT < kPgFrames : g.dT == 1;
  return (!strided || general) && g.kT >= 1 && g.kT <= 5 && g.kH * g.kW <= 64 &&  // (kT <= 8: tree)
         int64_t(g.B) * g.C * x_frames * g.S() * esz < (int64_t(1) << 31) &&
         int64_t(g.B) * g.C * y_frames * g.So() * esz < (int64_t(1) << 31);
}

hipError_t launch_pool_steps(const PoolGeom& g, const PoolLayout& L, char* state, const void* x,
                             int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                             int64_t n0, bool update, hipStream_t s) {
  if (g.dtype == CO_BF16)
    return pool_steps_t<bf16_t>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  return pool_steps_t<float>(g, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
}

}  // namespace coinf
