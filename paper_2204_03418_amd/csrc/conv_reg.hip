// Register-operand implicit-GEMM continual convolution step (groups = 1,
// small reduction depth K = kH*kW*C_in).
//
// The per-step contraction is the same GEMM as in the LDS-tiled kernel
// (m = output pixel of a stream, n = (temporal tap, output channel),
// k = (spatial tap, input channel)), and the same fused ring epilogue follows
// it (section 3.1: the arriving frame's contribution to every future output
// is computed at once and kept as a partial sum).  For layers whose K is
// small, staging tiles through LDS costs more than it saves: the step is a
// few hundred cycles of matrix work behind several dependent trips to
// memory.  Here one wave owns a tile of 16 output pixels x 16*WN columns and
// keeps every k-step's operands in registers:
//
//   * input pixels are gathered straight from the NCHW frame with buffer
//     loads, one value (fp32) or eight channels (bf16) per lane and k-step,
//     in the lane order of the matrix instruction; taps outside the frame
//     read an out-of-range offset, which returns zero, so every load issues
//     at once;
//   * weights were packed at init as 16-byte units in the exact lane order
//     of the instruction, so each lane fetches them with 16-byte loads;
//   * the ring partial sums the tile continues are requested with them.
//
// The wave then runs its MFMAs back to back onto the seeded accumulators and
// stores the ring / output.  No LDS and no barrier: one round trip to memory
// plus the matrix work.  Each lane computes its own input address, so any
// stride, dilation and spatial padding is handled.
#include <algorithm>
#include <type_traits>

#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// Tiles per workgroup of both kernels.  One tile (one wave, or the KSPLIT
// waves that share it) per workgroup measures fastest: the steps are bound
// by launch and memory latency, and small workgroups are dispatched and
// retired as soon as their own tile is done; in the persistent kernel the
// waves of a tile meet at the per-frame barrier without waiting for the
// waves of other tiles.
constexpr int kRegTiles = 1;

constexpr int kRegMaxTaps = 16;  // tap offsets passed (>= taps per wave x waves per tile)

struct RegArgs {
  int32_t M, N, So;
  int32_t m_frags, nf0, n_grps;  // column groups of WN fragments from fragment nf0
  int32_t blocks_per_xcd;
  int32_t ntaps, CS, CSU;        // spatial taps, channel blocks, weight units per tap
  int32_t dh[kRegMaxTaps], dw[kRegMaxTaps];  // input row / column offset of each tap
  int32_t x_bytes, w_bytes;
  int32_t ring_slot, ring_bytes;  // floats between ring slots; bytes of all slots
  int32_t y_bc, y_bytes;          // y plane stride (elements); bytes of y
  FastDiv fd_So, fd_Wo, fd_Cout, fd_ngrps;  // dividers: pixels per frame, Wo, C_out, n_grps
};

// Per-tap action and ring slot as one dword each (action | slot << 8), so
// the kernel reads them with scalar loads (there is no scalar byte load).
struct RegTaps {
  int32_t as[CO_MAX_TAPS];
};

// TAPS: spatial taps one wave holds.  KSPLIT: waves sharing one tile; wave h
// of a tile takes taps h*TAPS .. h*TAPS + TAPS - 1 and the partial sums meet
// in LDS, which halves each wave's serial gathers and MFMAs when a layer has
// too few tiles to give every SIMD more than one wave.  VEC: M % 4 == 0
// (whole 16-byte ring stores).  EXACT: the layer has exactly CSMAX channel
// blocks and C_in is a multiple of the block width, so no k-step is idle and
// no lane reads past C_in (no per-k-step selects).
template <typename T, int WN, int TAPS, int CSMAX, int KSPLIT, bool VEC, bool EXACT>
__global__ __launch_bounds__(64 * KSPLIT * kRegTiles) void conv_step_reg_kernel(
    ConvGeom g, RegArgs ra, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y,
    int64_t y_bc, const uint4* __restrict__ wp, const float* __restrict__ bias,
    float* __restrict__ ring, RegTaps tt) {
  constexpr bool kBF = sizeof(T) == 2;
  constexpr int CL = kBF ? 8 : 1;  // input channels per lane and k-step
  constexpr int CKS = 4 * CL;      // input channels per k-step (channel block)
  // 16-byte weight units per tap: fp32 packs four channel blocks per unit
  constexpr int CSUMAX = kBF ? CSMAX : (CSMAX + 3) / 4;
  const int lane = int(threadIdx.x) & 63;
  // wave index as a scalar, so everything derived from the tile stays uniform
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int lrow = lane & 15, lgrp = lane >> 4;

  // XCD-aware numbering: blocks are dealt to the 8 XCDs round-robin, so
  // consecutive logical blocks (neighbouring tiles) share an XCD's L2.
  const int bid = int(blockIdx.x);
  const int lb = (bid & 7) * ra.blocks_per_xcd + (bid >> 3);
  constexpr int TPW = kRegTiles;  // tiles per workgroup
  const int h = wave % KSPLIT, wslot = wave / KSPLIT;
  const int tile_raw = lb * TPW + wslot;
  const int tiles = ra.m_frags * ra.n_grps;
  if constexpr (KSPLIT == 1) {
    if (tile_raw >= tiles) return;  // whole waves; no barrier follows
  }
  // with a split, waves past the last tile keep to the barrier: they redo
  // tile 0 with every store masked
  const bool live = tile_raw < tiles;
  const int tile = live ? tile_raw : 0;
  const bool owner = live & (h == 0);  // the wave that stores the tile
  const int mf = fdiv(tile, ra.fd_ngrps);
  const int nfb = ra.nf0 + (tile - mf * ra.n_grps) * WN;

  // ---- epilogue data ------------------------------------------------------
  // lane (lrow, lgrp) of fragment f holds column n = (nfb+f)*16 + lrow and
  // the four consecutive pixels mf*16 + lgrp*4 .. +3 of the result.  The
  // taps a fragment spans are read with wave-uniform (scalar) loads, so the
  // ring reads issue in the same batch as the operand gathers.
  int e_act[WN], e_o[WN], e_off[WN];  // action, channel, ring element offset
  float e_bias[WN];
  const __amdgpu_buffer_rsrc_t br = make_rsrc(bias, g.Cout * 4);
  // column n = t*C_out + o: decode the wave's first column once, then step 16
  // columns per fragment (C_out >= 16, so o wraps at most once per step)
  const int n0 = nfb * 16;
  int tq = fdiv(n0, ra.fd_Cout), oq = n0 - tq * g.Cout;  // wave-uniform: fragment f's first column
#pragma unroll
  for (int f = 0; f < WN; ++f) {
    const int n = (nfb + f) * 16 + lrow;
    int t = tq, o = oq + lrow;
    if (o >= g.Cout) {  // per lane: the fragment crosses into the next tap
      o -= g.Cout;
      ++t;
    }
    // the fragment spans taps tq and tq + 1 at most: two scalar reads
    const int a0 = tt.as[min(tq, g.kT - 1)], a1 = tt.as[min(tq + 1, g.kT - 1)];
    const int as = t == tq ? a0 : a1;
    const bool in = n < ra.N;
    e_act[f] = in ? (as & 0xff) : CO_TAP_NONE;
    o = in ? o : 0;
    e_o[f] = o;
    e_off[f] = (as >> 8) * ra.ring_slot + o * ra.M;
    e_bias[f] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(br, o * 4, 0, 0));
    oq += 16;
    if (oq >= g.Cout) {  // uniform
      oq -= g.Cout;
      ++tq;
    }
  }
  const int P0 = mf * 16 + lgrp * 4;
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(ring, ra.ring_bytes);

  // ---- one batch of loads: ring partial sums, bias, then the operands ----
  // The ring holds a partial sum for taps that add to it (ACC, EMIT); other
  // taps read an out-of-range offset (zero).  The matrix work accumulates
  // onto them (the first chain of a split tile; the other starts from zero),
  // so the persistent kernel, whose partial sums stay in the accumulators,
  // folds each frame exactly as this step does.
  v4f prev[WN];
#pragma unroll
  for (int f = 0; f < WN; ++f) {
    // one 16-byte read per lane (slots end with four floats of padding, so a
    // ragged frame's last pixels stay in range; pixels past M are not stored)
    const bool rd = ((e_act[f] == CO_TAP_ACC) | (e_act[f] == CO_TAP_EMIT)) & (P0 < ra.M) & owner;
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(
        rr, rd ? (e_off[f] + P0) * 4 : kOutOfRange, 0, 0);
    prev[f] = v4f{__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                  __uint_as_float(v[3])};
  }

  // ---- operand gathers --------------------------------------------------
  // k-step (tap tp, channel block cb): lane (lrow, lgrp) supplies row m =
  // pixel lrow and channel(s) cb*CKS + lgrp*CL (+ 0..CL-1).  The tap's
  // per-lane offset and frame test are computed once per tap; a k-step adds
  // a uniform channel-block offset.  Taps outside the frame and channels past
  // C_in read an out-of-range offset (zero), so every load is in bounds.
  const int P = mf * 16 + lrow;
  const bool pvalid = P < ra.M;
  const int Pc = pvalid ? P : 0;
  const int b = fdiv(Pc, ra.fd_So), p = Pc - b * ra.So;
  const int i = fdiv(p, ra.fd_Wo), j = p - i * g.Wo;
  const int hb = i * g.sH - g.pH, wb = j * g.sW - g.pW;
  const int lane_c = lgrp * CL;
  constexpr uint32_t esz = sizeof(T);
  const uint32_t plane_b = uint32_t(x_bc) * esz;
  const uint32_t lane_b = (uint32_t(b) * uint32_t(g.Cin) + uint32_t(lane_c)) * plane_b;
  // channels of this lane inside the last channel block (it may be partial)
  const int nv_last = min(max(g.Cin - ((ra.CS - 1) * CKS + lane_c), 0), CL);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ra.x_bytes);

  using AReg = typename std::conditional<kBF, uint4, float>::type;
  AReg areg[TAPS][CSMAX];
  const int tp0 = h * TAPS;  // first tap of this wave
#pragma unroll
  for (int i = 0; i < TAPS; ++i) {
    const int tp = tp0 + i;
    // per-lane offset of the tap's pixel in channel block 0, or out of range;
    // a channel block adds a wave-uniform offset through the instruction's
    // scalar operand.  In the last block lanes past C_in read out of range.
    const int hi = hb + ra.dh[tp], wi = wb + ra.dw[tp];
    const bool ok = (tp < ra.ntaps) & pvalid & (unsigned(hi) < unsigned(g.H)) &
                    (unsigned(wi) < unsigned(g.W));
    const int vt = ok ? int(lane_b + (uint32_t(hi) * uint32_t(g.W) + uint32_t(wi)) * esz)
                      : kOutOfRange;
    if constexpr (kBF) {
      int vlast[8];  // last block: element e exists iff e < nv_last
#pragma unroll
      for (int e = 0; e < 8; ++e)
        vlast[e] = (ok & (e < nv_last)) ? vt + int(uint32_t(e) * plane_b) : kOutOfRange;
#pragma unroll
      for (int cb = 0; cb < CSMAX; ++cb) {
        const bool live = EXACT || cb < ra.CS;  // wave-uniform
        const bool last = !EXACT && cb == ra.CS - 1;
        const int sb = int(uint32_t(cb * CKS) * plane_b);
        uint32_t r[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int v = !live ? kOutOfRange : last ? vlast[e] : vt;
          const int so = last ? sb : sb + int(uint32_t(e) * plane_b);
          r[e] = __builtin_amdgcn_raw_buffer_load_b16(xr, v, so, 0);
        }
        areg[i][cb] = make_uint4(r[0] | (r[1] << 16), r[2] | (r[3] << 16),
                                 r[4] | (r[5] << 16), r[6] | (r[7] << 16));
      }
    } else {
      const int vl = nv_last > 0 ? vt : kOutOfRange;
#pragma unroll
      for (int cb = 0; cb < CSMAX; ++cb) {
        const bool live = EXACT || cb < ra.CS;  // wave-uniform
        const bool last = !EXACT && cb == ra.CS - 1;
        const int v = !live ? kOutOfRange : last ? vl : vt;
        areg[i][cb] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            xr, v, int(uint32_t(cb * CKS) * plane_b), 0));
      }
    }
  }

  // weights: unit (fragment nf, tap tp, unit cq) of this lane at
  // (((nf * ntaps + tp) * CSU + cq) * 64 + lane) * 16 bytes
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(wp, ra.w_bytes);
  uint4 breg[WN][TAPS][CSUMAX];
#pragma unroll
  for (int f = 0; f < WN; ++f)
#pragma unroll
    for (int i = 0; i < TAPS; ++i)
#pragma unroll
      for (int cq = 0; cq < CSUMAX; ++cq) {
        const int tp = tp0 + i;
        const bool okw = (tp < ra.ntaps) & (cq < ra.CSU);
        const int off = ((((nfb + f) * ra.ntaps + tp) * ra.CSU + cq) << 10) + lane * 16;
        const auto w4 =
            __builtin_amdgcn_raw_buffer_load_b128(wr, okw ? off : kOutOfRange, 0, 0);
        breg[f][i][cq] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      }

  // ---- matrix work --------------------------------------------------------
  // Straight-line MFMAs over every k-step the instantiation holds (k-steps
  // past the layer's taps / channel blocks multiply zeros): with no branch
  // here the loads above stay one batch, and each instruction waits only for
  // its own operands.
  __builtin_amdgcn_sched_barrier(0);
  v4f acc[WN];
#pragma unroll
  for (int f = 0; f < WN; ++f) acc[f] = h == 0 ? prev[f] : v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int tp = 0; tp < TAPS; ++tp) {
#pragma unroll
    for (int cb = 0; cb < CSMAX; ++cb) {
#pragma unroll
      for (int f = 0; f < WN; ++f) {
        if constexpr (kBF) {
          acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(v8bf, areg[tp][cb]), __builtin_bit_cast(v8bf, breg[f][tp][cb]),
              acc[f], 0, 0, 0);
        } else {
          const uint4 u4 = breg[f][tp][cb / 4];
          const uint32_t bw = (cb & 3) == 0 ? u4.x : (cb & 3) == 1 ? u4.y : (cb & 3) == 2 ? u4.z : u4.w;
          acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(areg[tp][cb], __uint_as_float(bw), acc[f],
                                                        0, 0, 0);
        }
      }
    }
  }

  if constexpr (KSPLIT == 2) {
    // the two waves of a tile exchange partial sums through LDS; both end
    // with the full sum, the owner stores it
    __shared__ v4f red[TPW][2][WN][64];
#pragma unroll
    for (int f = 0; f < WN; ++f) red[wslot][h][f][lane] = acc[f];
    __syncthreads();
#pragma unroll
    for (int f = 0; f < WN; ++f) acc[f] += red[wslot][1 - h][f][lane];
  }

  // ---- fused ring epilogue (branch-free) ----------------------------------
  // Stores go through buffer resources; a lane that must not store uses an
  // out-of-range offset, which the hardware drops.  With no branch after the
  // tile test the compiler cannot move any load of the batch down here.
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, ra.y_bytes);
  constexpr int yesz = int(sizeof(T));
  const int pb = fdiv(P0, ra.fd_So), pp = P0 - pb * ra.So;  // frame and pixel of the lane's first row
#pragma unroll
  for (int f = 0; f < WN; ++f) {
    const int act = e_act[f];
    const bool to_ring = ((act == CO_TAP_START) | (act == CO_TAP_ACC)) & owner;
    const bool to_y = ((act == CO_TAP_EMIT) | (act == CO_TAP_EMIT_FRESH)) & owner;
    const v4f v = acc[f];
    if constexpr (VEC) {  // M % 4 == 0: a lane's four pixels are all valid or none
      __builtin_amdgcn_raw_buffer_store_b128(
          __builtin_bit_cast(v4u, v), rr, (to_ring & (P0 < ra.M)) ? (e_off[f] + P0) * 4 : kOutOfRange,
          0, 0);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        __builtin_amdgcn_raw_buffer_store_b32(
            __float_as_uint(v[r]), rr,
            (to_ring & (P0 + r < ra.M)) ? (e_off[f] + P0 + r) * 4 : kOutOfRange, 0, 0);
    }
    const int o = e_o[f];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int bq = pb, pq = pp + r;
      if (ra.So >= 4) {  // uniform: four consecutive pixels cross at most one frame edge
        const bool wrap = pq >= ra.So;
        bq += wrap ? 1 : 0;
        pq -= wrap ? ra.So : 0;
      } else {
        bq = fdiv(P0 + r, ra.fd_So);
        pq = P0 + r - bq * ra.So;
      }
      const int yo = ((bq * g.Cout + o) * ra.y_bc + pq) * yesz;
      const int off = (to_y & (P0 + r < ra.M)) ? yo : kOutOfRange;
      const float val = v[r] + e_bias[f];
      if constexpr (sizeof(T) == 2)
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, __bf16(val)), yr, off,
                                              0, 0);
      else
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), yr, off, 0, 0);
    }
  }
}

// Pack W (C_out, C_in, kT, kH, kW) as [fragment][tap][unit][lane] 16-byte
// units, in the order the kernel loads them: an fp32 unit holds channel
// blocks 4cq .. 4cq+3 of one tap (one channel per lane each), a bf16 unit
// holds channel block cq (eight channels per lane); lane (lrow, lgrp) holds
// column n = nf*16 + lrow and the channels the same lane gathers from x.
template <typename T>
__global__ __launch_bounds__(kBlock) void pack_reg_kernel(ConvGeom g, RegConfig c,
                                                          const T* __restrict__ w,
                                                          const float* __restrict__ wscale,
                                                          uint4* __restrict__ out) {
  constexpr bool kBF = sizeof(T) == 2;
  const int ntaps = g.kH * g.kW;
  const int64_t total = int64_t(c.n_frags) * c.U * 64;
  const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const int lane = int(idx % 64);
  int64_t rest = idx / 64;
  const int cq = int(rest % c.CSU);
  rest /= c.CSU;
  const int tp = int(rest % ntaps);
  const int nf = int(rest / ntaps);
  const int n = nf * 16 + (lane & 15), lgrp = lane >> 4;
  const int t = n / g.Cout, o = n - t * g.Cout;
  const int u = tp / g.kW, v = tp - u * g.kW;
  const bool ncol = n < g.kT * g.Cout;
  auto weight = [&](int cb, int c_in) -> T {
    if (!ncol || cb >= c.CS || c_in >= g.Cin) return T(0);
    return scaled_weight<T>(w[(((int64_t(o) * g.Cin + c_in) * g.kT + t) * g.kH + u) * g.kW + v],
                            wscale, o);
  };
  uint32_t word[4] = {0u, 0u, 0u, 0u};
  if constexpr (kBF) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const uint32_t lo = weight(cq, cq * 32 + lgrp * 8 + e);
      const uint32_t hi = weight(cq, cq * 32 + lgrp * 8 + e + 1);
      word[e / 2] = lo | (hi << 16);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int cb = 4 * cq + e;
      word[e] = __float_as_uint(weight(cb, cb * 4 + lgrp));
    }
  }
  out[idx] = make_uint4(word[0], word[1], word[2], word[3]);
}

template <typename T, int WN, int TAPS, int CSMAX, int KSPLIT>
hipError_t reg_launch(const ConvGeom& g, const RegConfig& c, const ConvLayout& L, char* state,
                      const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  RegTaps tt;
  int t_lo = CO_MAX_TAPS, t_hi = -1;
  for (int t = 0; t < CO_MAX_TAPS; ++t) {
    const int sl = plan.slot[t] < 0 ? 0 : plan.slot[t];
    tt.as[t] = int32_t(plan.action[t]) | (sl << 8);
    if (plan.action[t] != CO_TAP_NONE) {
      t_lo = t < t_lo ? t : t_lo;
      t_hi = t;
    }
  }
  if (t_hi < 0) return hipSuccess;
  RegArgs ra;
  ra.M = int32_t(int64_t(g.B) * g.So());
  ra.N = g.kT * g.Cout;
  ra.So = int32_t(g.So());
  ra.m_frags = c.m_frags;
  // only the column fragments holding active taps
  ra.nf0 = (t_lo * g.Cout) / 16;
  const int nf_end = int(ceil_div(int64_t(t_hi + 1) * g.Cout, 16));
  ra.n_grps = int32_t(ceil_div(nf_end - ra.nf0, WN));
  const int64_t blocks = ceil_div(int64_t(ra.m_frags) * ra.n_grps, kRegTiles);
  ra.blocks_per_xcd = int32_t(ceil_div(blocks, 8));
  ra.ntaps = g.kH * g.kW;
  ra.CS = c.CS;
  ra.CSU = c.CSU;
  for (int tp = 0; tp < kRegMaxTaps; ++tp) {
    const int u = tp < ra.ntaps ? tp / g.kW : 0, v = tp < ra.ntaps ? tp % g.kW : 0;
    ra.dh[tp] = u * g.dH;
    ra.dw[tp] = v * g.dW;
  }
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  ra.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * esz);
  ra.w_bytes = int32_t(L.weight_bytes);
  ra.ring_slot = int32_t(L.ring_slot_elems);
  ra.y_bc = int32_t(io.y_bc);
  ra.y_bytes = io.y ? int32_t(((int64_t(g.B) * g.Cout - 1) * io.y_bc + g.So()) * esz) : 0;
  ra.ring_bytes = int32_t(int64_t(g.R) * L.ring_slot_elems * 4);
  ra.fd_So = make_fastdiv(uint32_t(ra.So));
  ra.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  ra.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  ra.fd_ngrps = make_fastdiv(uint32_t(ra.n_grps));
  const bool exact = c.CS == CSMAX && g.Cin % c.CKS == 0;
  auto kern = ra.M % 4 == 0
                  ? (exact ? conv_step_reg_kernel<T, WN, TAPS, CSMAX, KSPLIT, true, true>
                           : conv_step_reg_kernel<T, WN, TAPS, CSMAX, KSPLIT, true, false>)
                  : (exact ? conv_step_reg_kernel<T, WN, TAPS, CSMAX, KSPLIT, false, true>
                           : conv_step_reg_kernel<T, WN, TAPS, CSMAX, KSPLIT, false, false>);
  hipLaunchKernelGGL(kern, dim3(unsigned(8 * ra.blocks_per_xcd)),
                     dim3(64 * KSPLIT * kRegTiles), 0, s, g, ra, static_cast<const T*>(io.x),
                     io.x_bc, static_cast<T*>(io.y), io.y_bc,
                     reinterpret_cast<const uint4*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), tt);
  return hipGetLastError();
}

// ---- persistent forward_steps -------------------------------------------
//
// Temporal stride and dilation 1: at virtual time v = n + pT the arriving
// frame feeds output v - j through temporal tap j, and output v - (kT - 1) is
// complete.  A wave owns 16 output pixels x 16 output channels for every
// temporal tap, so the kT - 1 partial sums it continues are its own: they
// stay in registers for the whole clip (the ring is read at the start and
// written back at the end), and only the frames and the emitted outputs move
// through memory.  Weights stay in registers too.  Per frame and tap the
// products are summed over the k-steps in the order of the step kernel of
// the same instantiation, accumulated onto the partial sum (a split
// instantiation's second half added after), so forward_steps reproduces
// forward_step, and the matrix instructions do the fold.  A
// split instantiation (KSPLIT = 2) runs its two halves on two waves, which
// meet in LDS once per frame: twice the waves, half the serial matrix work
// per wave.
struct RegSteps {
  int32_t M, So, m_frags, o_frags, blocks_per_xcd;
  int32_t ntaps, CS, CSU;
  int32_t dh[kRegMaxTaps], dw[kRegMaxTaps];
  int32_t x_bytes, w_bytes, ring_bytes, ring_slot, y_bytes;
  int32_t fstride;  // bytes between consecutive frames of the clip
  int32_t y_bc;     // elements between (stream, channel) planes of y
  int32_t v0;       // virtual time of the first frame, capped at 2^29
  int32_t slot_v0;  // v0 mod R (uncapped)
  int32_t count, T, k0, update;
  int32_t o_groups;  // STG: workgroups per pixel fragment, ceil(o_frags / staging waves)
  int32_t nseg;      // time segments of the call
  int32_t seg_len;   // frames per segment (the last may be shorter)
  int32_t wgs;       // workgroups per segment
  FastDiv fd_So, fd_Wo, fd_ofr, fd_og;
};

// Waves per SIMD an instantiation is compiled for: two where its registers
// allow it without spilling (the bf16 1x1 shape with two channel blocks, in
// its compile-time form: the runtime-kT form needs more), so that time
// segments can put two waves on every SIMD.
template <typename T, int CSMAX, bool STG, bool FULL>
constexpr int reg_steps_wpe() {
  return (STG && FULL && sizeof(T) == 2 && CSMAX == 2) ? 2 : 1;
}

// STG (1x1 spatial taps, one chain per tile): the waves of a workgroup (4,
// or 8 where two waves share a SIMD) share one 16-pixel fragment and take
// consecutive 16-channel output fragments.  Each frame's input tile (16 pixels x every input
// channel) is gathered once per workgroup -- four consecutive channels of one
// pixel per thread -- and staged channels-last in LDS (double buffered, one
// barrier per frame); each wave reads its operands from there with one
// 16-byte (bf16) or 4-byte (fp32) read per k-step.  Without staging every
// wave gathered the same tile in 2-byte pieces, and the vector L1 stalled on
// the requests.  The operands, and so the results, are the same.
constexpr int kRegStgWaves = 4;
// Staging waves of a stride-1 instantiation: eight where it runs two waves
// per SIMD (a workgroup then fills both, and two workgroups instead of four
// gather each pixel fragment's frames), else kRegStgWaves.
template <typename T, int CSMAX, bool FULL>
constexpr int reg_stg_waves() {
  return reg_steps_wpe<T, CSMAX, true, FULL>() == 2 ? 2 * kRegStgWaves : kRegStgWaves;
}

template <typename T, int TAPS, int CSMAX, int KSPLIT, int KTM, bool FULL, bool STG>
__global__ __launch_bounds__(64 * (STG ? reg_stg_waves<T, CSMAX, FULL>() : KSPLIT * kRegTiles))
__attribute__((amdgpu_waves_per_eu(reg_steps_wpe<T, CSMAX, STG, FULL>(),
                                    reg_steps_wpe<T, CSMAX, STG, FULL>())))
void conv_steps_reg_kernel(ConvGeom g, RegSteps rs, const T* __restrict__ x, int64_t x_bc,
                           T* __restrict__ y, const uint4* __restrict__ wp,
                           const float* __restrict__ bias, float* __restrict__ ring) {
  static_assert(!STG || (TAPS == 1 && KSPLIT == 1), "staging: 1x1 taps, one chain");
  constexpr bool kBF = sizeof(T) == 2;
  constexpr int CL = kBF ? 8 : 1;
  constexpr int CKS = 4 * CL;
  constexpr int CSUMAX = kBF ? CSMAX : (CSMAX + 3) / 4;
  constexpr int TH = TAPS / KSPLIT;  // spatial taps per partial chain
  constexpr int AREGS = TAPS * CSMAX * CL;  // raw registers per frame
  constexpr int PF = AREGS <= 16 ? 4 : 2;  // frames in flight
  using AReg = typename std::conditional<kBF, uint4, float>::type;
  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int bid = int(blockIdx.x);
  int lb = (bid & 7) * rs.blocks_per_xcd + (bid >> 3);
  // Time segment: the clip's frames are dealt to rs.nseg groups of waves.
  // Segment s > 0 starts kT - 1 frames before its first frame s0, with zero
  // partial sums, and stores nothing before s0: every output it stores then
  // took all its taps here, starting from zero at its first tap and adding
  // in frame order, as stepping does, so the bits are the same.  Only
  // segment 0 reads the ring and only the last writes it back.
  const int seg = lb / rs.wgs;  // (wave-uniform, once)
  if (seg >= rs.nseg) return;   // whole workgroups
  lb -= seg * rs.wgs;
  const int s0 = seg * rs.seg_len, s1 = min(rs.count, s0 + rs.seg_len);
  const int tw = seg == 0 ? 0 : s0 - (g.kT - 1);
  // With KSPLIT = 2 the two chains of a tile run on two waves (h = 0 takes
  // spatial taps 0 .. TH - 1, h = 1 the rest); h = 1 hands its products to
  // h = 0 through LDS every frame, and h = 0 adds them exactly as a single
  // wave adds its two chains.  Waves past the last tile keep to the per-frame
  // barrier: they redo tile 0 with every store masked.
  constexpr int TPW = kRegTiles;  // tiles per workgroup
  const int h = STG ? 0 : wave % KSPLIT, wslot = STG ? 0 : wave / KSPLIT;
  int mf, of;
  bool owner;  // the wave that keeps the sums and stores
  if constexpr (STG) {
    // workgroup lb: pixel fragment mf, output fragments kRegStgWaves * group
    // + wave; waves past the last fragment stage and meet the barriers with
    // every store masked (their channels are past C_out)
    if (lb >= rs.m_frags * rs.o_groups) return;  // whole workgroups
    mf = fdiv(lb, rs.fd_og);
    of = (lb - mf * rs.o_groups) * reg_stg_waves<T, CSMAX, FULL>() + wave;
    owner = true;
  } else {
    const int tile_raw = lb * TPW + wslot;
    const bool live = tile_raw < rs.m_frags * rs.o_frags;
    if constexpr (KSPLIT == 1) {
      if (!live) return;  // whole waves; no barrier follows
    }
    const int tile = live ? tile_raw : 0;
    owner = live & (h == 0);
    mf = fdiv(tile, rs.fd_ofr);
    of = tile - mf * rs.o_frags;
  }
  // FULL: the layer uses every temporal tap of the instantiation (kT == KTM),
  // so the per-tap tests below are compile-time and the frame loop is
  // straight-line matrix work with no branch between the instructions
  const int kT = FULL ? KTM : g.kT;

  // ---- weights of this wave's spatial taps, once: column (tap j, channel o)
  // of the step kernel's packing
  const int o = of * 16 + lrow;
  const bool ocol = o < g.Cout;
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(wp, rs.w_bytes);
  const int tp0 = h * TH;  // first spatial tap of this wave's chain
  uint4 wreg[KTM][TH][CSUMAX];
#pragma unroll
  for (int j = 0; j < KTM; ++j) {
    const int n = j * g.Cout + o;
    const int nf = n >> 4, r = n & 15;
#pragma unroll
    for (int i2 = 0; i2 < TH; ++i2)
#pragma unroll
      for (int cq = 0; cq < CSUMAX; ++cq) {
        const int tp = tp0 + i2;
        const bool ok = ocol & (j < kT) & (tp < rs.ntaps) & (cq < rs.CSU);
        const int off = (((nf * rs.ntaps + tp) * rs.CSU + cq) << 10) + (lgrp * 16 + r) * 16;
        const auto w4 = __builtin_amdgcn_raw_buffer_load_b128(wr, ok ? off : kOutOfRange, 0, 0);
        wreg[j][i2][cq] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      }
  }
  // ---- outputs of this lane.  The matrix instructions take the weights as
  // their first operand and the frame as their second (the same registers as
  // the step kernel's, which holds the product transposed), so a lane's
  // results are output channels oc + r, r = 0..3, of pixel Po: an output
  // store then covers 16 consecutive pixels of four channel rows, where the
  // step kernel's layout scattered 2-byte stores over 16 channel rows.
  const int oc = of * 16 + lgrp * 4;
  const int Po = mf * 16 + lrow;
  constexpr uint32_t esz = sizeof(T);
  const __amdgpu_buffer_rsrc_t br = make_rsrc(bias, g.Cout * 4);
  float bo[4];
  int yoff[4];  // byte offset of (b, oc + r, frame 0, p) in y, or out of range
  int roff[4];  // float offset of (oc + r, Po) inside a ring slot, or -1
  {
    const bool pok = (Po < rs.M) & owner;
    const int b = fdiv(pok ? Po : 0, rs.fd_So), p = (pok ? Po : 0) - b * rs.So;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int orow = oc + r;
      const bool ok = pok & (orow < g.Cout);
      bo[r] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(br, orow < g.Cout ? orow * 4 : kOutOfRange, 0, 0));
      yoff[r] = ok ? int((uint32_t(b * g.Cout + orow) * uint32_t(rs.y_bc) + uint32_t(p)) * esz)
                   : kOutOfRange;
      roff[r] = ok ? orow * rs.M + Po : -1;
    }
  }
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, rs.y_bytes);
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(ring, rs.ring_bytes);
  const int R = g.R;

  // ---- partial sums: part[j] continues output v - j (1 <= j <= kT - 1)
  v4f part[KTM];
#pragma unroll
  for (int j = 1; j < KTM; ++j) {
    part[j] = v4f{0.f, 0.f, 0.f, 0.f};
    const int tau = rs.v0 - j;
    if (seg == 0 && j < kT && tau >= 0) {  // uniform
      const int sl = (rs.slot_v0 - j + R) % R;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        part[j][r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            rr, roff[r] >= 0 ? (sl * rs.ring_slot + roff[r]) * 4 : kOutOfRange, 0, 0));
    }
  }

  // ---- operand gathers of one frame (as in the step kernel; the frame
  // offset rides in the wave-uniform scalar operand)
  const int P = mf * 16 + lrow;
  const bool pvalid = P < rs.M;
  const int Pc = pvalid ? P : 0;
  const int b = fdiv(Pc, rs.fd_So), p = Pc - b * rs.So;
  const int i = fdiv(p, rs.fd_Wo), jw = p - i * g.Wo;
  const int hb = i * g.sH - g.pH, wb = jw * g.sW - g.pW;
  const int lane_c = lgrp * CL;
  const uint32_t plane_b = uint32_t(x_bc) * esz;
  const uint32_t lane_b = (uint32_t(b) * uint32_t(g.Cin) + uint32_t(lane_c)) * plane_b;
  const int nv_last = min(max(g.Cin - ((rs.CS - 1) * CKS + lane_c), 0), CL);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, rs.x_bytes);
  int vt[TH];
#pragma unroll
  for (int i2 = 0; i2 < TH; ++i2) {
    const int tp = tp0 + i2;
    const int hi = hb + rs.dh[tp], wi = wb + rs.dw[tp];
    const bool ok = (tp < rs.ntaps) & pvalid & (unsigned(hi) < unsigned(g.H)) &
                    (unsigned(wi) < unsigned(g.W));
    vt[i2] = ok ? int(lane_b + (uint32_t(hi) * uint32_t(g.W) + uint32_t(wi)) * esz) : kOutOfRange;
  }
  // Raw loaded bits (eight bf16 channels or one fp32 per lane and k-step),
  // packed into operands only when the frame is multiplied: packing right
  // after the loads would make the wave wait for them there.  Frames past
  // the clip (end padding, or past the call) issue the same loads at the
  // out-of-range offset, which return zero: every frame issues the same
  // memory operations, so the compiler's count of those in flight stays
  // exact around the frame loop and no wait covers more than its own frame.
  auto load_frame = [&](int t, uint32_t (&a)[TH][CSMAX][CL]) {
    const bool real = t < rs.T;  // uniform
    const int fo = real ? t * rs.fstride : 0;
#pragma unroll
    for (int i2 = 0; i2 < TH; ++i2)
#pragma unroll
      for (int cb = 0; cb < CSMAX; ++cb) {
        const bool lv = real & (cb < rs.CS), last = cb == rs.CS - 1;  // uniform
        const int sb = int(uint32_t(cb * CKS) * plane_b) + fo;
#pragma unroll
        for (int e = 0; e < CL; ++e) {
          const int v = (lv & (!last | (e < nv_last))) ? vt[i2] : kOutOfRange;
          a[i2][cb][e] = load_raw_at<T>(xr, v, sb + int(uint32_t(e) * plane_b));
        }
      }
  };
  auto operand = [&](const uint32_t (&r)[CL]) -> AReg {
    if constexpr (kBF)
      return make_uint4(r[0] | (r[1] << 16), r[2] | (r[3] << 16), r[4] | (r[5] << 16),
                        r[6] | (r[7] << 16));
    else
      return __uint_as_float(r[0]);
  };

  // ---- staging (STG): thread (px, q) gathers channels CPT (q + TQ k) ..
  // + CPT - 1 of pixel mf * 16 + px (TQ: the workgroup's threads over its 16
  // pixels); out-of-range reads (pixels past M, channels past C_in, frames
  // past the clip) return zero
  constexpr int SCH = CSMAX * CKS;            // staged channels (upper bound)
  constexpr int TQ = 4 * (STG ? reg_stg_waves<T, CSMAX, FULL>() : 1);  // unit slots
  // channels per thread and unit: four, or two where four would leave threads
  // without a unit (bf16: 64 channels over the 32 slots of eight waves)
  constexpr int CPT = (kBF && SCH / 4 < TQ) ? 2 : 4;
  constexpr int SQ = (SCH / CPT + TQ - 1) / TQ;  // units per thread
  constexpr int PU = SCH * int(esz) / 16 + 1;  // LDS row pitch, 16-byte units
  constexpr int SPF0 = SQ <= 2 ? 4 : 2;
  // frames per group: whole periods of the partial sums' rotation, so a
  // group ends with every sum back in the register it started in; frames in
  // flight: the group, or where two waves share a SIMD (registers for two) a
  // divisor of it, at most SPF0
  constexpr int FPG_S = KTM * ((SPF0 + KTM - 1) / KTM);
  // (two channels per staging thread leave registers for the whole group:
  // vector memory operations complete in issue order, so a frame's wait
  // for its staged loads also waits for every output store issued before
  // them, and loads issued a whole group ahead put that wait on stores a
  // group old)
  constexpr int SPF = !STG                                  ? 1
                      : reg_steps_wpe<T, CSMAX, STG, FULL>() == 1 ? FPG_S
                      : CPT == 2                            ? FPG_S
                      : FPG_S % 4 == 0                      ? 4
                      : FPG_S % 3 == 0                      ? 3
                      : FPG_S % 2 == 0                      ? 2
                                                            : FPG_S;
  __shared__ uint4 stg[STG ? 2 : 1][STG ? 16 * PU : 1];
  uint32_t sraw[SPF][STG ? SQ : 1][CPT];
  const int tid = int(threadIdx.x);
  const int spx = tid & 15, sq0 = tid >> 4;
  const int Ps = mf * 16 + spx;
  const bool ps_ok = Ps < rs.M;
  const int sb = fdiv(ps_ok ? Ps : 0, rs.fd_So), sp = (ps_ok ? Ps : 0) - sb * rs.So;
  const uint32_t s_base = uint32_t(sb) * uint32_t(g.Cin) * plane_b + uint32_t(sp) * esz;
  auto load_stage = [&](int t, uint32_t (&a)[STG ? SQ : 1][CPT]) {
    const bool real = t < rs.T;  // uniform
    const int fo = real ? t * rs.fstride : 0;
#pragma unroll
    for (int k = 0; k < SQ; ++k) {
      const int qd = sq0 + TQ * k;
#pragma unroll
      for (int e = 0; e < CPT; ++e) {
        const int c = CPT * qd + e;
        const bool ok = real & ps_ok & (c < g.Cin);
        a[k][e] = load_raw_at<T>(xr, ok ? int(s_base + uint32_t(c) * plane_b) : kOutOfRange, fo);
      }
    }
  };
  auto write_stage = [&](int buf, const uint32_t (&a)[STG ? SQ : 1][CPT]) {
    // every unit of the row, also those past C_in (the k-steps past the
    // layer's multiply them, as zeros, by zero weights)
    uint4* row = &stg[buf][spx * PU];
#pragma unroll
    for (int k = 0; k < SQ; ++k) {
      const int qd = sq0 + TQ * k;
      // (a compile-time test where the units fill the threads: a divergent
      // branch here would split the frame loop into blocks)
      if ((SCH / CPT) % TQ == 0 || qd < SCH / CPT) {
        if constexpr (kBF && CPT == 2)
          reinterpret_cast<uint32_t*>(row)[qd] = a[k][0] | (a[k][1] << 16);
        else if constexpr (kBF)
          reinterpret_cast<uint2*>(row)[qd] =
              make_uint2(a[k][0] | (a[k][1] << 16), a[k][2] | (a[k][3] << 16));
        else
          row[qd] = make_uint4(a[k][0], a[k][1], a[k][2], a[k][3]);
      }
    }
  };
  auto staged_operand = [&](int buf, int cb) -> AReg {
    const uint4* row = &stg[buf][lrow * PU];
    if constexpr (kBF)
      return row[cb * 4 + lgrp];
    else
      return reinterpret_cast<const float*>(row)[cb * 4 + lgrp];
  };

  uint32_t araw[STG ? 1 : PF][TH][CSMAX][CL];
  // products handed from chain 1 to chain 0: [tile][frame parity][tap j][lane]
  __shared__ v4f red[KSPLIT == 2 ? TPW : 1][2][KSPLIT == 2 ? KTM : 1][64];
  // in frame order (the loop below waits for frame u's loads with the later
  // frames' still in flight)
  // STG: operands of the frame being multiplied, read from LDS after the
  // previous frame's barrier
  AReg aq[STG ? CSMAX : 1];
  if constexpr (STG) {
#pragma unroll
    for (int u = 0; u < SPF; ++u) {
      load_stage(tw + u, sraw[u]);
      __builtin_amdgcn_sched_barrier(0);
    }
    write_stage(tw & 1, sraw[0]);
    load_stage(tw + SPF, sraw[0]);
    __syncthreads();
#pragma unroll
    for (int cb = 0; cb < CSMAX; ++cb) aq[cb] = staged_operand(tw & 1, cb);
  } else {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      load_frame(tw + u, araw[u]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  constexpr int FPG = STG ? FPG_S : PF;  // frames per group

  // Whole groups of PF frames, with no exit inside a group: frames past the
  // call (the last group's tail) run with their stores dropped and the
  // partial sums left as they are.
  // One frame.  In a steady group (STG only: every frame inside the call,
  // every temporal tap continuing an output that started on a real frame)
  // the fold needs no selects; the general form handles the stream's first
  // frames, end padding and the call's last group.  Both issue the same
  // memory operations in the same order.
  auto frame = [&](int t0, int u, auto steady_tag) {
    constexpr bool STEADY = decltype(steady_tag)::value;
    const int t = t0 + u;
    const bool dead = STEADY ? false : t >= s1;  // uniform
    const int v = rs.v0 + t;
    // every temporal tap's chain of k-steps, accumulated onto the sum it
    // continues (zero for an output that starts, and on a split tile's
    // second chain)
    v4f c[KTM];
#pragma unroll
    for (int j = 0; j < KTM; ++j) {
      const int first = STEADY ? 0 : (v - j >= g.pT ? 0 : g.pT - (v - j));
      c[j] = (h == 0 && j != 0 && j != first) ? part[j] : v4f{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i2 = 0; i2 < TH; ++i2)
#pragma unroll
      for (int cb = 0; cb < CSMAX; ++cb)
#pragma unroll
        for (int j = 0; j < KTM; ++j) {
          if (!FULL && j >= kT) continue;  // uniform
          AReg av;
          if constexpr (STG)
            av = aq[cb];
          else
            av = operand(araw[u][i2][cb]);
          if constexpr (kBF) {
            c[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(v8bf, wreg[j][i2][cb]), __builtin_bit_cast(v8bf, av), c[j],
                0, 0, 0);
          } else {
            const uint4 u4 = wreg[j][i2][cb / 4];
            const uint32_t bw = (cb & 3) == 0 ? u4.x : (cb & 3) == 1 ? u4.y : (cb & 3) == 2 ? u4.z : u4.w;
            c[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bw), av, c[j], 0, 0, 0);
          }
        }
    // the next frames' operands are requested before this frame's epilogue
    if constexpr (!STG) load_frame(t + PF, araw[u]);
    if constexpr (STG) {
      // frame t + 1 into LDS buffer (t + 1) & 1 (every wave read frame t - 1
      // from it before the previous barrier), frame t + 1 + SPF's gathers,
      // and after the barrier frame t + 1's operands: their LDS latency runs
      // under this frame's matrix work and epilogue
      const int un = (u + 1) % SPF;
      write_stage((t + 1) & 1, sraw[un]);
      load_stage(t + 1 + SPF, sraw[un]);
      __syncthreads();
#pragma unroll
      for (int cb = 0; cb < CSMAX; ++cb) aq[cb] = staged_operand((t + 1) & 1, cb);
    }
    v4f c1[KTM];  // chain 1's products (KSPLIT = 2), as chain 0 adds them
    if constexpr (KSPLIT == 2) {
      if (h == 1) {
#pragma unroll
        for (int j = 0; j < KTM; ++j) red[wslot][t & 1][j][lane] = c[j];
      }
      __syncthreads();  // (a slot is rewritten two frames later, after another barrier)
      // Both waves run the fold below: the helper's stores carry the
      // out-of-range offset and are dropped.  A branch around it would
      // give the two paths different counts of outstanding memory
      // operations, and the compiler would then wait for all of them
      // (the frames in flight included) before each frame's products.
#pragma unroll
      for (int j = 0; j < KTM; ++j) c1[j] = red[wslot][t & 1][j][lane];
    }
    // tap j completes output v - (kT - 1); the others carry on
    v4f nxt[KTM];
#pragma unroll
    for (int j = 0; j < KTM; ++j) {
      nxt[j] = v4f{0.f, 0.f, 0.f, 0.f};
      if (!FULL && j >= kT) continue;
      // output v - j exists once tau >= 0 (a uniform select, no branch:
      // the stores of a missing output carry the out-of-range offset)
      const int tau = v - j;
      const bool exists = STEADY ? true : (tau >= 0) & !dead;
      // (a segment's warm-up frames keep their sums but store nothing)
      const bool stores = STEADY ? true : exists & (t >= s0);
      v4f a = c[j];
      if constexpr (KSPLIT == 2) a = a + c1[j];
      if (j == kT - 1) {
        const int fo = stores ? (rs.k0 + t) * rs.So * int(esz) : 0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float val = a[r] + bo[r];
          const int yo = stores ? yoff[r] : kOutOfRange;
          if constexpr (kBF)
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, __bf16(val)),
                                                  yr, yo, fo, 0);
          else
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), yr, yo, fo, 0);
        }
      } else {
        nxt[j] = exists ? a : v4f{0.f, 0.f, 0.f, 0.f};
      }
    }
    // output v - j continues as v + 1 - (j + 1)
#pragma unroll
    for (int j = KTM - 1; j >= 1; --j) part[j] = dead ? part[j] : nxt[j - 1];
    // keep the frames in order: hoisting the next frame's matrix work
    // above this frame's loads would make it wait for operands requested
    // only just before, instead of PF frames earlier
    __builtin_amdgcn_sched_barrier(0);
  };
  for (int t0 = tw; t0 < s1; t0 += FPG) {
    // uniform: the outputs v - j of every frame of the group started at or
    // after the first real frame
    const bool steady = (rs.v0 + t0 >= g.pT + kT - 1) & (t0 >= s0) & (t0 + FPG <= s1);
    if constexpr (STG) {
      if (steady) {
#pragma unroll
        for (int u = 0; u < FPG; ++u) frame(t0, u, std::true_type{});
        continue;
      }
    }
#pragma unroll
    for (int u = 0; u < FPG; ++u) frame(t0, u, std::false_type{});
  }

  if (rs.update && h == 0 && s1 == rs.count) {
    const int v1 = rs.v0 + rs.count;
    const int slot1 = (rs.slot_v0 + rs.count) % R;
#pragma unroll
    for (int j = 1; j < KTM; ++j) {
      const int tau = v1 - j;
      if (j < kT && tau >= 0) {  // uniform
        const int sl = (slot1 - j + R) % R;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          __builtin_amdgcn_raw_buffer_store_b32(
              __float_as_uint(part[j][r]), rr,
              roff[r] >= 0 ? (sl * rs.ring_slot + roff[r]) * 4 : kOutOfRange, 0, 0);
      }
    }
  }
}

// Temporal stride or dilation above 1 (Principle 5) on the staged 1x1
// shapes.  Which output a tap feeds, and whether it starts, continues or
// completes it, depends on the frame, so the frame loop follows the host's
// step plans (a PlanTable: explicit for a stream's first frames, periodic
// after).  A lane's R partial sums (four output channels of one pixel) sit
// in LDS and are addressed by the plan's slot; per tap the arithmetic is the
// step kernel's: the matrix chain accumulates onto the slot (ACC, EMIT) or
// zero (START, EMIT_FRESH), and the sum goes back to the slot or out with the
// bias.  The ring's R slots are read once and written back once, stale ones
// included.  Time segments start rp.warm frames early, enough for every
// output they store to take all its taps inside the segment and for every
// slot to start afresh inside the last one.
struct RegPlan {
  PlanTable pt;
  int32_t warm;  // warm-up frames of a segment after the first
  int32_t t_e0;  // first emitting frame of the call (count if none)
};

template <typename T, int CSMAX, int KTM>
__global__ __launch_bounds__(64 * kRegStgWaves)
void conv_steps_regp_kernel(ConvGeom g, RegSteps rs, RegPlan rp, const T* __restrict__ x,
                            int64_t x_bc, T* __restrict__ y, const uint4* __restrict__ wp,
                            const float* __restrict__ bias, float* __restrict__ ring) {
  constexpr bool kBF = sizeof(T) == 2;
  constexpr int CL = kBF ? 8 : 1;
  constexpr int CKS = 4 * CL;
  constexpr int CSUMAX = kBF ? CSMAX : (CSMAX + 3) / 4;
  constexpr uint32_t esz = sizeof(T);
  using AReg = typename std::conditional<kBF, uint4, float>::type;
  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int bid = int(blockIdx.x);
  int lb = (bid & 7) * rs.blocks_per_xcd + (bid >> 3);
  const int seg = lb / rs.wgs;
  if (seg >= rs.nseg) return;  // whole workgroups
  lb -= seg * rs.wgs;
  if (lb >= rs.m_frags * rs.o_groups) return;
  const int s0 = seg * rs.seg_len, s1 = min(rs.count, s0 + rs.seg_len);
  const int tw = seg == 0 ? 0 : s0 - rp.warm;
  const int mf = fdiv(lb, rs.fd_og);
  const int of = (lb - mf * rs.o_groups) * kRegStgWaves + wave;
  const int kT = g.kT;

  // ---- weights, as in the kernel above (one spatial tap)
  const int o = of * 16 + lrow;
  const bool ocol = o < g.Cout;
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(wp, rs.w_bytes);
  uint4 wreg[KTM][CSUMAX];
#pragma unroll
  for (int j = 0; j < KTM; ++j) {
    const int n = j * g.Cout + o;
    const int nf = n >> 4, r = n & 15;
#pragma unroll
    for (int cq = 0; cq < CSUMAX; ++cq) {
      const bool ok = ocol & (j < kT) & (cq < rs.CSU);
      const int off = ((nf * rs.CSU + cq) << 10) + (lgrp * 16 + r) * 16;
      const auto w4 = __builtin_amdgcn_raw_buffer_load_b128(wr, ok ? off : kOutOfRange, 0, 0);
      wreg[j][cq] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
    }
  }
  // ---- outputs of this lane: channels oc + r of pixel Po
  const int oc = of * 16 + lgrp * 4;
  const int Po = mf * 16 + lrow;
  const __amdgpu_buffer_rsrc_t br = make_rsrc(bias, g.Cout * 4);
  float bo[4];
  int yoff[4], roff[4];
  {
    const bool pok = Po < rs.M;
    const int b = fdiv(pok ? Po : 0, rs.fd_So), p = (pok ? Po : 0) - b * rs.So;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int orow = oc + r;
      const bool ok = pok & (orow < g.Cout);
      bo[r] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(br, orow < g.Cout ? orow * 4 : kOutOfRange, 0, 0));
      yoff[r] = ok ? int((uint32_t(b * g.Cout + orow) * uint32_t(rs.y_bc) + uint32_t(p)) * esz)
                   : kOutOfRange;
      roff[r] = ok ? orow * rs.M + Po : -1;
    }
  }
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, rs.y_bytes);
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(ring, rs.ring_bytes);

  // ---- partial sums: slot q of this lane at pp[q * 64]
  __shared__ v4f parts[kRegStgWaves][kPlanMaxR][64];
  v4f* const pp = &parts[wave][0][lane];
  if (seg == 0) {
    for (int q = 0; q < g.R; ++q) {
      v4f a;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        a[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            rr, roff[r] >= 0 ? (q * rs.ring_slot + roff[r]) * 4 : kOutOfRange, 0, 0));
      pp[q * 64] = a;
    }
  }

  // ---- staging: each frame's 16-pixel tile, channels-last in LDS, double
  // buffered, as in the kernel above
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, rs.x_bytes);
  const uint32_t plane_b = uint32_t(x_bc) * esz;
  constexpr int SCH = CSMAX * CKS;
  constexpr int TQ = 4 * kRegStgWaves;  // quad slots: threads / 16 pixels
  constexpr int SQ = (SCH / 4 + TQ - 1) / TQ;
  constexpr int PU = SCH * int(esz) / 16 + 1;
  constexpr int SPF = SQ <= 2 ? 4 : 2;  // frames in flight
  __shared__ uint4 stg[2][16 * PU];
  uint32_t sraw[SPF][SQ][4];
  const int tid = int(threadIdx.x);
  const int spx = tid & 15, sq0 = tid >> 4;
  const int Ps = mf * 16 + spx;
  const bool ps_ok = Ps < rs.M;
  const int sb = fdiv(ps_ok ? Ps : 0, rs.fd_So), sp = (ps_ok ? Ps : 0) - sb * rs.So;
  const uint32_t s_base = uint32_t(sb) * uint32_t(g.Cin) * plane_b + uint32_t(sp) * esz;
  auto load_stage = [&](int t, uint32_t (&a)[SQ][4]) {
    const bool real = t < rs.T;  // uniform
    const int fo = real ? t * rs.fstride : 0;
#pragma unroll
    for (int k = 0; k < SQ; ++k) {
      const int qd = sq0 + TQ * k;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = 4 * qd + e;
        const bool ok = real & ps_ok & (c < g.Cin);
        a[k][e] = load_raw_at<T>(xr, ok ? int(s_base + uint32_t(c) * plane_b) : kOutOfRange, fo);
      }
    }
  };
  auto write_stage = [&](int buf, const uint32_t (&a)[SQ][4]) {
    uint4* row = &stg[buf][spx * PU];
#pragma unroll
    for (int k = 0; k < SQ; ++k) {
      const int qd = sq0 + TQ * k;
      if ((SCH / 4) % TQ == 0 || qd < SCH / 4) {
        if constexpr (kBF)
          reinterpret_cast<uint2*>(row)[qd] =
              make_uint2(a[k][0] | (a[k][1] << 16), a[k][2] | (a[k][3] << 16));
        else
          row[qd] = make_uint4(a[k][0], a[k][1], a[k][2], a[k][3]);
      }
    }
  };
  auto staged_operand = [&](int buf, int cb) -> AReg {
    const uint4* row = &stg[buf][lrow * PU];
    if constexpr (kBF)
      return row[cb * 4 + lgrp];
    else
      return reinterpret_cast<const float*>(row)[cb * 4 + lgrp];
  };
  AReg aq[CSMAX];
#pragma unroll
  for (int u = 0; u < SPF; ++u) {
    load_stage(tw + u, sraw[u]);
    __builtin_amdgcn_sched_barrier(0);
  }
  write_stage(tw & 1, sraw[0]);
  load_stage(tw + SPF, sraw[0]);
  __syncthreads();
#pragma unroll
  for (int cb = 0; cb < CSMAX; ++cb) aq[cb] = staged_operand(tw & 1, cb);

  // plan position and emission count at frame tw
  int ph = tw > rp.pt.n_start ? (tw - rp.pt.n_start) % rp.pt.period : 0;
  int k = tw > rp.t_e0 ? (tw - rp.t_e0 + g.sT - 1) / g.sT : 0;
  uint32_t touched = 0;  // slots written in this segment (uniform)
  auto frame = [&](int t, int u) {
    const bool dead = t >= s1;  // workgroup-uniform
    uint64_t code = 0;
    if (!dead) {
      if (t < rp.pt.n_start) {
        code = rp.pt.code_start[t];
      } else {
        code = rp.pt.code_period[ph];
        ph = ph + 1 == rp.pt.period ? 0 : ph + 1;
      }
    }
    const bool stores = t >= s0;  // (a segment's warm-up frames store nothing)
    bool emitted = false;
#pragma unroll
    for (int j = 0; j < KTM; ++j) {
      if (j >= kT) break;  // uniform
      const int act = int(code >> (6 * j)) & 7, sl = int(code >> (6 * j + 3)) & 7;
      if (act == CO_TAP_NONE) continue;  // uniform
      v4f c = (act == CO_TAP_ACC || act == CO_TAP_EMIT) ? pp[sl * 64] : v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cb = 0; cb < CSMAX; ++cb) {
        if constexpr (kBF) {
          c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, wreg[j][cb]),
                                                      __builtin_bit_cast(v8bf, aq[cb]), c, 0, 0, 0);
        } else {
          const uint4 u4 = wreg[j][cb / 4];
          const uint32_t bw = (cb & 3) == 0 ? u4.x : (cb & 3) == 1 ? u4.y : (cb & 3) == 2 ? u4.z : u4.w;
          c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bw), aq[cb], c, 0, 0, 0);
        }
      }
      if (act == CO_TAP_EMIT || act == CO_TAP_EMIT_FRESH) {
        const int fo = stores ? k * rs.So * int(esz) : 0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float val = c[r] + bo[r];
          const int yo = stores ? yoff[r] : kOutOfRange;
          if constexpr (kBF)
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, __bf16(val)), yr,
                                                  yo, fo, 0);
          else
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), yr, yo, fo, 0);
        }
        emitted = true;
      } else {
        pp[sl * 64] = c;
        touched |= 1u << sl;
      }
    }
    if (emitted) ++k;
    // frame t + 1 into LDS (as in the kernel above)
    const int un = (u + 1) % SPF;
    write_stage((t + 1) & 1, sraw[un]);
    load_stage(t + 1 + SPF, sraw[un]);
    __syncthreads();
#pragma unroll
    for (int cb = 0; cb < CSMAX; ++cb) aq[cb] = staged_operand((t + 1) & 1, cb);
  };
  for (int t0 = tw; t0 < s1; t0 += SPF) {
#pragma unroll
    for (int u = 0; u < SPF; ++u) frame(t0 + u, u);
  }

  // (a later segment's untouched slots hold nothing it read: with kT = 1
  // no slot is ever written, and otherwise every slot starts afresh in it)
  if (rs.update && s1 == rs.count) {
    for (int q = 0; q < g.R; ++q) {
      if (seg != 0 && !((touched >> q) & 1)) continue;  // uniform
      const v4f a = pp[q * 64];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        __builtin_amdgcn_raw_buffer_store_b32(
            __float_as_uint(a[r]), rr, roff[r] >= 0 ? (q * rs.ring_slot + roff[r]) * 4 : kOutOfRange,
            0, 0);
    }
  }
}

// Instantiations: (step-kernel shape id, largest kT).  Registers hold
// kT x taps x channel blocks of weights, so deep temporal kernels go with
// 1x1 spatial taps only.
struct RegStepsShape {
  int32_t cfg, ktm;
};
// (Step shapes 7 and 8 hold too many operand registers to add weights for
// even three temporal taps without spilling; their forward_steps loop over
// single steps.)
constexpr RegStepsShape kRegStepsShapes[] = {
    {0, 3}, {0, 9}, {1, 3}, {2, 3}, {3, 3}, {4, 3}, {5, 3}, {5, 9}, {6, 3}, {6, 9}, {9, 3},
};

int reg_steps_ktm(const ConvGeom& g) {
  int best = 0;
  for (const auto& sh : kRegStepsShapes)
    if (sh.cfg == g.cfg && g.kT <= sh.ktm && (best == 0 || sh.ktm < best)) best = sh.ktm;
  return best;
}

template <typename T, int TAPS, int CSMAX, int KSPLIT, int KTM>
hipError_t reg_steps_launch(const ConvGeom& g, const RegConfig& c, const ConvLayout& L,
                            char* state, const void* x, int64_t x_bc, int32_t nreal,
                            int32_t count, void* y, int64_t y_bc, int64_t n0, bool update,
                            hipStream_t s) {
  RegSteps rs;
  rs.M = int32_t(int64_t(g.B) * g.So());
  rs.So = int32_t(g.So());
  rs.m_frags = c.m_frags;
  rs.o_frags = int32_t(ceil_div(g.Cout, 16));
  const int64_t blocks = ceil_div(int64_t(rs.m_frags) * rs.o_frags, kRegTiles);
  rs.blocks_per_xcd = int32_t(ceil_div(blocks, 8));
  rs.ntaps = g.kH * g.kW;
  rs.CS = c.CS;
  rs.CSU = c.CSU;
  for (int tp = 0; tp < kRegMaxTaps; ++tp) {
    const int u = tp < rs.ntaps ? tp / g.kW : 0, v = tp < rs.ntaps ? tp % g.kW : 0;
    rs.dh[tp] = u * g.dH;
    rs.dw[tp] = v * g.dW;
  }
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  rs.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * x_bc + int64_t(nreal) * g.S()) * esz);
  rs.w_bytes = int32_t(L.weight_bytes);
  rs.ring_slot = int32_t(L.ring_slot_elems);
  rs.ring_bytes = int32_t(int64_t(g.R) * L.ring_slot_elems * 4);
  rs.y_bytes = int32_t(int64_t(g.B) * g.Cout * y_bc * esz);
  rs.fstride = int32_t(g.S() * esz);
  rs.y_bc = int32_t(y_bc);
  const int64_t v0 = n0 + g.pT;
  rs.v0 = int32_t(v0 < (int64_t(1) << 29) ? v0 : (int64_t(1) << 29));
  rs.slot_v0 = int32_t(v0 % g.R);
  rs.count = count;
  rs.T = nreal;
  rs.k0 = int32_t(n0 - (n0 > g.d ? n0 : g.d));
  rs.update = update ? 1 : 0;
  rs.fd_So = make_fastdiv(uint32_t(rs.So));
  rs.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  rs.fd_ofr = make_fastdiv(uint32_t(rs.o_frags));
  constexpr bool STG = TAPS == 1 && KSPLIT == 1;
  // staging waves per workgroup: the plan-driven kernel's, or the stride-1
  // instantiation's that this call runs
  const bool plan = STG && (g.sT != 1 || g.dT != 1);
  const int sw = plan || !STG ? kRegStgWaves
                 : g.kT == KTM ? reg_stg_waves<T, CSMAX, true>()
                               : reg_stg_waves<T, CSMAX, false>();
  rs.o_groups = int32_t(ceil_div(rs.o_frags, sw));
  rs.fd_og = make_fastdiv(uint32_t(rs.o_groups));
  // time segments: as many as keep every wave resident at the waves per
  // SIMD the instantiation is compiled for (1024 SIMDs), with each
  // segment's warm-up (kT - 1 frames) at most a quarter of its frames
  const int64_t wgs = STG ? int64_t(rs.m_frags) * rs.o_groups : blocks;
  const int64_t waves = wgs * (STG ? sw : KSPLIT * kRegTiles);
  constexpr int64_t kSimds = 1024;
  const int wpe = g.kT == KTM ? reg_steps_wpe<T, CSMAX, STG, true>()
                              : reg_steps_wpe<T, CSMAX, STG, false>();
  int64_t nseg = (wpe * kSimds) / std::max<int64_t>(waves, 1);
  if (g.kT > 1) nseg = std::min<int64_t>(nseg, count / (4 * (g.kT - 1)));
  nseg = std::max<int64_t>(1, std::min<int64_t>(nseg, 64));
  rs.seg_len = int32_t(ceil_div(count, nseg));
  rs.nseg = int32_t(ceil_div(count, rs.seg_len));
  rs.wgs = int32_t(wgs);
  rs.blocks_per_xcd = int32_t(ceil_div(wgs * rs.nseg, 8));
  if constexpr (STG) {
    if (g.sT != 1 || g.dT != 1) {
      // plan-driven: segments take max((kT - 1) dT, sT R) warm-up frames and
      // hold at least four times as many
      RegPlan rp;
      plan_table(g, n0, count, &rp.pt);
      rp.warm = std::max((g.kT - 1) * g.dT, g.sT * g.R);
      const int64_t te = n0 >= g.d ? (g.sT - (n0 - g.d) % g.sT) % g.sT : g.d - n0;
      rp.t_e0 = int32_t(std::min<int64_t>(te, count));
      // (every instantiation fits two waves per SIMD)
      int64_t ns = (2 * kSimds) / std::max<int64_t>(wgs * kRegStgWaves, 1);
      ns = std::min<int64_t>(ns, count / (4 * int64_t(rp.warm)));
      ns = std::max<int64_t>(1, std::min<int64_t>(ns, 64));
      rs.seg_len = int32_t(ceil_div(count, ns));
      rs.nseg = int32_t(ceil_div(count, rs.seg_len));
      rs.blocks_per_xcd = int32_t(ceil_div(wgs * rs.nseg, 8));
      hipLaunchKernelGGL((conv_steps_regp_kernel<T, CSMAX, KTM>),
                         dim3(unsigned(8 * rs.blocks_per_xcd)), dim3(64 * kRegStgWaves), 0, s, g,
                         rs, rp, static_cast<const T*>(x), x_bc, static_cast<T*>(y),
                         reinterpret_cast<const uint4*>(state + L.weight),
                         reinterpret_cast<const float*>(state + L.bias),
                         reinterpret_cast<float*>(state + L.ring));
      return hipGetLastError();
    }
  }
  auto kern = g.kT == KTM ? conv_steps_reg_kernel<T, TAPS, CSMAX, KSPLIT, KTM, true, STG>
                          : conv_steps_reg_kernel<T, TAPS, CSMAX, KSPLIT, KTM, false, STG>;
  hipLaunchKernelGGL(kern, dim3(unsigned(8 * rs.blocks_per_xcd)),
                     dim3(64 * (STG ? sw : KSPLIT * kRegTiles)),
                     0, s, g, rs, static_cast<const T*>(x), x_bc, static_cast<T*>(y),
                     reinterpret_cast<const uint4*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring));
  return hipGetLastError();
}

}  // namespace

bool reg_step_needs_staging(const ConvGeom& g, const StepIO& io) {
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  return ((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * esz >= (int64_t(1) << 31) ||
         (io.y && ((int64_t(g.B) * g.Cout - 1) * io.y_bc + g.So()) * esz >= (int64_t(1) << 31));
}

hipError_t launch_conv_step_reg(const ConvGeom& g, const ConvLayout& L, char* state,
                                const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  RegConfig c;
  if (!reg_config(g, g.cfg, &c)) return hipErrorInvalidValue;
  // 32-bit buffer offsets: the packed weights, the tile count and the ring
  // are held in reach when the algorithm is chosen; the reach of a frame
  // depends on its plane and output strides
  if (L.weight_bytes >= (int64_t(1) << 30) || int64_t(c.m_frags) * c.n_frags >= (int64_t(1) << 30) ||
      int64_t(g.R) * L.ring_slot_elems * 4 >= (int64_t(1) << 31))
    return hipErrorInvalidValue;
  if (reg_step_needs_staging(g, io)) return launch_conv_step_staged(g, L, state, io, plan, s);
  switch (c.id) {
    case 0: return reg_launch<float, 4, 1, 16, 1>(g, c, L, state, io, plan, s);
    case 1: return reg_launch<float, 2, 1, 32, 1>(g, c, L, state, io, plan, s);
    case 2: return reg_launch<float, 1, 9, 6, 1>(g, c, L, state, io, plan, s);
    case 3: return reg_launch<float, 2, 9, 3, 1>(g, c, L, state, io, plan, s);
    case 4: return reg_launch<float, 1, 5, 6, 2>(g, c, L, state, io, plan, s);
    case 5: return reg_launch<bf16_t, 4, 1, 2, 1>(g, c, L, state, io, plan, s);
    case 6: return reg_launch<bf16_t, 2, 1, 4, 1>(g, c, L, state, io, plan, s);
    case 7: return reg_launch<bf16_t, 1, 1, 16, 1>(g, c, L, state, io, plan, s);
    case 8: return reg_launch<bf16_t, 1, 9, 2, 1>(g, c, L, state, io, plan, s);
    case 9: return reg_launch<bf16_t, 2, 9, 1, 1>(g, c, L, state, io, plan, s);
    default: return hipErrorInvalidValue;
  }
}

bool reg_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames) {
  if (g.algo != CO_ALGO_GEMM_REG || reg_steps_ktm(g) == 0) return false;
  RegConfig c;
  if (!reg_config(g, g.cfg, &c)) return false;
  // temporal stride or dilation: the plan-driven kernel, staged 1x1 shapes
  const bool staged = c.id == 0 || c.id == 1 || c.id == 5 || c.id == 6;
  if ((g.sT != 1 || g.dT != 1) && !(staged && plan_table_fits(g))) return false;
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  const int64_t lim = int64_t(1) << 31;
  return int64_t(g.B) * g.Cin * x_frames * g.S() * esz < lim &&
         int64_t(g.B) * g.Cout * y_frames * g.So() * esz < lim &&
         int64_t(g.R) * int64_t(conv_layout(g).ring_slot_elems) * 4 < lim &&
         conv_layout(g).weight_bytes < (int64_t(1) << 30);
}

hipError_t launch_conv_steps_reg(const ConvGeom& g, const ConvLayout& L, char* state,
                                 const void* x, int64_t x_bc, int32_t nreal, int32_t count,
                                 void* y, int64_t y_bc, int64_t n0, bool update, hipStream_t s) {
  RegConfig c;
  if (!reg_config(g, g.cfg, &c)) return hipErrorInvalidValue;
  const int ktm = reg_steps_ktm(g);
#define CO_STEPS(TY, TAPS, CSMAX, KSPLIT, KTM) \
  reg_steps_launch<TY, TAPS, CSMAX, KSPLIT, KTM>(g, c, L, state, x, x_bc, nreal, count, y, y_bc, \
                                                 n0, update, s)
  switch (c.id * 16 + ktm) {
    case 0 * 16 + 3: return CO_STEPS(float, 1, 16, 1, 3);
    case 0 * 16 + 9: return CO_STEPS(float, 1, 16, 1, 9);
    case 1 * 16 + 3: return CO_STEPS(float, 1, 32, 1, 3);
    case 2 * 16 + 3: return CO_STEPS(float, 9, 6, 1, 3);
    case 3 * 16 + 3: return CO_STEPS(float, 9, 3, 1, 3);
    case 4 * 16 + 3: return CO_STEPS(float, 10, 6, 2, 3);
    case 5 * 16 + 3: return CO_STEPS(bf16_t, 1, 2, 1, 3);
    case 5 * 16 + 9: return CO_STEPS(bf16_t, 1, 2, 1, 9);
    case 6 * 16 + 3: return CO_STEPS(bf16_t, 1, 4, 1, 3);
    case 6 * 16 + 9: return CO_STEPS(bf16_t, 1, 4, 1, 9);
    case 9 * 16 + 3: return CO_STEPS(bf16_t, 9, 1, 1, 3);
    default: return hipErrorInvalidValue;
  }
#undef CO_STEPS
}

hipError_t launch_pack_reg(const ConvGeom& g, const ConvLayout& L, char* state,
                           const void* weight, const float* wscale, hipStream_t s) {
  RegConfig c;
  if (!reg_config(g, g.cfg, &c)) return hipErrorInvalidValue;
  const int64_t total = int64_t(c.n_frags) * c.U * 64;
  uint4* out = reinterpret_cast<uint4*>(state + L.weight);
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(pack_reg_kernel<bf16_t>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                       static_cast<const bf16_t*>(weight), wscale, out);
  else
    hipLaunchKernelGGL(pack_reg_kernel<float>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                       static_cast<const float*>(weight), wscale, out);
  return hipGetLastError();
}

}  // namespace coinf
