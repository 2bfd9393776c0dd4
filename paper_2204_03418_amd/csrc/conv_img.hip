// Frame-resident implicit-GEMM continual convolution step (bf16, groups = 1).
//
// The per-step contraction is the GEMM of the other matrix-core steps
// (section 3.1: the arriving frame's contribution to every future output is
// computed at once and kept as a partial sum),
//
//   m = output pixel of a stream, n = (temporal tap t, output channel o),
//   k = (input channel block, spatial tap),
//
// with the same fused ring epilogue.  It targets many streams of small
// frames (e.g. 64 streams of 14x14 with 192 channels), where one stream's
// whole frame, every channel of it, fits in LDS:
//
//   * a workgroup of four waves owns stream b and a slab of 16*NF columns;
//     it stages the frame once, channels-last with a zero halo (consecutive
//     rows share their halo column), so every spatial tap of every k-step
//     reads the same staged pixels at a uniform offset;
//   * the slab's weights stream through LDS in stages of kImgKC k-steps,
//     double buffered, copied straight from global memory into LDS in the
//     order and swizzle the fragment reads use (packed at init);
//   * the frame's 16-pixel fragments are dealt to the waves, `mo` each; a
//     single fragment left over is shared out by column fragments, so the
//     four SIMDs carry (nearly) equal matrix work;
//   * each wave holds NF column fragments per pixel fragment, so a k-step
//     reads (pixel fragments + NF) 1 KB operands from LDS for
//     (pixel fragments * NF) v_mfma_f32_16x16x32_bf16.
//
// Accumulators start from the ring partial sums of the taps that add to them
// (ACC, EMIT), read at the start together with the frame.
#include <type_traits>

#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));

constexpr int kImgThreads = kImgThreadsHost;  // eight waves, two per SIMD

struct ImgArgs {
  int32_t M, N, So;
  int32_t slab0, slab_cnt, wgs, blocks_per_xcd;
  int32_t pix_units, cols, a_units;
  int32_t nsteps, nchunks;
  int32_t items, pairs, wq;  // staging items, items per channel octet, items per row
  int32_t pair;              // even width: two pixels per staging load
  int32_t x_bytes, ring_bytes, y_bytes;  // buffer extents (bytes)
  int32_t ring_slot;         // floats between ring slots
  FastDiv fd_pairs, fd_wq, fd_Cout, fd_Wo, fd_slabs;  // dividers of the index decompositions
};

// Per-tap action and ring slot as one dword each (action | slot << 8), read
// with scalar loads.
struct ImgTaps {
  int32_t as[CO_MAX_TAPS];
};

// One workgroup per CU (its LDS) of eight waves, two per SIMD (a single
// wave cannot issue matrix instructions back to back).  Waves g and g + 4
// form a pair: they own the same accumulator fragments and split the
// k-steps between them (even / odd), and their partial sums meet in LDS at
// the end.  A pair owns MO pixel-fragment rows (all NF column fragments)
// and, when the frame leaves one row over (R = 1), SS column fragments of
// that shared row: pair g takes columns g, g + 4, g + 8, ... (a pair with
// fewer computes a dummy one that is never stored), so every wave runs the
// same instruction stream.
template <int KH, int KW, int MO, int R, int NF>
__global__ __launch_bounds__(kImgThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void
conv_step_img_kernel(ConvGeom g, ImgArgs ia, const bf16_t* __restrict__ x, int64_t x_bc,
                     bf16_t* __restrict__ y, int64_t y_bc, const uint4* __restrict__ wp,
                     const float* __restrict__ bias, float* __restrict__ ring, ImgTaps tt) {
  static_assert(R == 0 || R == 1, "at most one shared fragment row");
  constexpr int KHW = KH * KW;
  constexpr int SS = R * ((NF + 3) / 4);    // shared column fragments per pair
  constexpr int NA = MO + R;                // frame operands per k-step
  constexpr int NS = 16 * NF;               // columns per slab
  constexpr int BSTEP = NF * 64;            // 16-byte units of one k-step of weights
  constexpr int BCHUNK = kImgKC * BSTEP;    // units of one weight stage
  constexpr int BROUNDS = (BCHUNK + kImgThreads - 1) / kImgThreads;
  constexpr int NACC = MO * NF + SS;        // accumulator fragments of a pair
  constexpr int HALF = (NACC + 1) / 2;      // fragments finished by the even wave
  extern __shared__ uint4 smem[];

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pr = wave & 3;   // pair: accumulator fragments
  const int kh = wave >> 2;  // k-steps of parity kh
  const int lrow = lane & 15, lgrp = lane >> 4;

  // XCD-aware numbering: blocks are dealt to the 8 XCDs round-robin, so the
  // slabs of one stream (consecutive logical blocks) share an XCD's L2.
  const int bid = int(blockIdx.x);
  const int lb = (bid & 7) * ia.blocks_per_xcd + (bid >> 3);
  if (lb >= ia.wgs) return;  // whole workgroups: no barrier is skipped
  const int b = fdiv(lb, ia.fd_slabs);
  const int slab = ia.slab0 + (lb - b * ia.slab_cnt);

  uint4* const As = smem;
  uint4* const Bs = smem + ia.a_units;

  // ---- frame staging loads: item = (pixel pair or pixel, channel octet) ----
  // Eight channel planes per item, one 4-byte (pair) or 2-byte load each;
  // all are issued before anything waits.
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ia.x_bytes);
  const int plane_b = int(x_bc * 2);
  const int pw = ia.pair ? 2 : 1;
  uint32_t ra[kImgItems][8];
  int a_dst[kImgItems];
#pragma unroll
  for (int ii = 0; ii < kImgItems; ++ii) {
    const int it = tid + ii * kImgThreads;
    const bool ok = it < ia.items;
    const int itc = ok ? it : 0;
    const int co = fdiv(itc, ia.fd_pairs), pp = itc - co * ia.pairs;
    const int r = fdiv(pp, ia.fd_wq), c = (pp - r * ia.wq) * pw;
    a_dst[ii] = ok ? ((r + g.pH) * ia.cols + c + g.pW) * ia.pix_units + co : -1;
    const int src = ok ? int(uint32_t((b * g.Cin + co * 8)) * uint32_t(plane_b) +
                             uint32_t(r * g.W + c) * 2u)
                       : kOutOfRange;
    if (ia.pair) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        ra[ii][e] = __builtin_amdgcn_raw_buffer_load_b32(xr, src, e * plane_b, 0);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        ra[ii][e] = uint32_t(__builtin_amdgcn_raw_buffer_load_b16(xr, src, e * plane_b, 0));
    }
  }

  // ---- weight stages: straight from global memory into LDS ------------
  auto copy_b = [&](int c) {
    const uint4* src = wp + (int64_t(slab) * ia.nchunks + c) * BCHUNK;
    uint4* dst = Bs + (c & 1) * BCHUNK;
#pragma unroll
    for (int rr = 0; rr < BROUNDS; ++rr) {
      const int u0 = rr * kImgThreads + wave * 64;  // this wave's 1 KB
      if (u0 < BCHUNK)
        __builtin_amdgcn_global_load_lds(src + u0 + lane,
                                         (__attribute__((address_space(3))) void*)(dst + u0),
                                         16, 0, 0);
    }
  };
  copy_b(0);
  if (ia.nchunks > 1) copy_b(1);

  // ---- frame into LDS: zero halo, then the staged items -------------------
  for (int u = tid; u < ia.a_units; u += kImgThreads) As[u] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
#pragma unroll
  for (int ii = 0; ii < kImgItems; ++ii) {
    if (a_dst[ii] < 0) continue;
    const uint32_t* r = ra[ii];
    if (ia.pair) {
      As[a_dst[ii]] = make_uint4((r[0] & 0xffffu) | (r[1] << 16), (r[2] & 0xffffu) | (r[3] << 16),
                                 (r[4] & 0xffffu) | (r[5] << 16), (r[6] & 0xffffu) | (r[7] << 16));
      As[a_dst[ii] + ia.pix_units] =
          make_uint4((r[0] >> 16) | (r[1] & 0xffff0000u), (r[2] >> 16) | (r[3] & 0xffff0000u),
                     (r[4] >> 16) | (r[5] & 0xffff0000u), (r[6] >> 16) | (r[7] & 0xffff0000u));
    } else {
      As[a_dst[ii]] = make_uint4(r[0] | (r[1] << 16), r[2] | (r[3] << 16), r[4] | (r[5] << 16),
                                 r[6] | (r[7] << 16));
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- accumulator fragments of this pair --------------------------------
  // a = 0 .. MO*NF - 1: own row a / NF, column a % NF; a = MO*NF + s: shared
  // slot s, column 4s + pr of the shared row (a dummy past the last column).
  // Fragments a < HALF are finished by the even wave, the rest by the odd.
  auto acc_row = [&](int a) { return a < MO * NF ? pr * MO + a / NF : 4 * MO; };
  auto acc_col = [&](int a) { return a < MO * NF ? a % NF : 4 * (a - MO * NF) + pr; };
  // lane (lrow, lgrp) of accumulator a holds column slab*NS + 16*col + lrow
  // and the four pixels 16*row + 4*lgrp .. +3 of stream b.  The column's tap
  // t and channel o come from two wave-uniform tap-table reads (a 16-column
  // fragment spans at most two taps, as C_out >= 16).
  struct ColInfo {
    int act, o, off;
  };
  auto col_info = [&](int col) {
    const int n0 = slab * NS + col * 16;  // uniform
    const int t0 = fdiv(n0, ia.fd_Cout);
    const int o0 = n0 - t0 * g.Cout;
    const int as0 = tt.as[min(t0, g.kT - 1)], as1 = tt.as[min(t0 + 1, g.kT - 1)];
    int o = o0 + lrow;
    const bool wrap = o >= g.Cout;
    o -= wrap ? g.Cout : 0;
    const int as = wrap ? as1 : as0;
    const bool in = col < NF && n0 + lrow < ia.N;
    return ColInfo{in ? (as & 0xff) : CO_TAP_NONE, o,
                   (as >> 8) * ia.ring_slot + o * ia.M + b * ia.So};
  };
  const bool vec = (ia.So & 3) == 0;
  const __amdgpu_buffer_rsrc_t rr_ = make_rsrc(ring, ia.ring_bytes);

  // accumulators: the finishing wave of a fragment seeds it with the ring
  // partial sum for the taps that add to it (ACC, EMIT) and with the bias
  // for the taps that complete an output (EMIT, EMIT_FRESH), so the epilogue
  // only stores; every other lane reads an out-of-range offset (zero), and
  // the loads are one branch-free batch.  The bias depends on the column
  // fragment only: one value per column fragment and lane.
  const __amdgpu_buffer_rsrc_t br = make_rsrc(bias, g.Cout * 4);
  float bcol[NF + SS];
#pragma unroll
  for (int cf = 0; cf < NF + SS; ++cf) {
    const ColInfo ci = col_info(cf < NF ? cf : 4 * (cf - NF) + pr);
    const bool emit = ci.act == CO_TAP_EMIT || ci.act == CO_TAP_EMIT_FRESH;
    bcol[cf] = __uint_as_float(
        __builtin_amdgcn_raw_buffer_load_b32(br, emit ? ci.o * 4 : kOutOfRange, 0, 0));
  }
  v4f acc[NACC];
#pragma unroll
  for (int a = 0; a < NACC; ++a) {
    const int P0 = acc_row(a) * 16 + lgrp * 4;
    const ColInfo ci = col_info(acc_col(a));
    const bool fin = (a < HALF) == (kh == 0) && P0 < ia.So;
    const bool rd = fin && (ci.act == CO_TAP_ACC || ci.act == CO_TAP_EMIT);
    const auto v =
        __builtin_amdgcn_raw_buffer_load_b128(rr_, rd ? (ci.off + P0) * 4 : kOutOfRange, 0, 0);
    acc[a] = __builtin_bit_cast(v4f, v);
  }
#pragma unroll
  for (int a = 0; a < NACC; ++a) {
    const int P0 = acc_row(a) * 16 + lgrp * 4;
    const bool fin = (a < HALF) == (kh == 0);
    acc[a] += fin ? bcol[a < MO * NF ? a % NF : NF + (a - MO * NF)] : 0.f;
    if (!vec) {  // a ragged frame: the last fragment's lanes may reach the next stream
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[a][q] = P0 + q < ia.So ? acc[a][q] : 0.f;
    }
  }

  // per-lane LDS unit of each frame operand row at k-step (block 0, tap 0,
  // 0); rows past the frame read its last pixel (never stored)
  int abase[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = i < MO ? pr * MO + i : 4 * MO;
    const int p = min(row * 16 + lrow, ia.So - 1);
    const int pi = fdiv(p, ia.fd_Wo), pj = p - pi * g.Wo;
    abase[i] = (pi * ia.cols + pj) * ia.pix_units + lgrp;
  }
  // weight unit of column lrow of a fragment, channel group lgrp (swizzled
  // so every 8 consecutive lanes hit distinct banks)
  const int bsw = (lrow * 4) + (lgrp ^ ((lrow >> 2) & 3));

  // uniform LDS unit offset of k-step k: channel block k / KHW, spatial tap k % KHW
  auto a_off = [&](int k) {
    const int cb = k / KHW, uv = k - cb * KHW;
    const int u = uv / KW, v = uv - u * KW;
    return (u * ia.cols + v) * ia.pix_units + cb * 4;
  };
  // operands of one k-step, in the order the matrix instructions consume them
  v8bf af[1][NA], bfr[1][NF];
  auto load = [&](auto Q, int k, const uint4* Bst) {
    constexpr int q = decltype(Q)::value;
    const int off = a_off(k);
#pragma unroll
    for (int i = 0; i < NA; ++i) af[q][i] = __builtin_bit_cast(v8bf, As[abase[i] + off]);
#pragma unroll
    for (int nf = 0; nf < NF; ++nf) bfr[q][nf] = __builtin_bit_cast(v8bf, Bst[nf * 64 + bsw]);
  };
  // own rows by column fragment, then the shared row's columns 4s + pr,
  // whose weight fragments are picked from the loaded ones (a wave-uniform
  // select)
  auto mma = [&](auto Q) {
    constexpr int q = decltype(Q)::value;
#pragma unroll
    for (int nf = 0; nf < NF; ++nf)
#pragma unroll
      for (int i = 0; i < MO; ++i)
        acc[i * NF + nf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[q][i], bfr[q][nf],
                                                                   acc[i * NF + nf], 0, 0, 0);
    if constexpr (R > 0) {
#pragma unroll
      for (int s2 = 0; s2 < SS; ++s2) {
        const v8bf c0 = bfr[q][min(4 * s2 + 0, NF - 1)], c1 = bfr[q][min(4 * s2 + 1, NF - 1)];
        const v8bf c2 = bfr[q][min(4 * s2 + 2, NF - 1)], c3 = bfr[q][min(4 * s2 + 3, NF - 1)];
        const v8bf bs = pr == 0 ? c0 : pr == 1 ? c1 : pr == 2 ? c2 : c3;
        acc[MO * NF + s2] =
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[q][MO], bs, acc[MO * NF + s2], 0, 0, 0);
      }
    }
  };
  using B0 = std::integral_constant<int, 0>;

  __builtin_amdgcn_s_waitcnt(0);  // weight stages 0 (and 1), the seeds and the frame
  __syncthreads();
  // Stage c holds k-steps kImgKC*c .. +kImgKC-1 (kImgKC = 3); this wave takes
  // those of parity kh: two (j = 0, 2) or one (j = 1).  A step requests
  // its operands, then runs its matrix instructions; the other wave of the
  // SIMD issues its own while this one waits.  After a stage: wait for this wave's copies of the next
  // stage, the barrier for everyone's (which also tells that this stage is
  // read), then start the copy two stages ahead.
  static_assert(kImgKC == 3, "the stage schedule below assumes three k-steps per stage");
  for (int c = 0; c < ia.nchunks; ++c) {
    const uint4* Bc = Bs + (c & 1) * BCHUNK;
    const int k0 = c * kImgKC;
#pragma unroll
    for (int j = 0; j < kImgKC; ++j)
      if (((k0 + j) & 1) == kh) {
        load(B0{}, k0 + j, Bc + j * BSTEP);
        mma(B0{});
      }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (c + 2 < ia.nchunks) copy_b(c + 2);
  }

  // ---- the pair's partial sums meet in LDS -----------------------------------
  // (the last stage ended with a barrier: the frame and weights are read)
#pragma unroll
  for (int a = 0; a < NACC; ++a) {
    const bool mine = (a < HALF) == (kh == 0);
    if (!mine) smem[(pr * NACC + a) * 64 + lane] = __builtin_bit_cast(uint4, acc[a]);
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < NACC; ++a) {
    const bool mine = (a < HALF) == (kh == 0);
    if (mine) acc[a] += __builtin_bit_cast(v4f, smem[(pr * NACC + a) * 64 + lane]);
  }

  // ---- fused ring epilogue ---------------------------------------------------
  // A fragment's lanes take one of two stores (ring or output); a store is
  // issued only for the lanes that make it.
  const bool yvec = vec && (y_bc & 3) == 0 && (reinterpret_cast<uintptr_t>(y) & 7) == 0;
#pragma unroll
  for (int a = 0; a < NACC; ++a) {
    const bool mine = (a < HALF) == (kh == 0);
    if (!mine) continue;
    const int P0 = acc_row(a) * 16 + lgrp * 4;
    const ColInfo ci = col_info(acc_col(a));
    if (P0 >= ia.So) continue;
    const v4f v = acc[a];
    if (ci.act == CO_TAP_START || ci.act == CO_TAP_ACC) {
      float* dst = ring + ci.off + P0;
      if (vec) {
        *reinterpret_cast<v4f*>(dst) = v;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (P0 + q < ia.So) dst[q] = v[q];
      }
    } else if (ci.act == CO_TAP_EMIT || ci.act == CO_TAP_EMIT_FRESH) {
      bf16_t* dst = y + (int64_t(b) * g.Cout + ci.o) * y_bc + P0;
      if (yvec) {
        const uint32_t lo = uint32_t(f32_to_bf16(v[0])) | (uint32_t(f32_to_bf16(v[1])) << 16);
        const uint32_t hi = uint32_t(f32_to_bf16(v[2])) | (uint32_t(f32_to_bf16(v[3])) << 16);
        *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (P0 + q < ia.So) dst[q] = f32_to_bf16(v[q]);
      }
    }
  }
}

// Pack W (C_out, C_in, kT, kH, kW) bf16 as [slab][stage][k-step][column][4
// units of 8 channels], zero padded: k-step = block * kH*kW + spatial tap,
// column n of slab s is n' = s*16*NF + n -> (t = n' / C_out, o = n' % C_out),
// and unit p of column n holds channel group p ^ ((n >> 2) & 3).
__global__ __launch_bounds__(kBlock) void pack_img_kernel(ConvGeom g, ImgConfig c,
                                                          const bf16_t* __restrict__ w,
                                                          const float* __restrict__ wscale,
                                                          uint4* __restrict__ out) {
  const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= c.weight_units) return;
  const int NS = 16 * c.NF;
  const int phys = int(idx & 3);
  int64_t rest = idx >> 2;
  const int n = int(rest % NS);
  rest /= NS;
  const int k = int(rest % (int64_t(c.nchunks) * kImgKC));
  const int s = int(rest / (int64_t(c.nchunks) * kImgKC));
  const int grp = phys ^ ((n >> 2) & 3);
  const int khw = g.kH * g.kW;
  const int cb = k / khw, uv = k - cb * khw;
  const int u = uv / g.kW, v = uv - u * g.kW;
  const int nn = s * NS + n;
  const int t = nn / g.Cout, o = nn - t * g.Cout;
  const bool col = nn < g.kT * g.Cout && k < c.nsteps;
  uint32_t word[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t pr = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int ch = cb * 32 + grp * 8 + 2 * e + h;
      uint32_t val = 0;
      if (col && ch < g.Cin)
        val = scaled_weight<bf16_t>(
            w[((((int64_t(o) * g.Cin + ch) * g.kT + t) * g.kH + u) * g.kW) + v], wscale, o);
      pr |= val << (16 * h);
    }
    word[e] = pr;
  }
  out[idx] = make_uint4(word[0], word[1], word[2], word[3]);
}

template <int KH, int KW, int MO, int R>
hipError_t img_launch(const ConvGeom& g, const ImgConfig& c, const ConvLayout& L, char* state,
                      const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  auto kern = conv_step_img_kernel<KH, KW, MO, R, kImgNF>;
  static bool attr_set = false;
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             int(kLdsBytes));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  ImgTaps tt;
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
  const int NS = 16 * c.NF;
  ImgArgs ia;
  ia.M = int32_t(int64_t(g.B) * g.So());
  ia.N = g.kT * g.Cout;
  ia.So = int32_t(g.So());
  // only the slabs holding active taps
  ia.slab0 = (t_lo * g.Cout) / NS;
  ia.slab_cnt = int32_t(ceil_div(int64_t(t_hi + 1) * g.Cout, NS)) - ia.slab0;
  ia.wgs = g.B * ia.slab_cnt;
  ia.blocks_per_xcd = int32_t(ceil_div(ia.wgs, 8));
  ia.pix_units = c.pix_units;
  ia.cols = c.cols;
  ia.a_units = c.a_units;
  ia.nsteps = c.nsteps;
  ia.nchunks = c.nchunks;
  ia.items = c.items;
  ia.pairs = c.pairs;
  ia.pair = c.pair;
  ia.wq = c.pair ? g.W / 2 : g.W;
  ia.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * 2);
  ia.ring_slot = int32_t(L.ring_slot_elems);
  ia.fd_pairs = make_fastdiv(uint32_t(c.pairs));
  ia.fd_wq = make_fastdiv(uint32_t(ia.wq));
  ia.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  ia.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  ia.fd_slabs = make_fastdiv(uint32_t(ia.slab_cnt));
  ia.ring_bytes = int32_t(int64_t(g.R) * L.ring_slot_elems * 4);
  ia.y_bytes = io.y ? int32_t(((int64_t(g.B) * g.Cout - 1) * io.y_bc + g.So()) * 2) : 0;
  hipLaunchKernelGGL(kern, dim3(unsigned(8 * ia.blocks_per_xcd)), dim3(kImgThreads),
                     size_t(c.lds_bytes), s, g, ia, static_cast<const bf16_t*>(io.x), io.x_bc,
                     static_cast<bf16_t*>(io.y), io.y_bc,
                     reinterpret_cast<const uint4*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), tt);
  return hipGetLastError();
}

// (own, shared) fragment rows per wave that are instantiated; img_config
// accepts only these.
template <int KH, int KW>
hipError_t img_dispatch(const ConvGeom& g, const ImgConfig& c, const ConvLayout& L, char* state,
                        const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  switch (c.mo * 4 + c.mr) {
    case 1 * 4 + 0: return img_launch<KH, KW, 1, 0>(g, c, L, state, io, plan, s);
    case 2 * 4 + 1: return img_launch<KH, KW, 2, 1>(g, c, L, state, io, plan, s);
    case 3 * 4 + 1: return img_launch<KH, KW, 3, 1>(g, c, L, state, io, plan, s);
    case 4 * 4 + 0: return img_launch<KH, KW, 4, 0>(g, c, L, state, io, plan, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool img_step_needs_staging(const ConvGeom& g, const StepIO& io) {
  ImgConfig c;
  if (!img_config(g, &c)) return false;
  // 32-bit offsets: the reachable part of x and of y below 2^31 bytes;
  // pixel pairs need 4-byte aligned rows
  const int64_t x_extent = ((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * 2;
  const bool pair_ok = !c.pair || ((reinterpret_cast<uintptr_t>(io.x) & 3) == 0 &&
                                   (io.x_bc & 1) == 0);
  const int64_t y_extent = ((int64_t(g.B) * g.Cout - 1) * io.y_bc + g.So()) * 2;
  return x_extent >= (int64_t(1) << 31) || (io.y && y_extent >= (int64_t(1) << 31)) || !pair_ok;
}

hipError_t launch_conv_step_img(const ConvGeom& g, const ConvLayout& L, char* state,
                                const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  ImgConfig c;
  if (!img_config(g, &c)) return hipErrorInvalidValue;
  if (int64_t(g.R) * L.ring_slot_elems * 4 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
  if (img_step_needs_staging(g, io)) return launch_conv_step_staged(g, L, state, io, plan, s);
  if (g.kH == 3 && g.kW == 3) return img_dispatch<3, 3>(g, c, L, state, io, plan, s);
  if (g.kH == 1 && g.kW == 1) return img_dispatch<1, 1>(g, c, L, state, io, plan, s);
  return hipErrorInvalidValue;
}

hipError_t launch_pack_img(const ConvGeom& g, const ConvLayout& L, char* state,
                           const void* weight, const float* wscale, hipStream_t s) {
  ImgConfig c;
  if (!img_config(g, &c)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_img_kernel, dim3(grid_for(c.weight_units)), dim3(kBlock), 0, s, g, c,
                     static_cast<const bf16_t*>(weight), wscale,
                     reinterpret_cast<uint4*>(state + L.weight));
  return hipGetLastError();
}

}  // namespace coinf
