// Warp-specialized implicit-GEMM continual convolution step (bf16, 3x3
// spatial taps, spatial stride and dilation 1) for layers with enough
// 448 x 64 output tiles to give every CU one.
//
// The per-step contraction (section 3.1: the arriving frame against every
// temporal tap, eagerly) is the GEMM of conv_gemm.hip:
//   C[m = (b, i, j)][n = t * C_out + o] = sum over k = (u, v, c) of
//   x_t[b][c][i + u - pH][j + v - pW] * W[o][c][t][u][v],
// with the same fused ring epilogue (start / add / complete, bias and the
// rounding of y once, at emission).
//
// A workgroup of eight waves owns a tile of 448 pixels x 64 columns:
// * four consumer waves, one per SIMD, each own 112 pixels x 64 columns
//   (7 x 4 fragments of v_mfma_f32_16x16x32_bf16) with the whole K in
//   their accumulators.  A k-step is one spatial tap of one 32-channel
//   chunk.  Input fragments come from LDS; weight fragments come straight
//   from L2 into a ring of three register sets, two k-steps ahead, so the
//   weights never pass through LDS.  A consumer's only memory requests are
//   these weight loads, so waiting for a k-step's weights never waits for
//   anything else.
// * four producer waves stage the next chunk's input rows into the other
//   of two LDS buffers while the consumers compute (NCHW to channels-last:
//   a pixel is five 16-byte units, four of eight channels and one pad, so
//   consecutive pixels fall in different bank groups).  Their loads run a
//   chunk ahead of the buffer they fill.
// One barrier per chunk hands the buffers over.
//
// Staged rows: the images the tile touches, one after another with pH zero
// rows between consecutive images (one image's bottom halo is the next
// one's top halo), and rows that share their zero halo column.  Every
// spatial tap (u, v) is then the offset u * cols + v from a fragment's base
// pixel.  The zero rows are written once, at the start, and never staged.
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
typedef uint32_t v2u32 __attribute__((ext_vector_type(2)));

constexpr int kKHW = 9;                      // 3 x 3 spatial taps
constexpr int kWM = kWsWM, kWN = kWsWN;      // fragments per consumer wave
constexpr int kMWG = 16 * kWM * kWsWaves;    // 448 pixels per tile
constexpr int kNWG = 16 * kWN;               // 64 columns per tile
constexpr int kThreads = 128 * kWsWaves;     // consumers + producers
constexpr int kPThreads = 64 * kWsWaves;     // producer threads
constexpr int kAI = kGemmStageItems / kPThreads;  // staging items per producer thread
constexpr int kNB = 3;                       // weight register sets (k-steps in flight)

struct WsArgs {
  int32_t M, N, So;
  int32_t m_tiles, n_tile0, n_tile_cnt, tiles_per_xcd;
  int32_t n_chunks, cols, a_units, rows;  // rows: staged rows allocated per buffer
  int32_t x_bytes, w_bytes, ring_bytes, y_bytes;
  int32_t yvec;  // y is 8-byte aligned: four outputs go out as one store
  // dividers: pixels per frame, Wo, Ho, H, C_out, column tiles, staging items per row
  FastDiv fd_So, fd_Wo, fd_Ho, fd_H, fd_Cout, fd_ntc, fd_wpi;
};

// Raw loads of one staging item -- 8 channels of one pixel, or of two
// adjacent pixels when rows have even width -- and their packing into the
// pixels' 16-byte LDS units (bit operations only).
__device__ __forceinline__ uint32_t load_pair(__amdgpu_buffer_rsrc_t r, int voff, int soff,
                                              bool pair) {
  return pair ? __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0)
              : uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0));
}

__device__ __forceinline__ void pack_pair(const uint32_t (&r)[8], uint4& u0, uint4& u1) {
  u0.x = (r[0] & 0xffffu) | (r[1] << 16);
  u0.y = (r[2] & 0xffffu) | (r[3] << 16);
  u0.z = (r[4] & 0xffffu) | (r[5] << 16);
  u0.w = (r[6] & 0xffffu) | (r[7] << 16);
  u1.x = (r[0] >> 16) | (r[1] & 0xffff0000u);
  u1.y = (r[2] >> 16) | (r[3] & 0xffff0000u);
  u1.z = (r[4] >> 16) | (r[5] & 0xffff0000u);
  u1.w = (r[6] >> 16) | (r[7] & 0xffff0000u);
}

template <bool PAIR>
__global__ __launch_bounds__(kThreads) void conv_step_gemm_ws_kernel(
    ConvGeom g, WsArgs wa, const bf16_t* __restrict__ x, int64_t x_bc, bf16_t* __restrict__ y,
    int64_t y_bc, const uint4* __restrict__ wp, const float* __restrict__ bias,
    float* __restrict__ ring, int64_t ring_slot, TapTable tt) {
  extern __shared__ uint4 smem[];
  const int tid = int(threadIdx.x);
  const int lane = tid & 63, wave = tid >> 6;

  // XCD-aware numbering: blocks are dealt to the 8 XCDs round-robin, so
  // logical tile L = xcd * tiles_per_xcd + k keeps neighbours on one XCD.
  const int bid = int(blockIdx.x);
  const int L = (bid & 7) * wa.tiles_per_xcd + (bid >> 3);
  if (L >= wa.m_tiles * wa.n_tile_cnt) return;  // the whole workgroup
  const int m_tile = fdiv(L, wa.fd_ntc);
  const int n_tile = wa.n_tile0 + (L - m_tile * wa.n_tile_cnt);
  const int m0 = m_tile * kMWG;
  const int m1 = min(m0 + kMWG, wa.M);
  const int r0 = fdiv(m0, wa.fd_Wo), r1 = fdiv(m1 - 1, wa.fd_Wo);
  const int b0 = fdiv(r0, wa.fd_Ho), i0 = r0 - b0 * g.Ho;
  const int b1 = fdiv(r1, wa.fd_Ho), i1 = r1 - b1 * g.Ho;
  const int a_units = wa.a_units;

  for (int u = tid; u < 2 * a_units; u += kThreads) smem[u] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();  // zero rows, halo columns and trash pixels

  if (wave >= kWsWaves) {
    // ------------------------------------------------------------ producer
    const int pt = tid - kPThreads;
    // real input rows of the tile, flattened q = b * H + ih
    const int q0 = b0 * g.H + max(0, i0 - g.pH);
    const int q1 = b1 * g.H + min(g.H - 1, i1 + 2 - g.pH);
    const int nreal = q1 - q0 + 1;
    constexpr int PW = PAIR ? 2 : 1;
    const int wp_items = g.W / PW;
    const int a_items = nreal * 4 * wp_items;
    const int trash = wa.rows * wa.cols + wa.cols;  // two pixels past the staged rows
    int a_src[kAI], a_dst[kAI], a_dst1[kAI], a_grp[kAI];
#pragma unroll
    for (int ai = 0; ai < kAI; ++ai) {
      const int it = pt + ai * kPThreads;
      a_src[ai] = 0;
      a_grp[ai] = 0;
      a_dst[ai] = trash * kGemmPixUnits;
      a_dst1[ai] = (trash + 1) * kGemmPixUnits;
      if (it < a_items) {
        // items run along a row, then down the tile's rows, then over the
        // four channel groups: the lanes of one load instruction read
        // consecutive rows of one channel plane
        const int rest = fdiv(it, wa.fd_wpi);
        const int xp = it - rest * wp_items;
        const int grp = (rest >= nreal) + (rest >= 2 * nreal) + (rest >= 3 * nreal);
        const int q = q0 + rest - grp * nreal;
        const int b = fdiv(q, wa.fd_H), ih = q - b * g.H;
        const int xcol = xp * PW;
        a_src[ai] = int(((int64_t(b) * g.Cin + grp * 8) * x_bc + int64_t(ih) * g.W + xcol) * 2);
        a_grp[ai] = grp;
        const int row = (b - b0) * (g.H + g.pH) + ih - (i0 - g.pH);
        const int pix = row * wa.cols + xcol + g.pW;
        a_dst[ai] = pix * kGemmPixUnits + grp;
        a_dst1[ai] = (pix + 1) * kGemmPixUnits + grp;
      }
    }
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, wa.x_bytes);
    const int plane_bytes = int(x_bc * 2);
    uint32_t ra[2][kAI][8];
    // Channels past C_in read the out-of-range offset (zero).
    auto prefetch = [&](uint32_t(&r)[kAI][8], int ch) {
      const int cbase = ch * 32;
#pragma unroll
      for (int ai = 0; ai < kAI; ++ai)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool cin = cbase + a_grp[ai] * 8 + e < g.Cin;
          r[ai][e] = load_pair(xr, cin ? a_src[ai] : kOutOfRange, (cbase + e) * plane_bytes, PAIR);
        }
    };
    auto store = [&](uint32_t(&r)[kAI][8], int buf) {
      uint4* As = smem + buf * a_units;
#pragma unroll
      for (int ai = 0; ai < kAI; ++ai) {
        uint4 p0, p1;
        pack_pair(r[ai], p0, p1);
        As[a_dst[ai]] = p0;
        if (PAIR) As[a_dst1[ai]] = p1;
      }
    };
    const int n = wa.n_chunks;
    prefetch(ra[0], 0);
    if (n > 1) prefetch(ra[1], 1);
    __builtin_amdgcn_sched_barrier(0);
    store(ra[0], 0);
    __syncthreads();
    // phase ch: the consumers compute chunk ch from buffer ch & 1 while
    // chunk ch + 1 goes into the other buffer and chunk ch + 2's loads start
    // into the register set chunk ch came from
    for (int ch = 0; ch < n; ch += 2) {
      if (ch + 1 < n) {
        if (ch + 2 < n) prefetch(ra[0], ch + 2);
        __builtin_amdgcn_sched_barrier(0);
        store(ra[1], 1);
      }
      __syncthreads();
      if (ch + 1 < n) {
        if (ch + 2 < n) {
          if (ch + 3 < n) prefetch(ra[1], ch + 3);
          __builtin_amdgcn_sched_barrier(0);
          store(ra[0], 0);
        }
        __syncthreads();
      }
    }
    return;
  }

  // -------------------------------------------------------------- consumer
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int w = wave;

  // This lane's columns: the tap's action, the output channel, the bias and
  // the byte offset of the channel's plane in the tap's ring slot (the ring
  // is below 2^31 bytes; the host guarantees B*Ho*Wo % 4 == 0, so a lane's
  // four pixels are one 16-byte unit of the plane).
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(ring, wa.ring_bytes);
  int e_act[kWN], e_o[kWN], e_ring[kWN];
  float e_bias[kWN];  // requested here, used only by the epilogue
#pragma unroll
  for (int nf = 0; nf < kWN; ++nf) {
    const int ncol = n_tile * kNWG + nf * 16 + lrow;
    const int nn = ncol < wa.N ? ncol : wa.N - 1;
    const int t = fdiv(nn, wa.fd_Cout), o = nn - t * g.Cout;
    e_act[nf] = ncol < wa.N ? int(tt.action[t]) : CO_TAP_NONE;
    e_o[nf] = o;
    const int sl = tt.slot[t] < 0 ? 0 : tt.slot[t];
    e_ring[nf] = int((int64_t(sl) * ring_slot + int64_t(o) * wa.M) * 4);
    e_bias[nf] = bias[o];
  }

  // Accumulators start from the partial sum the ring holds for the taps
  // that add to it (ACC, EMIT), else from zero: every lane issues its loads
  // in one batch, the others at the out-of-range offset (which reads zero).
  v4f acc[kWM][kWN];
#pragma unroll
  for (int mf = 0; mf < kWM; ++mf) {
    const int P0 = m0 + (w * kWM + mf) * 16 + lgrp * 4;
#pragma unroll
    for (int nf = 0; nf < kWN; ++nf) {
      const bool rd = (e_act[nf] == CO_TAP_ACC || e_act[nf] == CO_TAP_EMIT) && P0 < wa.M;
      acc[mf][nf] = __builtin_bit_cast(
          v4f, __builtin_amdgcn_raw_buffer_load_b128(rr, rd ? e_ring[nf] + P0 * 4 : kOutOfRange,
                                                     0, 0));
    }
  }

  // LDS unit of this lane's input fragment (pixel lrow, channels 8 lgrp ..)
  // at spatial tap (0, 0), per pixel fragment
  int abase[kWM];
#pragma unroll
  for (int mf = 0; mf < kWM; ++mf) {
    const int P = m0 + (w * kWM + mf) * 16 + lrow;
    int pix = 0;  // pixels past M read staged data that is never stored
    if (P < wa.M) {
      const int b = fdiv(P, wa.fd_So), p = P - b * wa.So;
      const int i = fdiv(p, wa.fd_Wo), j = p - i * g.Wo;
      pix = ((b - b0) * (g.H + g.pH) + i - i0) * wa.cols + j;
    }
    abase[mf] = pix * kGemmPixUnits + lgrp;
  }

  // weight fragment (chunk ch, tap uv, column fragment nf) of this lane:
  // packed as [n_tile][chunk][tap][fragment][lane] x 16 bytes; the loads for
  // the k-steps past the last chunk read the next tile's weights or the
  // out-of-range zero, and are never used
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(wp, wa.w_bytes);
  const int wlane = lane * 16;
  const int wtile = n_tile * wa.n_chunks;
  v8bf bq[kNB][kWN];
  auto load_b = [&](v8bf(&b)[kWN], int ch, int uv) {
    const int base = ((wtile + ch) * kKHW + uv) * kWN * 1024;
#pragma unroll
    for (int nf = 0; nf < kWN; ++nf)
      b[nf] = __builtin_bit_cast(
          v8bf, __builtin_amdgcn_raw_buffer_load_b128(wr, wlane, base + nf * 1024, 0));
  };
#pragma unroll
  for (int k = 0; k < kNB - 1; ++k) load_b(bq[k], 0, k);
  __syncthreads();  // chunk 0 staged

  const int cols5 = wa.cols * kGemmPixUnits;
  const int n = wa.n_chunks;
  v8bf af[kWM];  // input fragments of the current tap, refilled one by one
  for (int ch = 0; ch < n; ++ch) {
    const uint4* As = smem + (ch & 1) * a_units;
    auto tap_off = [&](int uv) { return (uv / 3) * cols5 + (uv % 3) * kGemmPixUnits; };
#pragma unroll
    for (int mf = 0; mf < kWM; ++mf) af[mf] = __builtin_bit_cast(v8bf, As[abase[mf]]);
#pragma unroll
    for (int uv = 0; uv < kKHW; ++uv) {
      // weights kNB - 1 k-steps ahead, into the set k-step uv - 1 used (the
      // set index depends on the tap only: kKHW is a multiple of kNB)
      static_assert(kKHW % kNB == 0, "weight set index must not depend on the chunk");
      load_b(bq[(uv + kNB - 1) % kNB], ch + (uv + kNB - 1) / kKHW, (uv + kNB - 1) % kKHW);
      __builtin_amdgcn_sched_barrier(0);
      // each input fragment feeds its four matrix instructions, then its
      // register is refilled with the next tap's fragment, which has the
      // rest of this tap's instructions to arrive
#pragma unroll
      for (int mf = 0; mf < kWM; ++mf) {
#pragma unroll
        for (int nf = 0; nf < kWN; ++nf)
          acc[mf][nf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mf], bq[uv % kNB][nf],
                                                                acc[mf][nf], 0, 0, 0);
        if (uv + 1 < kKHW)
          af[mf] = __builtin_bit_cast(v8bf, As[abase[mf] + tap_off(uv + 1)]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __syncthreads();  // chunk ch + 1 staged; buffer ch & 1 free
  }

  // Fused ring epilogue, branch-free: lane (lrow, lgrp) of fragment (mf, nf)
  // holds column n_tile * 64 + nf * 16 + lrow and the four consecutive pixels
  // lgrp * 4 .. + 3 of the fragment (one frame: Ho*Wo % 4 == 0).  START and
  // ACC store the partial sum to the ring; EMIT and EMIT_FRESH add the bias
  // and write y; every other store goes to the out-of-range offset, which
  // drops it.
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(y, wa.y_bytes);
#pragma unroll
  for (int mf = 0; mf < kWM; ++mf) {
    const int P0 = m0 + (w * kWM + mf) * 16 + lgrp * 4;
    const bool in = P0 < wa.M;
    const int Pc = in ? P0 : 0;
    const int b = fdiv(Pc, wa.fd_So), p = Pc - b * wa.So;
#pragma unroll
    for (int nf = 0; nf < kWN; ++nf) {
      const int act = e_act[nf];
      const v4f v = acc[mf][nf];
      const bool st = in && (act == CO_TAP_START || act == CO_TAP_ACC);
      const bool em = in && (act == CO_TAP_EMIT || act == CO_TAP_EMIT_FRESH);
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, v), rr,
                                             st ? e_ring[nf] + P0 * 4 : kOutOfRange, 0, 0);
      const float bo = e_bias[nf];
      const uint32_t lo =
          uint32_t(f32_to_bf16(v[0] + bo)) | (uint32_t(f32_to_bf16(v[1] + bo)) << 16);
      const uint32_t hi =
          uint32_t(f32_to_bf16(v[2] + bo)) | (uint32_t(f32_to_bf16(v[3] + bo)) << 16);
      const int yoff = em ? int(((int64_t(b) * g.Cout + e_o[nf]) * y_bc + p) * 2) : kOutOfRange;
      if (wa.yvec) {
        __builtin_amdgcn_raw_buffer_store_b64(v2u32{lo, hi}, yr, yoff, 0, 0);
      } else {
        __builtin_amdgcn_raw_buffer_store_b16(bf16_t(lo), yr, yoff, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b16(bf16_t(lo >> 16), yr, yoff, 2, 0);
        __builtin_amdgcn_raw_buffer_store_b16(bf16_t(hi), yr, yoff, 4, 0);
        __builtin_amdgcn_raw_buffer_store_b16(bf16_t(hi >> 16), yr, yoff, 6, 0);
      }
    }
  }
}

// Pack W (C_out, C_in, kT, 3, 3) as [n_tile][chunk][tap][fragment][lane]
// 16-byte units: lane (r, q) of fragment nf holds channels chunk * 32 + 8 q ..
// + 7 of column n_tile * 64 + nf * 16 + r (the matrix instruction's B operand
// order), zero past C_in and past kT * C_out.
__global__ __launch_bounds__(kBlock) void pack_gemm_ws_kernel(ConvGeom g, GemmConfig c,
                                                              const bf16_t* __restrict__ w,
                                                              const float* __restrict__ wscale,
                                                              uint4* __restrict__ out) {
  const int64_t total = int64_t(c.n_tiles) * c.n_chunks * kKHW * kWN * 64;
  const int64_t U = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (U >= total) return;
  const int lane = int(U % 64);
  int64_t rest = U / 64;
  const int nf = int(rest % kWN);
  rest /= kWN;
  const int uv = int(rest % kKHW);
  rest /= kKHW;
  const int ch = int(rest % c.n_chunks);
  const int nt = int(rest / c.n_chunks);
  const int n = nt * kNWG + nf * 16 + (lane & 15);
  const int t = n / g.Cout, o = n - t * g.Cout;
  const int u = uv / 3, v = uv % 3;
  union {
    bf16_t e[8];
    uint4 q;
  } pk;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int cc = ch * 32 + (lane >> 4) * 8 + e;
    bf16_t val = 0;
    if (n < g.kT * g.Cout && cc < g.Cin)
      val = scaled_weight<bf16_t>(w[((((int64_t(o) * g.Cin + cc) * g.kT + t) * 3 + u) * 3) + v],
                                  wscale, o);
    pk.e[e] = val;
  }
  out[U] = pk.q;
}

template <bool PAIR>
hipError_t ws_launch(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L, char* state,
                     const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  auto kern = conv_step_gemm_ws_kernel<PAIR>;
  static bool attr_set = false;
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             int(kLdsBytes));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  TapTable tt;
  int t_lo = CO_MAX_TAPS, t_hi = -1;
  for (int t = 0; t < CO_MAX_TAPS; ++t) {
    tt.action[t] = plan.action[t];
    tt.slot[t] = plan.slot[t];
    if (plan.action[t] != CO_TAP_NONE) {
      t_lo = t < t_lo ? t : t_lo;
      t_hi = t;
    }
  }
  if (t_hi < 0) return hipSuccess;
  WsArgs wa;
  wa.M = int32_t(int64_t(g.B) * g.So());
  wa.N = g.kT * g.Cout;
  wa.So = int32_t(g.So());
  wa.m_tiles = c.m_tiles;
  // only the column tiles holding active taps
  wa.n_tile0 = (t_lo * g.Cout) / kNWG;
  wa.n_tile_cnt = int32_t(ceil_div(int64_t(t_hi + 1) * g.Cout, kNWG)) - wa.n_tile0;
  const int64_t tiles = int64_t(wa.m_tiles) * wa.n_tile_cnt;
  wa.tiles_per_xcd = int32_t(ceil_div(tiles, 8));
  wa.n_chunks = c.n_chunks;
  wa.cols = c.cols;
  wa.a_units = int32_t(c.a_units);
  wa.rows = c.max_slots;
  wa.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * 2);
  wa.w_bytes = int32_t(L.weight_bytes);
  wa.ring_bytes = int32_t(int64_t(g.R) * L.ring_slot_elems * 4);
  wa.y_bytes = io.y ? int32_t(((int64_t(g.B) * g.Cout - 1) * io.y_bc + g.So()) * 2) : 0;
  wa.yvec = (reinterpret_cast<uintptr_t>(io.y) % 8) == 0 && (io.y_bc % 4) == 0 ? 1 : 0;
  wa.fd_So = make_fastdiv(uint32_t(wa.So));
  wa.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  wa.fd_Ho = make_fastdiv(uint32_t(g.Ho));
  wa.fd_H = make_fastdiv(uint32_t(g.H));
  wa.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  wa.fd_ntc = make_fastdiv(uint32_t(wa.n_tile_cnt));
  wa.fd_wpi = make_fastdiv(uint32_t(PAIR ? g.W / 2 : g.W));
  hipLaunchKernelGGL(kern, dim3(unsigned(8 * wa.tiles_per_xcd)), dim3(kThreads),
                     size_t(c.lds_bytes), s, g, wa, static_cast<const bf16_t*>(io.x), io.x_bc,
                     static_cast<bf16_t*>(io.y), io.y_bc,
                     reinterpret_cast<const uint4*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems, tt);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_step_gemm_ws(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L,
                                    char* state, const StepIO& io, const co_step_plan& plan,
                                    hipStream_t s) {
  // 32-bit buffer offsets over the packed weights, the ring and y
  if (!c.ws || g.kH != 3 || g.kW != 3 || g.dtype != CO_BF16 || g.So() % 4 != 0 ||
      L.weight_bytes >= (int64_t(1) << 31) ||
      int64_t(g.R) * L.ring_slot_elems * 4 >= (int64_t(1) << 31) ||
      (io.y && ((int64_t(g.B) * g.Cout - 1) * io.y_bc + g.So()) * 2 >= (int64_t(1) << 31)))
    return hipErrorInvalidValue;
  if (g.W % 2 == 0) return ws_launch<true>(g, c, L, state, io, plan, s);
  return ws_launch<false>(g, c, L, state, io, plan, s);
}

hipError_t launch_pack_gemm_ws(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L,
                               char* state, const void* weight, const float* wscale,
                               hipStream_t s) {
  const int64_t total = int64_t(c.n_tiles) * c.n_chunks * kKHW * kWN * 64;
  if (total * 16 != L.weight_bytes) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_gemm_ws_kernel, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                     static_cast<const bf16_t*>(weight), wscale,
                     reinterpret_cast<uint4*>(state + L.weight));
  return hipGetLastError();
}

}  // namespace coinf
