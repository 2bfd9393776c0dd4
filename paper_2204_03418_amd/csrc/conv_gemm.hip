// Implicit-GEMM continual convolution step on CDNA4 matrix cores (groups = 1).
//
// The per-step contraction of the arriving frame against every temporal tap
// (section 3.1: intermediate results for future outputs are computed eagerly)
// is one GEMM per step:
//
//   C[m][n] = sum_k A[m][k] * B[k][n]
//   m = (b, i, j)        output pixel of stream b            M = B*Ho*Wo
//   n = (tap t, out o)   n = t*C_out + o                      N = kT*C_out
//   k = (u, v, c)        spatial tap, input channel innermost K = kH*kW*C_in
//   A[m][k] = x_t[b][c][i + u - pH][j + v - pW]  (zero outside the frame)
//   B[k][n] = W[o][c][t][u][v]
//
// followed by a fused ring epilogue: column n of the tile updates ring slot
// slot[t] of output channel o according to the tap's action (start, add, or
// complete the output frame, add the bias and write y).  No atomics: each
// (slot, o, pixel) element is touched by exactly one tap in a step.
//
// Data movement.  A workgroup owns a tile of M_WG pixels x N_WG columns.
// Per chunk of CK input channels it stages the input rows its pixels need
// (every row of every stream the tile touches, halo included) into LDS in a
// channels-last layout, transposing the NCHW frame on the way, and copies the
// matching block of pre-packed weights.  Each lane then reads 16-byte operand
// fragments (8 bf16 or 4 fp32 channels of one pixel / one column) straight
// from LDS for v_mfma_f32_16x16x32_bf16 or v_mfma_f32_16x16x4_f32.  Operand
// addresses are a per-lane base plus compile-time offsets (spatial tap,
// stage), so they cost no registers or ALU work inside the loop; padded
// pixels (A) and column-swizzled units (B) keep the reads free of LDS bank
// conflicts.  Tiles are
// numbered so that consecutive tiles run on the same XCD and share its L2.
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kPixUnits = kGemmPixUnits;  // 16-byte units per staged pixel (4 + 1 pad)

// Physical unit of logical channel group `grp` of weight column `n`: the XOR
// spreads 8 consecutive columns over 8 bank groups (it depends on n only, so
// a column's address stays base + tap offset).
__device__ __forceinline__ int bswz(int n, int grp) { return grp ^ ((n >> 1) & 3); }

struct GemmArgs {
  int32_t M, N, So;
  int32_t m_tiles, n_tile0, n_tile_cnt, tiles_per_xcd;
  int32_t n_chunks, cols, max_slots;
  int32_t a_units;  // 16-byte units of one A stage
  int32_t pair;     // rows are read two pixels per load (even width, aligned)
  int32_t x_bytes;  // bytes of x reachable from the frame pointer
  // dividers: pixels per frame, Wo, Ho, H, C_out, column tiles, staging items per row
  FastDiv fd_So, fd_Wo, fd_Ho, fd_H, fd_Cout, fd_ntc, fd_wpi;
};

template <typename T>
struct FragOf;
template <>
struct FragOf<bf16_t> {
  using type = v8bf;
};
template <>
struct FragOf<float> {
  using type = v4f;
};

__device__ __forceinline__ void mma(v4f& acc, const v8bf& a, const v8bf& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}

// fp32: the four channels of a lane's 16-byte unit feed four k = 4 steps;
// A and B use the same channel order, so the sum is the full dot product.
__device__ __forceinline__ void mma(v4f& acc, const v4f& a, const v4f& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc, 0, 0, 0);
}

template <typename T>
__device__ __forceinline__ void store_out(T* y, int64_t i, float v) {
  y[i] = from_f32<T>(v);
}

// Four consecutive outputs; one 8- or 16-byte store when aligned.
template <typename T>
__device__ __forceinline__ void store4(T* y, float a, float b, float c, float d, bool vec);
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* y, float a, float b, float c, float d,
                                               bool vec) {
  if (vec) {
    const uint32_t lo = uint32_t(f32_to_bf16(a)) | (uint32_t(f32_to_bf16(b)) << 16);
    const uint32_t hi = uint32_t(f32_to_bf16(c)) | (uint32_t(f32_to_bf16(d)) << 16);
    *reinterpret_cast<uint2*>(y) = make_uint2(lo, hi);
  } else {
    y[0] = f32_to_bf16(a);
    y[1] = f32_to_bf16(b);
    y[2] = f32_to_bf16(c);
    y[3] = f32_to_bf16(d);
  }
}
template <>
__device__ __forceinline__ void store4<float>(float* y, float a, float b, float c, float d,
                                              bool vec) {
  if (vec) {
    *reinterpret_cast<float4*>(y) = make_float4(a, b, c, d);
  } else {
    y[0] = a;
    y[1] = b;
    y[2] = c;
    y[3] = d;
  }
}

// Raw global loads of one staging item -- KL channels of one pixel, or of two
// adjacent pixels when rows have even width (one 4- or 8-byte load per
// channel) -- and their packing into the two pixels' 16-byte LDS units.
// Bit operations only, so the values stay in registers.
template <typename T>
struct Stage;
template <>
struct Stage<bf16_t> {
  using Pair = uint32_t;  // two bf16 of one channel: pixel x (low), x+1 (high)
  static __device__ __forceinline__ Pair load(__amdgpu_buffer_rsrc_t r, int voff, int soff,
                                              bool pair) {
    return pair ? __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0)
                : uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0));
  }
  static __device__ __forceinline__ void pack(const Pair (&r)[8], uint4& u0, uint4& u1) {
    u0.x = (r[0] & 0xffffu) | (r[1] << 16);
    u0.y = (r[2] & 0xffffu) | (r[3] << 16);
    u0.z = (r[4] & 0xffffu) | (r[5] << 16);
    u0.w = (r[6] & 0xffffu) | (r[7] << 16);
    u1.x = (r[0] >> 16) | (r[1] & 0xffff0000u);
    u1.y = (r[2] >> 16) | (r[3] & 0xffff0000u);
    u1.z = (r[4] >> 16) | (r[5] & 0xffff0000u);
    u1.w = (r[6] >> 16) | (r[7] & 0xffff0000u);
  }
};
template <>
struct Stage<float> {
  using Pair = uint2;  // two fp32 of one channel: pixel x, x+1
  static __device__ __forceinline__ Pair load(__amdgpu_buffer_rsrc_t r, int voff, int soff,
                                              bool pair) {
    if (pair) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
      return make_uint2(v[0], v[1]);
    }
    return make_uint2(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0), 0u);
  }
  static __device__ __forceinline__ void pack(const Pair (&r)[4], uint4& u0, uint4& u1) {
    u0 = make_uint4(r[0].x, r[1].x, r[2].x, r[3].x);
    u1 = make_uint4(r[0].y, r[1].y, r[2].y, r[3].y);
  }
};

template <typename T, int KH, int KW, int WM, int WN, int NWM, int NWN, bool PAIR>
__global__ __launch_bounds__(64 * NWM * NWN) void conv_step_gemm_kernel(
    ConvGeom g, GemmArgs ga, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y,
    int64_t y_bc, const uint4* __restrict__ wp, const float* __restrict__ bias,
    float* __restrict__ ring, int64_t ring_slot, TapTable tt) {
  using Frag = typename FragOf<T>::type;
  using Pair = typename Stage<T>::Pair;
  constexpr int KL = 16 / int(sizeof(T));  // channels per 16-byte unit
  constexpr int CK = 4 * KL;               // channels per LDS chunk
  constexpr int KHW = KH * KW;
  constexpr int NT = 64 * NWM * NWN;
  constexpr int M_WG = 16 * WM * NWM;
  constexpr int N_WG = 16 * WN * NWN;
  constexpr int AI = (kGemmStageItems + NT - 1) / NT;     // A items per thread
  constexpr int B_UNITS = KHW * N_WG * 4;
  constexpr int BI = (B_UNITS + NT - 1) / NT;            // B copies per thread
  extern __shared__ uint4 smem[];

  const int tid = int(threadIdx.x);
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % NWM, wn = wave / NWM;
  const int lrow = lane & 15, lgrp = lane >> 4;

  // XCD-aware numbering: blocks are dealt to the 8 XCDs round-robin, so
  // logical tile L = xcd * tiles_per_xcd + k keeps neighbours on one XCD.
  const int bid = int(blockIdx.x);
  const int L = (bid & 7) * ga.tiles_per_xcd + (bid >> 3);
  if (L >= ga.m_tiles * ga.n_tile_cnt) return;
  const int m_tile = fdiv(L, ga.fd_ntc);
  const int n_tile = ga.n_tile0 + (L - m_tile * ga.n_tile_cnt);
  const int m0 = m_tile * M_WG;
  const int m1 = min(m0 + M_WG, ga.M);

  // input rows of the tile: flattened (stream, row) index q in [q0, q1]
  const int r0 = fdiv(m0, ga.fd_Wo), r1 = fdiv(m1 - 1, ga.fd_Wo);
  const int b0 = fdiv(r0, ga.fd_Ho), i0 = r0 - b0 * g.Ho;
  const int b1 = fdiv(r1, ga.fd_Ho), i1 = r1 - b1 * g.Ho;
  const int q0 = b0 * g.H + max(0, i0 - g.pH);
  const int q1 = b1 * g.H + min(g.H - 1, i1 + KH - 1 - g.pH);
  const int nslots = q1 - q0 + 1;
  const int zero_slot = ga.max_slots;

  // LDS: [A stage 0][A stage 1][B stage 0][B stage 1].  An A stage holds
  // rows of `cols` = W + pW pixels (consecutive rows share their zero halo
  // column), the zero row, and two trash pixels that absorb the writes of
  // staging items a thread does not have.  A pixel is 5 units of 16 bytes:
  // 4 channel groups and one pad, so 8 consecutive pixels hit 8 different
  // bank groups and a tap offset stays a plain address offset.
  const int a_pixels = (ga.max_slots + 2) * ga.cols;
  const int a_units = ga.a_units;  // == (a_pixels + 2) * kPixUnits, sized on the host
  uint4* const As0 = smem;
  uint4* const Bs0 = smem + 2 * a_units;
  for (int u = tid; u < 2 * a_units; u += NT) smem[u] = make_uint4(0u, 0u, 0u, 0u);

  // LDS pixel index of each of this lane's A rows, per spatial tap row u
  int pixbase[WM][KH];
#pragma unroll
  for (int mf = 0; mf < WM; ++mf) {
    const int P = m0 + (wm * WM + mf) * 16 + lrow;
    const bool valid = P < ga.M;
    const int Pc = valid ? P : 0;
    const int b = fdiv(Pc, ga.fd_So), p = Pc - b * ga.So;
    const int i = fdiv(p, ga.fd_Wo), j = p - i * g.Wo;
#pragma unroll
    for (int u = 0; u < KH; ++u) {
      const int ih = i + u - g.pH;
      const int slot = (valid && ih >= 0 && ih < g.H) ? b * g.H + ih - q0 : zero_slot;
      pixbase[mf][u] = slot * ga.cols + j;
    }
  }

  // staging items of this thread: (slot, channel group, pixel or pixel pair).
  // Items past the tile read element 0 and land in the trash pixels.
  constexpr int PW = PAIR ? 2 : 1;
  const int wp_items = g.W / PW;
  const int a_items = nslots * 4 * wp_items;
  int a_src[AI];      // byte offset of the item without the chunk's channel base
  int a_dst[AI];      // LDS unit index of the item's first pixel
  int a_dst1[AI];     // ... and of its second pixel (PAIR)
  int a_grp[AI];
#pragma unroll
  for (int ai = 0; ai < AI; ++ai) {
    const int it = tid + ai * NT;
    a_src[ai] = 0;
    a_grp[ai] = 0;
    a_dst[ai] = a_pixels * kPixUnits;
    a_dst1[ai] = (a_pixels + 1) * kPixUnits;
    if (it < a_items) {
      // items run along a row, then down the tile's rows, then over the
      // four channel groups: the lanes of one load instruction read
      // consecutive rows of the same channel plane (a few whole cache lines)
      const int rest = fdiv(it, ga.fd_wpi);
      const int xp = it - rest * wp_items;
      const int grp = rest / nslots;
      const int sl = rest - grp * nslots;
      const int q = q0 + sl;
      const int b = fdiv(q, ga.fd_H), ih = q - b * g.H;
      const int xcol = xp * PW;
      a_src[ai] = int(((int64_t(b) * g.Cin + grp * KL) * x_bc + int64_t(ih) * g.W + xcol) *
                      int64_t(sizeof(T)));
      a_grp[ai] = grp;
      const int pix = sl * ga.cols + xcol + g.pW;
      a_dst[ai] = pix * kPixUnits + grp;
      a_dst1[ai] = (pix + 1) * kPixUnits + grp;
    }
  }

  Pair ra[AI][KL];
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, ga.x_bytes);
  const int plane_bytes = int(x_bc * int64_t(sizeof(T)));
  // Channels past C_in (a ragged last chunk) read the out-of-range offset
  // (zero) and are masked again when stored.  `part` < 0: all of chunk ch's
  // loads; else the share issued during spatial tap `part`, so the loads
  // trickle out between the matrix instructions instead of queueing all at
  // once in front of them.
  auto prefetch = [&](int ch, int part) {
    const int cbase = ch * CK;
#pragma unroll
    for (int ai = 0; ai < AI; ++ai)
#pragma unroll
      for (int e = 0; e < KL; ++e)
        if (part < 0 || (ai * KL + e) % KHW == part) {
          const bool cin = cbase + a_grp[ai] * KL + e < g.Cin;
          ra[ai][e] = Stage<T>::load(xr, cin ? a_src[ai] : kOutOfRange,
                                     (cbase + e) * plane_bytes, PAIR);
        }
  };
  auto store_a = [&](int buf, int ch) {
    uint4* As = As0 + buf * a_units;
    const bool ragged = ch * CK + CK > g.Cin;
#pragma unroll
    for (int ai = 0; ai < AI; ++ai) {
      if (ragged) {  // channels past C_in were read clamped: zero them
        const int c0 = ch * CK + a_grp[ai] * KL;
#pragma unroll
        for (int e = 0; e < KL; ++e)
          if (c0 + e >= g.Cin) ra[ai][e] = Pair{};
      }
      uint4 p0, p1;
      Stage<T>::pack(ra[ai], p0, p1);
      As[a_dst[ai]] = p0;
      if (PAIR) As[a_dst1[ai]] = p1;
    }
  };
  // B: the pre-packed block of (n_tile, ch) goes straight from global memory
  // into LDS (global_load_lds_dwordx4; each wave fills 1 KB contiguously)
  auto copy_b = [&](int ch, int buf, int part) {
    const uint4* wsrc = wp + (int64_t(n_tile) * ga.n_chunks + ch) * B_UNITS;
    uint4* Bs = Bs0 + buf * B_UNITS;
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) {
      const int u0 = wave * 64 + bi * NT;  // first unit of this wave's 1 KB
      if ((part < 0 || bi % KHW == part) && u0 < B_UNITS)
        __builtin_amdgcn_global_load_lds(wsrc + u0 + lane,
                                         (__attribute__((address_space(3))) void*)(Bs + u0),
                                         16, 0, 0);
    }
  };

  v4f acc[WM][WN];
#pragma unroll
  for (int mf = 0; mf < WM; ++mf)
#pragma unroll
    for (int nf = 0; nf < WN; ++nf) acc[mf][nf] = v4f{0.f, 0.f, 0.f, 0.f};

  // epilogue data of this lane's columns, resolved before the main loop so
  // the tap table reads are long done when the epilogue runs
  int e_act[WN], e_o[WN];
  float e_bias[WN];
  float* e_ring[WN];
  const bool e_yvec = (y_bc % 4) == 0 &&
                      (reinterpret_cast<uintptr_t>(y) % (4 * sizeof(T))) == 0;
#pragma unroll
  for (int nf = 0; nf < WN; ++nf) {
    const int n = n_tile * N_WG + (wn * WN + nf) * 16 + lrow;
    const int nn = n < ga.N ? n : ga.N - 1;
    const int t = fdiv(nn, ga.fd_Cout), o = nn - t * g.Cout;
    e_act[nf] = n < ga.N ? int(tt.action[t]) : CO_TAP_NONE;
    e_o[nf] = o;
    e_bias[nf] = bias[o];
    const int sl = tt.slot[t] < 0 ? 0 : tt.slot[t];
    e_ring[nf] = ring + int64_t(sl) * ring_slot + int64_t(o) * ga.M;
  }

  // Accumulators start from the partial sum the ring already holds for the
  // taps that add to it (ACC, EMIT) and from zero otherwise, so the MFMAs
  // accumulate straight onto the ring value; the reads are issued here and
  // land while the first chunk is staged.
  const bool vec_epi = (ga.M % 4) == 0;
#pragma unroll
  for (int nf = 0; nf < WN; ++nf) {
    const bool rd = e_act[nf] == CO_TAP_ACC || e_act[nf] == CO_TAP_EMIT;
#pragma unroll
    for (int mf = 0; mf < WM; ++mf) {
      const int P0 = m0 + (wm * WM + mf) * 16 + lgrp * 4;
      if (rd && P0 < ga.M) {
        if (vec_epi) {
          acc[mf][nf] = *reinterpret_cast<const v4f*>(e_ring[nf] + P0);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (P0 + r < ga.M) acc[mf][nf][r] = e_ring[nf][P0 + r];
        }
      }
    }
  }

  // B fragment LDS units of this lane (column n, logical unit lgrp)
  int bbase[WN];
#pragma unroll
  for (int nf = 0; nf < WN; ++nf) {
    const int n = (wn * WN + nf) * 16 + lrow;
    bbase[nf] = n * 4 + bswz(n, lgrp);
  }

  __syncthreads();  // zero fill done
  copy_b(0, 0, -1);
  prefetch(0, -1);
  store_a(0, 0);
  __builtin_amdgcn_s_waitcnt(0);  // LDS-direct loads of B have landed
  __syncthreads();
  for (int ch = 0; ch < ga.n_chunks; ++ch) {
    const bool more = ch + 1 < ga.n_chunks;
    const uint4* As = As0 + (ch & 1) * a_units;
    const uint4* Bs = Bs0 + (ch & 1) * B_UNITS;
    Frag af[2][WM], bf[2][WN];
    auto load_frags = [&](int uv, int k) {
      const int u = uv / KW, v = uv % KW;
#pragma unroll
      for (int mf = 0; mf < WM; ++mf)
        af[k][mf] = __builtin_bit_cast(Frag, As[(pixbase[mf][u] + v) * kPixUnits + lgrp]);
#pragma unroll
      for (int nf = 0; nf < WN; ++nf)
        bf[k][nf] = __builtin_bit_cast(Frag, Bs[uv * N_WG * 4 + bbase[nf]]);
    };
    load_frags(0, 0);
#pragma unroll
    for (int uv = 0; uv < KHW; ++uv) {
      // the next tap's fragments are requested before this tap's MFMAs, so
      // LDS latency hides behind WM*WN matrix instructions
      if (uv + 1 < KHW) load_frags(uv + 1, (uv + 1) & 1);
      if (more) {  // next chunk's global loads are in flight during the MFMAs
        copy_b(ch + 1, (ch + 1) & 1, uv);
        prefetch(ch + 1, uv);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mf = 0; mf < WM; ++mf)
#pragma unroll
        for (int nf = 0; nf < WN; ++nf) mma(acc[mf][nf], af[uv & 1][mf], bf[uv & 1][nf]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (more) store_a((ch + 1) & 1, ch + 1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  // Fused ring epilogue.  Lane (lrow, lgrp) of fragment (mf, nf) holds column
  // n = ... + lrow and the four consecutive pixels lgrp*4 .. lgrp*4+3.  The
  // ring is (slot, C_out, B*Ho*Wo), so those four pixels are contiguous.
  if (vec_epi) {
    // the accumulators already include the ring value: stores only
#pragma unroll
    for (int mf = 0; mf < WM; ++mf) {
      const int P0 = m0 + (wm * WM + mf) * 16 + lgrp * 4;
      if (P0 >= ga.M) continue;
      const int b = fdiv(P0, ga.fd_So), p = P0 - b * ga.So;
      const bool same_frame = p + 3 < ga.So;
#pragma unroll
      for (int nf = 0; nf < WN; ++nf) {
        const int act = e_act[nf];
        const v4f v = acc[mf][nf];
        if (act == CO_TAP_START || act == CO_TAP_ACC) {
          *reinterpret_cast<v4f*>(e_ring[nf] + P0) = v;
        } else if (act == CO_TAP_EMIT || act == CO_TAP_EMIT_FRESH) {
          const float bo = e_bias[nf];
          const int o = e_o[nf];
          if (same_frame) {
            T* yp = y + (int64_t(b) * g.Cout + o) * y_bc + p;
            store4<T>(yp, v[0] + bo, v[1] + bo, v[2] + bo, v[3] + bo, e_yvec);
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int bb = fdiv(P0 + r, ga.fd_So), pp = (P0 + r) - bb * ga.So;
              store_out<T>(y, (int64_t(bb) * g.Cout + o) * y_bc + pp, v[r] + bo);
            }
          }
        }
      }
    }
  } else {
    // ragged pixel count: element-wise
#pragma unroll
    for (int nf = 0; nf < WN; ++nf) {
      const int act = e_act[nf];
      if (act == CO_TAP_NONE) continue;
#pragma unroll
      for (int mf = 0; mf < WM; ++mf) {
        const int P0 = m0 + (wm * WM + mf) * 16 + lgrp * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int P = P0 + r;
          if (P >= ga.M) continue;
          const float v = acc[mf][nf][r];
          if (act == CO_TAP_START || act == CO_TAP_ACC) {
            e_ring[nf][P] = v;
          } else {
            const int b = fdiv(P, ga.fd_So), p = P - b * ga.So;
            store_out<T>(y, (int64_t(b) * g.Cout + e_o[nf]) * y_bc + p, v + e_bias[nf]);
          }
        }
      }
    }
  }
}

// Pack W (C_out, C_in, kT, kH, kW) into [n_tile][chunk][uv][N_WG][4 units of
// KL channels], zero padded, in exactly the order the kernel reads from LDS.
template <typename T>
__global__ __launch_bounds__(kBlock) void pack_gemm_kernel(ConvGeom g, GemmConfig c,
                                                           const T* __restrict__ w,
                                                           const float* __restrict__ wscale,
                                                           uint4* __restrict__ out) {
  constexpr int KL = 16 / int(sizeof(T));
  const int64_t khw = int64_t(g.kH) * g.kW;
  const int64_t total = int64_t(c.n_tiles) * c.n_chunks * khw * c.N_WG * 4;
  const int64_t U = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (U >= total) return;
  const int phys = int(U % 4);
  int64_t rest = U / 4;
  const int nl = int(rest % c.N_WG);
  rest /= c.N_WG;
  const int uv = int(rest % khw);
  rest /= khw;
  const int ch = int(rest % c.n_chunks);
  const int nt = int(rest / c.n_chunks);
  const int grp = phys ^ ((nl >> 1) & 3);  // inverse of bswz
  const int n = nt * c.N_WG + nl;
  const int t = n / g.Cout, o = n - t * g.Cout;
  const int u = uv / g.kW, v = uv % g.kW;
  union {
    T v[KL];
    uint4 q;
  } pk;
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    const int cc = ch * c.CK + grp * KL + e;
    T val = T(0);
    if (n < g.kT * g.Cout && cc < g.Cin)
      val = scaled_weight<T>(w[((((int64_t(o) * g.Cin + cc) * g.kT + t) * g.kH + u) * g.kW) + v],
                             wscale, o);
    pk.v[e] = val;
  }
  out[U] = pk.q;
}

// ---- persistent forward_steps (bf16) -----------------------------------
//
// Temporal stride and dilation 1: the frame at virtual time v feeds output
// v - j through temporal tap j.  A workgroup owns M_WG pixels x O_WG output
// channels for every tap (column c = t * O_WG + o_local), so the partial sums
// of its outputs never leave its registers: the ring is read once at the
// start of a call and written once at the end.  Each wave holds WM pixel
// fragments x one channel fragment x every tap.  A frame is the step kernel's
// GEMM with the same k order (32-channel chunks outer, spatial taps inner),
// and each tap's accumulators start from the partial sum exactly as the step
// kernel starts them from the ring, so the results equal stepping bit for
// bit.
//
// Pipeline: input chunks are staged as in the step kernel (double buffered);
// weights stream in stages of one chunk x one kernel row (triple buffered,
// requested two stages ahead with global_load_lds).  At the end of a stage a
// wave waits until at most the memory requests it issued in that stage are
// outstanding -- the next stage's weights, requested a stage earlier, have
// then landed -- and the workgroup meets at a barrier.

struct GemmSteps {
  int32_t M, So;
  int32_t m_tiles, o_tiles, tiles_per_xcd;
  int32_t n_chunks, cols, max_slots, a_units;
  int32_t x_bytes;
  int32_t fstride;    // bytes between consecutive frames of the clip
  int32_t y_bc;       // y elements between (stream, channel) planes
  int32_t ring_slot;  // floats between ring slots
  int32_t v0;         // virtual time of the first frame, capped at 2^29
  int32_t slot_v0;    // v0 mod R (uncapped)
  int32_t count, T, k0, update;
  int32_t yvec;       // four outputs of a lane can go out as one 8-byte store
  FastDiv fd_So, fd_Wo, fd_Ho, fd_H, fd_ot, fd_wpi;
};

// s_waitcnt immediate: wait until at most n vector memory requests are
// outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14; expcnt and
// lgkmcnt at their maxima, i.e. not waited for).
constexpr int vm_wait(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

template <int KH, int KW, bool PAIR>
__global__ __launch_bounds__(64 * kStepsNWM * kStepsNWN) void conv_steps_gemm_kernel(
    ConvGeom g, GemmSteps gs, const bf16_t* __restrict__ x, int64_t x_bc,
    bf16_t* __restrict__ y, const uint4* __restrict__ wp, const float* __restrict__ bias,
    float* __restrict__ ring) {
  using T = bf16_t;
  using Frag = v8bf;
  using Pair = typename Stage<T>::Pair;
  constexpr int WM = kStepsWM, NWM = kStepsNWM, NWN = kStepsNWN, KTM = kStepsKT;
  constexpr int KL = 8, CK = 32;
  constexpr int NT = 64 * NWM * NWN;
  constexpr int M_WG = 16 * WM * NWM;
  constexpr int O_WG = 16 * NWN;
  constexpr int N_WG = KTM * O_WG;
  constexpr int AI = (kStepsStageItems + NT - 1) / NT;
  constexpr int B_UNITS = KW * N_WG * 4;        // one weight stage
  constexpr int BI = (B_UNITS + NT - 1) / NT;  // weight copies per thread and stage
  constexpr int ALOADS = AI * KL;              // input loads per thread and chunk
  static_assert(B_UNITS >= NT && B_UNITS % 64 == 0, "weight stage shape");
  extern __shared__ uint4 smem[];

  const int tid = int(threadIdx.x);
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % NWM, wn = wave / NWM;
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int bid = int(blockIdx.x);
  const int L = (bid & 7) * gs.tiles_per_xcd + (bid >> 3);
  if (L >= gs.m_tiles * gs.o_tiles) return;
  const int m_tile = fdiv(L, gs.fd_ot);
  const int o_tile = L - m_tile * gs.o_tiles;
  const int m0 = m_tile * M_WG;
  const int m1 = min(m0 + M_WG, gs.M);
  const int kT = g.kT;

  // input rows of the tile: flattened (stream, row) index q in [q0, q1]
  const int r0 = fdiv(m0, gs.fd_Wo), r1 = fdiv(m1 - 1, gs.fd_Wo);
  const int b0 = fdiv(r0, gs.fd_Ho), i0 = r0 - b0 * g.Ho;
  const int b1 = fdiv(r1, gs.fd_Ho), i1 = r1 - b1 * g.Ho;
  const int q0 = b0 * g.H + max(0, i0 - g.pH);
  const int q1 = b1 * g.H + min(g.H - 1, i1 + KH - 1 - g.pH);
  const int nslots = q1 - q0 + 1;
  const int zero_slot = gs.max_slots;

  // LDS: [A stage 0][A stage 1][B stage 0][B stage 1][B stage 2], the A
  // stages laid out as in the step kernel
  const int a_pixels = (gs.max_slots + 2) * gs.cols;
  const int a_units = gs.a_units;
  uint4* const As0 = smem;
  uint4* const Bs0 = smem + 2 * a_units;
  for (int u = tid; u < 2 * a_units; u += NT) smem[u] = make_uint4(0u, 0u, 0u, 0u);

  int pixbase[WM][KH];
#pragma unroll
  for (int mf = 0; mf < WM; ++mf) {
    const int P = m0 + (wm * WM + mf) * 16 + lrow;
    const bool valid = P < gs.M;
    const int Pc = valid ? P : 0;
    const int b = fdiv(Pc, gs.fd_So), p = Pc - b * gs.So;
    const int i = fdiv(p, gs.fd_Wo), j = p - i * g.Wo;
#pragma unroll
    for (int u = 0; u < KH; ++u) {
      const int ih = i + u - g.pH;
      const int slot = (valid && ih >= 0 && ih < g.H) ? b * g.H + ih - q0 : zero_slot;
      pixbase[mf][u] = slot * gs.cols + j;
    }
  }

  constexpr int PW = PAIR ? 2 : 1;
  const int wp_items = g.W / PW;
  const int a_items = nslots * 4 * wp_items;
  int a_src[AI], a_dst[AI], a_dst1[AI], a_grp[AI];
#pragma unroll
  for (int ai = 0; ai < AI; ++ai) {
    const int it = tid + ai * NT;
    a_src[ai] = 0;
    a_grp[ai] = 0;
    a_dst[ai] = a_pixels * kPixUnits;
    a_dst1[ai] = (a_pixels + 1) * kPixUnits;
    if (it < a_items) {
      // items run along a row, then down the tile's rows, then over the
      // four channel groups: the lanes of one load instruction read
      // consecutive rows of the same channel plane (a few whole cache lines)
      const int rest = fdiv(it, gs.fd_wpi);
      const int xp = it - rest * wp_items;
      const int grp = rest / nslots;
      const int sl = rest - grp * nslots;
      const int q = q0 + sl;
      const int b = fdiv(q, gs.fd_H), ih = q - b * g.H;
      const int xcol = xp * PW;
      a_src[ai] = int(((int64_t(b) * g.Cin + grp * KL) * x_bc + int64_t(ih) * g.W + xcol) *
                      int64_t(sizeof(T)));
      a_grp[ai] = grp;
      const int pix = sl * gs.cols + xcol + g.pW;
      a_dst[ai] = pix * kPixUnits + grp;
      a_dst1[ai] = (pix + 1) * kPixUnits + grp;
    }
  }

  Pair ra[AI][KL];
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, gs.x_bytes);
  const int plane_bytes = int(x_bc * int64_t(sizeof(T)));
  // input loads of chunk ch of frame t; end-padding frames stage zeros and
  // issue nothing (the return value says whether loads went out)
  auto prefetch = [&](int t, int ch) -> bool {
    if (t >= gs.T) {
#pragma unroll
      for (int ai = 0; ai < AI; ++ai)
#pragma unroll
        for (int e = 0; e < KL; ++e) ra[ai][e] = Pair{};
      return false;
    }
    const int cbase = ch * CK;
    const int fo = t * gs.fstride;
#pragma unroll
    for (int ai = 0; ai < AI; ++ai)
#pragma unroll
      for (int e = 0; e < KL; ++e) {
        const bool cin = cbase + a_grp[ai] * KL + e < g.Cin;
        ra[ai][e] = Stage<T>::load(xr, cin ? a_src[ai] : kOutOfRange,
                                   (cbase + e) * plane_bytes + fo, PAIR);
      }
    return true;
  };
  auto store_a = [&](int buf, int ch) {
    uint4* As = As0 + buf * a_units;
    const bool ragged = ch * CK + CK > g.Cin;
#pragma unroll
    for (int ai = 0; ai < AI; ++ai) {
      if (ragged) {
        const int c0 = ch * CK + a_grp[ai] * KL;
#pragma unroll
        for (int e = 0; e < KL; ++e)
          if (c0 + e >= g.Cin) ra[ai][e] = Pair{};
      }
      uint4 p0, p1;
      Stage<T>::pack(ra[ai], p0, p1);
      As[a_dst[ai]] = p0;
      if (PAIR) As[a_dst1[ai]] = p1;
    }
  };
  // weight stage st (chunk st / KH, kernel row st % KH) into buffer buf; every
  // wave issues BI copies (a copy past the stage repeats one inside it, with
  // identical data), so the outstanding-request counts below are uniform
  auto copy_b = [&](int st, int buf) {
    const uint4* wsrc = wp + (int64_t(o_tile) * gs.n_chunks * KH + st) * B_UNITS;
    uint4* Bs = Bs0 + buf * B_UNITS;
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) {
      int u0 = wave * 64 + bi * NT;
      if (u0 >= B_UNITS) u0 -= NT;
      __builtin_amdgcn_global_load_lds(wsrc + u0 + lane,
                                       (__attribute__((address_space(3))) void*)(Bs + u0), 16,
                                       0, 0);
    }
  };
  auto wait_stage = [&](bool a, bool b) {
    if (a) {
      if (b)
        __builtin_amdgcn_s_waitcnt(vm_wait(ALOADS + BI));
      else
        __builtin_amdgcn_s_waitcnt(vm_wait(ALOADS));
    } else {
      if (b)
        __builtin_amdgcn_s_waitcnt(vm_wait(BI));
      else
        __builtin_amdgcn_s_waitcnt(0);
    }
  };

  // this lane's output channel, B columns, outputs and partial sums
  const int o = o_tile * O_WG + wn * 16 + lrow;
  const bool ocol = o < g.Cout;
  const float bo = ocol ? bias[o] : 0.f;
  int bcol[KTM];
#pragma unroll
  for (int j = 0; j < KTM; ++j) {
    const int cc = j * O_WG + wn * 16 + lrow;
    bcol[j] = cc * 4 + bswz(cc, lgrp);
  }
  // first of the four pixels of fragment mf this lane holds (recomputed
  // where needed rather than kept in registers across the frame loop)
  auto pix0 = [&](int mf) { return m0 + (wm * WM + mf) * 16 + lgrp * 4; };
  const int R = g.R;
  // part[mf][j - 1]: partial sum of output v - j, continued by tap j >= 1
  v4f part[WM][KTM - 1];
#pragma unroll
  for (int j = 1; j < KTM; ++j)
#pragma unroll
    for (int mf = 0; mf < WM; ++mf) {
      part[mf][j - 1] = v4f{0.f, 0.f, 0.f, 0.f};
      const int tau = gs.v0 - j;
      if (j < kT && tau >= 0) {
        const int sl = (gs.slot_v0 - j + R) % R;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (ocol && pix0(mf) + r < gs.M)
            part[mf][j - 1][r] =
                ring[int64_t(sl) * gs.ring_slot + int64_t(o) * gs.M + pix0(mf) + r];
      }
    }

  const int spf = gs.n_chunks * KH;  // weight stages per frame
  const int total_stages = gs.count * spf;
  __syncthreads();  // zero fill done
  copy_b(0, 0);
  if (total_stages > 1) copy_b(1 % spf, 1);
  prefetch(0, 0);
  store_a(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  v4f c[WM][KTM];
  int gst = 0;  // stages done
  int gch = 0;  // chunks done
  for (int t = 0; t < gs.count; ++t) {
    const int v = gs.v0 + t;
    // accumulators start from the partial sum of the output each tap
    // continues, or from zero where the tap starts it (as the step kernel)
#pragma unroll
    for (int j = 0; j < KTM; ++j) {
      const int tau = v - j;
      const int first = tau >= g.pT ? 0 : g.pT - tau;
      // (tap 0 always starts its output: v >= pT)
      const bool seed = j >= 1 && j < kT && tau >= 0 && j != first;
#pragma unroll
      for (int mf = 0; mf < WM; ++mf)
        c[mf][j] = seed ? part[mf][j > 0 ? j - 1 : 0] : v4f{0.f, 0.f, 0.f, 0.f};
    }
    for (int ch = 0; ch < gs.n_chunks; ++ch, ++gch) {
      const uint4* As = As0 + (gch & 1) * a_units;
      const bool lastc = ch + 1 == gs.n_chunks;
      const int nch = lastc ? 0 : ch + 1;
      const int ntf = lastc ? t + 1 : t;
      const bool anext = ntf < gs.count;
#pragma unroll
      for (int u = 0; u < KH; ++u, ++gst) {
        bool aload = false;
        if (u == 0 && anext) aload = prefetch(ntf, nch);
        const bool b2 = gst + 2 < total_stages;
        if (b2) copy_b((gst + 2) % spf, (gst + 2) % 3);
        const uint4* Bs = Bs0 + (gst % 3) * B_UNITS;
        // a tap's pixel fragments are requested one tap ahead; its weight
        // fragments (shared by all WM rows) just before use
        Frag af[2][WM], bf[KTM];
        auto load_a = [&](int vv, int k) {
#pragma unroll
          for (int mf = 0; mf < WM; ++mf)
            af[k][mf] = __builtin_bit_cast(Frag, As[(pixbase[mf][u] + vv) * kPixUnits + lgrp]);
        };
        load_a(0, 0);
#pragma unroll
        for (int vv = 0; vv < KW; ++vv) {
#pragma unroll
          for (int j = 0; j < KTM; ++j)
            bf[j] = __builtin_bit_cast(Frag, Bs[vv * N_WG * 4 + bcol[j]]);
          // weights before the next tap's pixels: LDS reads complete in
          // order, so the matrix instructions wait for these three only
          __builtin_amdgcn_sched_barrier(0);
          if (vv + 1 < KW) load_a(vv + 1, (vv + 1) & 1);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int j = 0; j < KTM; ++j)
#pragma unroll
            for (int mf = 0; mf < WM; ++mf) mma(c[mf][j], af[vv & 1][mf], bf[j]);
          __builtin_amdgcn_sched_barrier(0);
        }
        if (u == KH - 1 && anext) store_a((gch + 1) & 1, nch);
        wait_stage(aload, b2);
        __syncthreads();
      }
    }
    // the output tap kT - 1 completes goes out with the bias; the others'
    // sums carry on as the partial sums of the next frame
    const int ko = gs.k0 + t;
#pragma unroll
    for (int j = 0; j < KTM; ++j) {
      if (j != kT - 1 || v - j < 0) continue;  // uniform
#pragma unroll
      for (int mf = 0; mf < WM; ++mf) {
        const int p0 = pix0(mf);
        if (!ocol || p0 >= gs.M) continue;
        const v4f a = c[mf][j];
        if (gs.yvec) {  // the four pixels lie in one stream's frame
          const int b = fdiv(p0, gs.fd_So), p = p0 - b * gs.So;
          bf16_t* yp = y + (int64_t(b) * g.Cout + o) * gs.y_bc + int64_t(ko) * gs.So + p;
          store4<T>(yp, a[0] + bo, a[1] + bo, a[2] + bo, a[3] + bo, true);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int P = p0 + r;
            if (P >= gs.M) continue;
            const int b = fdiv(P, gs.fd_So), p = P - b * gs.So;
            store_out<T>(y, (int64_t(b) * g.Cout + o) * gs.y_bc + int64_t(ko) * gs.So + p,
                         a[r] + bo);
          }
        }
      }
    }
#pragma unroll
    for (int j = KTM - 1; j >= 1; --j) {
      const bool carry = j - 1 < kT - 1 && v - (j - 1) >= 0;
#pragma unroll
      for (int mf = 0; mf < WM; ++mf)
        part[mf][j - 1] = carry ? c[mf][j - 1] : v4f{0.f, 0.f, 0.f, 0.f};
    }
  }

  if (gs.update) {
    const int v1 = gs.v0 + gs.count;
    const int s1 = (gs.slot_v0 + gs.count) % R;
#pragma unroll
    for (int j = 1; j < KTM; ++j) {
      if (j >= kT || v1 - j < 0) continue;  // uniform
      const int sl = (s1 - j + R) % R;
#pragma unroll
      for (int mf = 0; mf < WM; ++mf)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (ocol && pix0(mf) + r < gs.M)
            ring[int64_t(sl) * gs.ring_slot + int64_t(o) * gs.M + pix0(mf) + r] = part[mf][j - 1][r];
    }
  }
}

// The same persistent frame loop with the weight fragments read from global
// memory (L2) straight into registers instead of through LDS.  Measured on
// MI355X, streaming the 0.5 MB of weights a workgroup uses per frame through
// LDS made LDS bandwidth the limit: every weight byte was written once and
// read twice there, on top of the pixel fragments.  Read from memory, the two
// waves that share a weight fragment meet in L1, LDS carries only the staged
// input rows, and the workgroup meets at one barrier per 32-channel chunk
// instead of one per kernel row.  Each lane keeps a ring of kStepsBRing
// weight fragment sets, requested kStepsBDist k-steps ahead of use (across
// chunk and frame boundaries: every frame reads the same weights).
//
// Arithmetic is the step kernel's: 16x16x32 bf16 MFMAs in the same k order
// (32-channel chunks outer, spatial taps inner), accumulators seeded with the
// partial sums, so a clip gives the bits of stepping frame by frame.  The
// partial sums stay in the accumulators across frames: after the completing
// tap's output goes out, tap j's accumulators become tap j + 1's.
constexpr int kStepsBRing = 3;  // weight fragment sets in flight per lane
constexpr int kStepsBDist = 2;  // k-steps between a weight request and its use
// Wave layout of this kernel (the workgroup tile is the config's M_WG x O_WG)
constexpr int kWregWM = kStepsWM, kWregNWM = kStepsNWM, kWregNWN = kStepsNWN;
static_assert(16 * kWregWM * kWregNWM == 16 * kStepsWM * kStepsNWM &&
                  kWregNWN == kStepsNWN,
              "the register-weight kernel covers the config's workgroup tile");
constexpr int kWregThreads = 64 * kWregNWM * kWregNWN;

template <int KH, int KW, bool PAIR>
__global__ __launch_bounds__(kWregThreads) void conv_steps_gemm_wreg_kernel(
    ConvGeom g, GemmSteps gs, const bf16_t* __restrict__ x, int64_t x_bc,
    bf16_t* __restrict__ y, const uint4* __restrict__ wp, const float* __restrict__ bias,
    float* __restrict__ ring) {
  using T = bf16_t;
  using Frag = v8bf;
  using Pair = typename Stage<T>::Pair;
  constexpr int WM = kWregWM, NWM = kWregNWM, NWN = kWregNWN, KTM = kStepsKT;
  constexpr int KL = 8, CK = 32;
  constexpr int KHW = KH * KW;  // k-steps per chunk
  constexpr int NT = 64 * NWM * NWN;
  constexpr int M_WG = 16 * WM * NWM;
  constexpr int O_WG = 16 * NWN;
  constexpr int N_WG = KTM * O_WG;
  constexpr int AI = (kStepsStageItems + NT - 1) / NT;
  constexpr int NB = kStepsBRing, DB = kStepsBDist;
  static_assert(KHW % NB == 0 && DB < NB, "weight ring: a chunk's k-steps fill whole rounds");
  constexpr int LPS = (AI * KL + KHW - 1) / KHW;  // input loads per k-step
  static_assert(LPS * KHW >= AI * KL, "input loads spread over the chunk's k-steps");
  extern __shared__ uint4 smem[];

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  // wave index as a scalar: everything derived from it stays wave-uniform
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % NWM, wn = wave / NWM;
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int bid = int(blockIdx.x);
  const int L = (bid & 7) * gs.tiles_per_xcd + (bid >> 3);
  if (L >= gs.m_tiles * gs.o_tiles) return;
  const int m_tile = fdiv(L, gs.fd_ot);
  const int o_tile = L - m_tile * gs.o_tiles;
  const int m0 = m_tile * M_WG;
  const int m1 = min(m0 + M_WG, gs.M);
  const int kT = g.kT;

  // input rows of the tile: flattened (stream, row) index q in [q0, q1]
  const int r0 = fdiv(m0, gs.fd_Wo), r1 = fdiv(m1 - 1, gs.fd_Wo);
  const int b0 = fdiv(r0, gs.fd_Ho), i0 = r0 - b0 * g.Ho;
  const int b1 = fdiv(r1, gs.fd_Ho), i1 = r1 - b1 * g.Ho;
  const int q0 = b0 * g.H + max(0, i0 - g.pH);
  const int q1 = b1 * g.H + min(g.H - 1, i1 + KH - 1 - g.pH);
  const int nslots = q1 - q0 + 1;
  const int zero_slot = gs.max_slots;

  // LDS: [A stage 0][A stage 1], laid out as in the step kernel
  const int a_pixels = (gs.max_slots + 2) * gs.cols;
  const int a_units = gs.a_units;
  uint4* const As0 = smem;
  for (int u = tid; u < 2 * a_units; u += NT) smem[u] = make_uint4(0u, 0u, 0u, 0u);

  int pixbase[WM][KH];
#pragma unroll
  for (int mf = 0; mf < WM; ++mf) {
    const int P = m0 + (wm * WM + mf) * 16 + lrow;
    const bool valid = P < gs.M;
    const int Pc = valid ? P : 0;
    const int b = fdiv(Pc, gs.fd_So), p = Pc - b * gs.So;
    const int i = fdiv(p, gs.fd_Wo), j = p - i * g.Wo;
#pragma unroll
    for (int u = 0; u < KH; ++u) {
      const int ih = i + u - g.pH;
      const int slot = (valid && ih >= 0 && ih < g.H) ? b * g.H + ih - q0 : zero_slot;
      pixbase[mf][u] = slot * gs.cols + j;
    }
  }

  constexpr int PW = PAIR ? 2 : 1;
  const int wp_items = g.W / PW;
  const int a_items = nslots * 4 * wp_items;
  int a_src[AI], a_dst[AI], a_dst1[AI], a_grp[AI];
#pragma unroll
  for (int ai = 0; ai < AI; ++ai) {
    const int it = tid + ai * NT;
    a_src[ai] = 0;
    a_grp[ai] = 0;
    a_dst[ai] = a_pixels * kPixUnits;
    a_dst1[ai] = (a_pixels + 1) * kPixUnits;
    if (it < a_items) {
      // items run along a row, then down the tile's rows, then over the
      // four channel groups: the lanes of one load instruction read
      // consecutive rows of the same channel plane (a few whole cache lines)
      const int rest = fdiv(it, gs.fd_wpi);
      const int xp = it - rest * wp_items;
      const int grp = rest / nslots;
      const int sl = rest - grp * nslots;
      const int q = q0 + sl;
      const int b = fdiv(q, gs.fd_H), ih = q - b * g.H;
      const int xcol = xp * PW;
      a_src[ai] = int(((int64_t(b) * g.Cin + grp * KL) * x_bc + int64_t(ih) * g.W + xcol) *
                      int64_t(sizeof(T)));
      a_grp[ai] = grp;
      const int pix = sl * gs.cols + xcol + g.pW;
      a_dst[ai] = pix * kPixUnits + grp;
      a_dst1[ai] = (pix + 1) * kPixUnits + grp;
    }
  }

  Pair ra[AI][KL];
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, gs.x_bytes);
  const int plane_bytes = int(x_bc * int64_t(sizeof(T)));
  // input load e of chunk ch of frame t (one per k-step, so they trickle out
  // between the matrix instructions).  Branch-free: end-padding frames and
  // frames past the call read the out-of-range offset, i.e. zeros.
  auto prefetch_one = [&](int t, int ch, int e) {
    const int cbase = ch * CK;
    const bool live = t < gs.T;  // uniform
#pragma unroll
    for (int ai = 0; ai < AI; ++ai)
#pragma unroll
      for (int ee = 0; ee < KL; ++ee) {
        if (ai * KL + ee != e) continue;
        const bool cin = live && cbase + a_grp[ai] * KL + ee < g.Cin;
        ra[ai][ee] = Stage<T>::load(xr, cin ? a_src[ai] : kOutOfRange,
                                    live ? (cbase + ee) * plane_bytes + t * gs.fstride : 0, PAIR);
      }
  };
  auto store_a = [&](int buf, int ch) {
    uint4* As = As0 + buf * a_units;
    const bool ragged = ch * CK + CK > g.Cin;
#pragma unroll
    for (int ai = 0; ai < AI; ++ai) {
      if (ragged) {
        const int c0 = ch * CK + a_grp[ai] * KL;
#pragma unroll
        for (int e = 0; e < KL; ++e)
          if (c0 + e >= g.Cin) ra[ai][e] = Pair{};
      }
      uint4 p0, p1;
      Stage<T>::pack(ra[ai], p0, p1);
      As[a_dst[ai]] = p0;
      if (PAIR) As[a_dst1[ai]] = p1;
    }
  };

  // weights of this workgroup's channel tile: k-step ks = ch * KHW + uv is a
  // block of N_WG columns x 4 units; lane (lrow, lgrp) reads its column's unit
  // of logical channel group lgrp (the packing swizzles units within a column)
  const int steps_per_frame = gs.n_chunks * KHW;
  const int wblk_bytes = N_WG * 64;
  const __amdgpu_buffer_rsrc_t wr =
      make_rsrc(wp + int64_t(o_tile) * steps_per_frame * N_WG * 4, steps_per_frame * wblk_bytes);
  int boff[KTM];
#pragma unroll
  for (int j = 0; j < KTM; ++j) {
    const int cc = j * O_WG + wn * 16 + lrow;
    boff[j] = (cc * 4 + bswz(cc, lgrp)) * 16;
  }
  Frag bq[NB][KTM];
  auto load_b = [&](int ks, int slot) {
    const int so = ks * wblk_bytes;
#pragma unroll
    for (int j = 0; j < KTM; ++j)
      bq[slot][j] = __builtin_bit_cast(Frag, __builtin_amdgcn_raw_buffer_load_b128(wr, boff[j], so, 0));
  };

  // this lane's output channel and the first of its four pixels per fragment
  const int o = o_tile * O_WG + wn * 16 + lrow;
  const bool ocol = o < g.Cout;
  const float bo = ocol ? bias[o] : 0.f;
  auto pix0 = [&](int mf) { return m0 + (wm * WM + mf) * 16 + lgrp * 4; };
  const int R = g.R;

  // c[mf][j]: the running sum of output v - j (v = virtual time of the frame
  // being processed).  On entry, taps j >= 1 continue the ring's partial sums
  // unless the stream is at its first frame (then every output starts there).
  v4f c[WM][KTM];
#pragma unroll
  for (int j = 0; j < KTM; ++j)
#pragma unroll
    for (int mf = 0; mf < WM; ++mf) {
      c[mf][j] = v4f{0.f, 0.f, 0.f, 0.f};
      const int tau = gs.v0 - j;
      if (j >= 1 && j < kT && tau >= 0 && gs.v0 > g.pT) {
        const int sl = (gs.slot_v0 - j + R) % R;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (ocol && pix0(mf) + r < gs.M)
            c[mf][j][r] = ring[int64_t(sl) * gs.ring_slot + int64_t(o) * gs.M + pix0(mf) + r];
      }
    }

  __syncthreads();  // zero fill done
#pragma unroll
  for (int d = 0; d < DB; ++d) load_b(d % steps_per_frame, d);
#pragma unroll
  for (int e = 0; e < AI * KL; ++e) prefetch_one(0, 0, e);
  store_a(0, 0);
  __syncthreads();

  int gch = 0;  // chunks done
  for (int t = 0; t < gs.count; ++t) {
    const int v = gs.v0 + t;
#pragma unroll 1
    for (int ch = 0; ch < gs.n_chunks; ++ch, ++gch) {
      const uint4* As = As0 + (gch & 1) * a_units;
      const bool lastc = ch + 1 == gs.n_chunks;
      const int nch = lastc ? 0 : ch + 1;
      const int ntf = lastc ? t + 1 : t;
      const int ks0 = ch * KHW;
      // input fragments of the current tap, refilled one by one: each feeds
      // its KTM matrix instructions, then takes the next tap's fragment,
      // which has the rest of this tap's instructions to arrive (one set of
      // registers instead of two)
      Frag af[WM];
      auto a_at = [&](int uv, int mf) {
        return __builtin_bit_cast(
            Frag, As[(pixbase[mf][uv / KW] + uv % KW) * kPixUnits + lgrp]);
      };
#pragma unroll
      for (int mf = 0; mf < WM; ++mf) af[mf] = a_at(0, mf);
#pragma unroll
      for (int uv = 0; uv < KHW; ++uv) {
        // weights DB k-steps ahead (wrapping into the next frame's first
        // chunk), then the next chunk's input share
        int ks = ks0 + uv + DB;
        if (ks >= steps_per_frame) ks -= steps_per_frame;
        load_b(ks, (uv + DB) % NB);
#pragma unroll
        for (int e = uv * LPS; e < uv * LPS + LPS; ++e)
          if (e < AI * KL) prefetch_one(ntf, nch, e);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mf = 0; mf < WM; ++mf) {
#pragma unroll
          for (int j = 0; j < KTM; ++j) mma(c[mf][j], af[mf], bq[uv % NB][j]);
          if (uv + 1 < KHW) af[mf] = a_at(uv + 1, mf);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // unconditional, also after the call's last chunk (into a buffer no
      // one reads again): a store under a branch lets the compiler sink the
      // input loads from their k-steps into that branch, right before it,
      // which exposes a full memory round trip per chunk
      store_a((gch + 1) & 1, nch);
      __syncthreads();
    }
    // the output tap kT - 1 completes goes out with the bias
    const int ko = gs.k0 + t;
#pragma unroll
    for (int j = 0; j < KTM; ++j) {
      if (j != kT - 1 || v - j < 0) continue;  // uniform
#pragma unroll
      for (int mf = 0; mf < WM; ++mf) {
        const int p0 = pix0(mf);
        if (!ocol || p0 >= gs.M) continue;
        const v4f a = c[mf][j];
        if (gs.yvec) {  // the four pixels lie in one stream's frame
          const int b = fdiv(p0, gs.fd_So), p = p0 - b * gs.So;
          bf16_t* yp = y + (int64_t(b) * g.Cout + o) * gs.y_bc + int64_t(ko) * gs.So + p;
          store4<T>(yp, a[0] + bo, a[1] + bo, a[2] + bo, a[3] + bo, true);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int P = p0 + r;
            if (P >= gs.M) continue;
            const int b = fdiv(P, gs.fd_So), p = P - b * gs.So;
            store_out<T>(y, (int64_t(b) * g.Cout + o) * gs.y_bc + int64_t(ko) * gs.So + p,
                         a[r] + bo);
          }
        }
      }
    }
    // tap j's running sums carry on as tap j + 1's; tap 0 starts afresh
#pragma unroll
    for (int j = KTM - 1; j >= 1; --j)
#pragma unroll
      for (int mf = 0; mf < WM; ++mf) c[mf][j] = c[mf][j - 1];
#pragma unroll
    for (int mf = 0; mf < WM; ++mf) c[mf][0] = v4f{0.f, 0.f, 0.f, 0.f};
  }

  if (gs.update) {
    const int v1 = gs.v0 + gs.count;
    const int s1 = (gs.slot_v0 + gs.count) % R;
#pragma unroll
    for (int j = 1; j < KTM; ++j) {
      if (j >= kT || v1 - j < 0) continue;  // uniform
      const int sl = (s1 - j + R) % R;
#pragma unroll
      for (int mf = 0; mf < WM; ++mf)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (ocol && pix0(mf) + r < gs.M)
            ring[int64_t(sl) * gs.ring_slot + int64_t(o) * gs.M + pix0(mf) + r] = c[mf][j][r];
    }
  }
}

// Pack W (C_out, C_in, kT, kH, kW) into [o_tile][chunk][u][v][column][4 units]
// (column = t * O_WG + o_local), zero padded, with the units swizzled as the
// persistent kernel reads them.
__global__ __launch_bounds__(kBlock) void pack_gemm_steps_kernel(ConvGeom g, GemmStepsConfig c,
                                                                 const bf16_t* __restrict__ w,
                                                                 const float* __restrict__ wscale,
                                                                 uint4* __restrict__ out) {
  const int64_t total = c.weight_bytes / 16;
  const int64_t U = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (U >= total) return;
  const int phys = int(U % 4);
  int64_t rest = U / 4;
  const int col = int(rest % c.N_WG);
  rest /= c.N_WG;
  const int v = int(rest % g.kW);
  rest /= g.kW;
  const int u = int(rest % g.kH);
  rest /= g.kH;
  const int ch = int(rest % c.n_chunks);
  const int ot = int(rest / c.n_chunks);
  const int grp = phys ^ ((col >> 1) & 3);  // inverse of bswz
  const int t = col / c.O_WG, o = ot * c.O_WG + col % c.O_WG;
  union {
    bf16_t v[8];
    uint4 q;
  } pk;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int cc = ch * 32 + grp * 8 + e;
    bf16_t val = 0;
    if (t < g.kT && o < g.Cout && cc < g.Cin)
      val = scaled_weight<bf16_t>(
          w[((((int64_t(o) * g.Cin + cc) * g.kT + t) * g.kH + u) * g.kW) + v], wscale, o);
    pk.v[e] = val;
  }
  out[U] = pk.q;
}

template <int KH, int KW, bool PAIR>
hipError_t gemm_steps_launch(const ConvGeom& g, const GemmStepsConfig& c, const ConvLayout& L,
                             char* state, const void* x, int64_t x_bc, int32_t nreal,
                             int32_t count, void* y, int64_t y_bc, int64_t n0, bool update,
                             hipStream_t s) {
  // the register-weight kernel wherever a chunk's k-steps fill whole rounds
  // of its weight ring (3x3 kernels), else weights through LDS
  constexpr bool wreg = (KH * KW) % kStepsBRing == 0;
  auto kern = [] {
    if constexpr (wreg)
      return conv_steps_gemm_wreg_kernel<KH, KW, PAIR>;
    else
      return conv_steps_gemm_kernel<KH, KW, PAIR>;
  }();
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(kLdsBytes));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  GemmSteps gs;
  gs.M = int32_t(int64_t(g.B) * g.So());
  gs.So = int32_t(g.So());
  gs.m_tiles = c.m_tiles;
  gs.o_tiles = c.o_tiles;
  gs.tiles_per_xcd = int32_t(ceil_div(int64_t(c.m_tiles) * c.o_tiles, 8));
  gs.n_chunks = c.n_chunks;
  gs.cols = c.cols;
  gs.max_slots = c.max_slots;
  gs.a_units = int32_t(c.a_units);
  gs.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * x_bc + int64_t(nreal) * g.S()) * 2);
  gs.fstride = int32_t(g.S() * 2);
  gs.y_bc = int32_t(y_bc);
  gs.ring_slot = int32_t(L.ring_slot_elems);
  const int64_t v0 = n0 + g.pT;
  gs.v0 = int32_t(v0 < (int64_t(1) << 29) ? v0 : (int64_t(1) << 29));
  gs.slot_v0 = int32_t(v0 % g.R);
  gs.count = count;
  gs.T = nreal;
  gs.k0 = int32_t(n0 - (n0 > g.d ? n0 : g.d));
  gs.update = update ? 1 : 0;
  gs.yvec = (g.So() % 4 == 0 && (reinterpret_cast<uintptr_t>(y) % 8) == 0) ? 1 : 0;
  gs.fd_So = make_fastdiv(uint32_t(gs.So));
  gs.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  gs.fd_Ho = make_fastdiv(uint32_t(g.Ho));
  gs.fd_H = make_fastdiv(uint32_t(g.H));
  gs.fd_ot = make_fastdiv(uint32_t(c.o_tiles));
  gs.fd_wpi = make_fastdiv(uint32_t(PAIR ? g.W / 2 : g.W));
  // the register-weight kernel keeps only the two input stages in LDS
  const size_t lds = wreg ? size_t(2 * c.a_units * 16) : size_t(c.lds_bytes);
  hipLaunchKernelGGL(kern, dim3(unsigned(8 * gs.tiles_per_xcd)),
                     dim3(wreg ? kWregThreads : 64 * kStepsNWM * kStepsNWN), lds, s, g, gs,
                     static_cast<const bf16_t*>(x), x_bc, static_cast<bf16_t*>(y),
                     reinterpret_cast<const uint4*>(state + L.steps_weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring));
  return hipGetLastError();
}

template <typename T, int KH, int KW, int WM, int WN, int NWM, int NWN, bool PAIR>
hipError_t gemm_launch(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L, char* state,
                       const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  auto kern = conv_step_gemm_kernel<T, KH, KW, WM, WN, NWM, NWN, PAIR>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
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
  GemmArgs ga;
  ga.M = int32_t(int64_t(g.B) * g.So());
  ga.N = g.kT * g.Cout;
  ga.So = int32_t(g.So());
  ga.m_tiles = c.m_tiles;
  // only the column tiles holding active taps
  ga.n_tile0 = (t_lo * g.Cout) / c.N_WG;
  const int n_end = int(ceil_div(int64_t(t_hi + 1) * g.Cout, c.N_WG));
  ga.n_tile_cnt = n_end - ga.n_tile0;
  const int64_t tiles = int64_t(ga.m_tiles) * ga.n_tile_cnt;
  ga.tiles_per_xcd = int32_t(ceil_div(tiles, 8));
  ga.n_chunks = c.n_chunks;
  ga.cols = c.cols;
  ga.max_slots = c.max_slots;
  ga.a_units = int32_t(c.a_units);
  ga.pair = PAIR ? 1 : 0;
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  ga.x_bytes = int32_t(((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * esz);
  ga.fd_So = make_fastdiv(uint32_t(ga.So));
  ga.fd_Wo = make_fastdiv(uint32_t(g.Wo));
  ga.fd_Ho = make_fastdiv(uint32_t(g.Ho));
  ga.fd_H = make_fastdiv(uint32_t(g.H));
  ga.fd_Cout = make_fastdiv(uint32_t(g.Cout));
  ga.fd_ntc = make_fastdiv(uint32_t(ga.n_tile_cnt));
  ga.fd_wpi = make_fastdiv(uint32_t(PAIR ? g.W / 2 : g.W));
  hipLaunchKernelGGL(kern, dim3(unsigned(8 * ga.tiles_per_xcd)), dim3(64 * NWM * NWN),
                     size_t(c.lds_bytes), s, g, ga, static_cast<const T*>(io.x), io.x_bc,
                     static_cast<T*>(io.y), io.y_bc,
                     reinterpret_cast<const uint4*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems, tt);
  return hipGetLastError();
}

template <int KH, int KW, bool PAIR>
hipError_t gemm_dispatch_cfg(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L,
                             char* state, const StepIO& io, const co_step_plan& plan,
                             hipStream_t s) {
  switch (c.id) {
    case 0: return gemm_launch<bf16_t, KH, KW, 7, 2, 4, 2, PAIR>(g, c, L, state, io, plan, s);
    case 1: return gemm_launch<bf16_t, KH, KW, 2, 2, 1, 4, PAIR>(g, c, L, state, io, plan, s);
    case 2: return gemm_launch<float, KH, KW, 2, 2, 1, 4, PAIR>(g, c, L, state, io, plan, s);
    case 3: return gemm_launch<float, KH, KW, 1, 1, 4, 1, PAIR>(g, c, L, state, io, plan, s);
    default: return hipErrorInvalidValue;
  }
}

template <int KH, int KW>
hipError_t gemm_dispatch_taps(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L,
                              char* state, const StepIO& io, const co_step_plan& plan,
                              hipStream_t s) {
  if (g.W % 2 == 0) return gemm_dispatch_cfg<KH, KW, true>(g, c, L, state, io, plan, s);
  return gemm_dispatch_cfg<KH, KW, false>(g, c, L, state, io, plan, s);
}

}  // namespace

bool gemm_step_needs_staging(const ConvGeom& g, const StepIO& io) {
  // even rows are read as aligned pixel pairs, and the staging reads use
  // 32-bit buffer offsets over the reachable part of x
  const size_t esz = g.dtype == CO_BF16 ? 2 : 4;
  return (g.W % 2 == 0 &&
          ((reinterpret_cast<uintptr_t>(io.x) % (2 * esz)) != 0 || (io.x_bc % 2) != 0)) ||
         ((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * int64_t(esz) >= (int64_t(1) << 31);
}

hipError_t launch_conv_step_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                                 const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  GemmConfig c;
  if (!gemm_config(g, g.cfg, &c)) return hipErrorInvalidValue;
  // A frame pointer or plane stride that breaks the pixel-pair alignment, or
  // a frame past 32-bit reach, is copied into a contiguous buffer first.
  if (gemm_step_needs_staging(g, io)) return launch_conv_step_staged(g, L, state, io, plan, s);
  if (c.ws) return launch_conv_step_gemm_ws(g, c, L, state, io, plan, s);
  if (g.kH == 3 && g.kW == 3) return gemm_dispatch_taps<3, 3>(g, c, L, state, io, plan, s);
  if (g.kH == 1 && g.kW == 1) return gemm_dispatch_taps<1, 1>(g, c, L, state, io, plan, s);
  return hipErrorInvalidValue;
}

bool gemm_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames,
                          const void* x) {
  GemmStepsConfig c;
  if (!gemm_steps_config(g, &c)) return false;
  const int64_t x_bc = x_frames * g.S();
  // even rows are staged two pixels per load: 4-byte aligned pixel pairs
  if (g.W % 2 == 0 && ((x_bc % 2) != 0 || (reinterpret_cast<uintptr_t>(x) % 4) != 0))
    return false;
  const int64_t lim = int64_t(1) << 31;
  return (int64_t(g.B) * g.Cin * x_bc) * 2 < lim && int64_t(g.B) * g.Cout * y_frames * g.So() < lim &&
         int64_t(g.R) * conv_layout(g).ring_slot_elems < lim;
}

hipError_t launch_conv_steps_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                                  const void* x, int64_t x_bc, int32_t nreal, int32_t count,
                                  void* y, int64_t y_bc, int64_t n0, bool update, hipStream_t s) {
  GemmStepsConfig c;
  if (!gemm_steps_config(g, &c) || L.steps_weight_bytes != c.weight_bytes)
    return hipErrorInvalidValue;
  const bool pair = g.W % 2 == 0;
  if (g.kH == 3 && g.kW == 3)
    return pair ? gemm_steps_launch<3, 3, true>(g, c, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s)
                : gemm_steps_launch<3, 3, false>(g, c, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  if (g.kH == 1 && g.kW == 1)
    return pair ? gemm_steps_launch<1, 1, true>(g, c, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s)
                : gemm_steps_launch<1, 1, false>(g, c, L, state, x, x_bc, nreal, count, y, y_bc, n0, update, s);
  return hipErrorInvalidValue;
}

hipError_t launch_pack_gemm_steps(const ConvGeom& g, const ConvLayout& L, char* state,
                                  const void* weight, const float* wscale, hipStream_t s) {
  GemmStepsConfig c;
  if (!gemm_steps_config(g, &c)) return hipSuccess;
  const int64_t total = c.weight_bytes / 16;
  hipLaunchKernelGGL(pack_gemm_steps_kernel, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                     static_cast<const bf16_t*>(weight), wscale,
                     reinterpret_cast<uint4*>(state + L.steps_weight));
  return hipGetLastError();
}

hipError_t launch_pack_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                            const void* weight, const float* wscale, hipStream_t s) {
  GemmConfig c;
  if (!gemm_config(g, g.cfg, &c)) return hipErrorInvalidValue;
  if (c.ws) return launch_pack_gemm_ws(g, c, L, state, weight, wscale, s);
  const int64_t total = int64_t(c.n_tiles) * c.n_chunks * g.kH * g.kW * c.N_WG * 4;
  uint4* out = reinterpret_cast<uint4*>(state + L.weight);
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(pack_gemm_kernel<bf16_t>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                       static_cast<const bf16_t*>(weight), wscale, out);
  else
    hipLaunchKernelGGL(pack_gemm_kernel<float>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                       static_cast<const float*>(weight), wscale, out);
  return hipGetLastError();
}

}  // namespace coinf
