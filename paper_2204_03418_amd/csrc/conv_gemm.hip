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
      const int rest = fdiv(it, ga.fd_wpi);
      const int xp = it - rest * wp_items;
      const int grp = rest & 3;
      const int sl = rest >> 2;
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
  // channels past C_in read the next stream's planes or past the buffer end
  // (zero); they are masked when stored
  // `part` < 0: all of chunk ch's loads; else the share issued during
  // spatial tap `part`, so the loads trickle out between the matrix
  // instructions instead of queueing all at once in front of them
  auto prefetch = [&](int ch, int part) {
    const int cbase = ch * CK;
#pragma unroll
    for (int ai = 0; ai < AI; ++ai)
#pragma unroll
      for (int e = 0; e < KL; ++e)
        if (part < 0 || (ai * KL + e) % KHW == part)
          ra[ai][e] = Stage<T>::load(xr, a_src[ai], (cbase + e) * plane_bytes, PAIR);
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
      val = w[((((int64_t(o) * g.Cin + cc) * g.kT + t) * g.kH + u) * g.kW) + v];
    pk.v[e] = val;
  }
  out[U] = pk.q;
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

hipError_t launch_conv_step_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                                 const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  GemmConfig c;
  if (!gemm_config(g, g.cfg, &c)) return hipErrorInvalidValue;
  // Even-width rows are staged two pixels per load; a frame pointer or plane
  // stride that breaks that alignment takes the direct kernel (same ring).
  const size_t esz = g.dtype == CO_BF16 ? 2 : 4;
  if (g.W % 2 == 0 &&
      ((reinterpret_cast<uintptr_t>(io.x) % (2 * esz)) != 0 || (io.x_bc % 2) != 0))
    return launch_conv_step_direct(g, L, state, io, plan, false, s);
  // staging reads use 32-bit buffer offsets over the reachable part of x
  if (((int64_t(g.B) * g.Cin - 1) * io.x_bc + g.S()) * int64_t(esz) >= (int64_t(1) << 31))
    return launch_conv_step_direct(g, L, state, io, plan, false, s);
  if (g.kH == 3 && g.kW == 3) return gemm_dispatch_taps<3, 3>(g, c, L, state, io, plan, s);
  if (g.kH == 1 && g.kW == 1) return gemm_dispatch_taps<1, 1>(g, c, L, state, io, plan, s);
  return hipErrorInvalidValue;
}

hipError_t launch_pack_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                            const void* weight, hipStream_t s) {
  GemmConfig c;
  if (!gemm_config(g, g.cfg, &c)) return hipErrorInvalidValue;
  const int64_t total = int64_t(c.n_tiles) * c.n_chunks * g.kH * g.kW * c.N_WG * 4;
  uint4* out = reinterpret_cast<uint4*>(state + L.weight);
  if (g.dtype == CO_BF16)
    hipLaunchKernelGGL(pack_gemm_kernel<bf16_t>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                       static_cast<const bf16_t*>(weight), out);
  else
    hipLaunchKernelGGL(pack_gemm_kernel<float>, dim3(grid_for(total)), dim3(kBlock), 0, s, g, c,
                       static_cast<const float*>(weight), out);
  return hipGetLastError();
}

}  // namespace coinf
