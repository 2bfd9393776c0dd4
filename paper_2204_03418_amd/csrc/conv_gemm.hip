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
// from LDS for v_mfma_f32_16x16x32_bf16 or v_mfma_f32_16x16x4_f32.  16-byte
// units of a pixel are XOR-swizzled against LDS bank conflicts.  Tiles are
// numbered so that consecutive tiles run on the same XCD and share its L2.
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

struct GemmArgs {
  int32_t M, N, So;
  int32_t m_tiles, n_tile0, n_tile_cnt, tiles_per_xcd;
  int32_t n_chunks, cols, max_slots;
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

// Physical 16-byte unit of logical unit `grp` of pixel/column `idx`.
__device__ __forceinline__ int swz(int idx, int grp) { return grp ^ ((idx >> 1) & 3); }

template <typename T>
__device__ __forceinline__ void store_out(T* y, int64_t i, float v) {
  y[i] = from_f32<T>(v);
}

template <typename T, int KH, int KW, int WM, int WN, int NWM, int NWN>
__global__ __launch_bounds__(64 * NWM * NWN) void conv_step_gemm_kernel(
    ConvGeom g, GemmArgs ga, const T* __restrict__ x, int64_t x_bc, T* __restrict__ y,
    int64_t y_bc, const uint4* __restrict__ wp, const float* __restrict__ bias,
    float* __restrict__ ring, int64_t ring_slot, TapTable tt) {
  using Frag = typename FragOf<T>::type;
  constexpr int KL = 16 / int(sizeof(T));  // channels per 16-byte unit
  constexpr int CK = 4 * KL;               // channels per LDS chunk
  constexpr int KHW = KH * KW;
  constexpr int NT = 64 * NWM * NWN;
  constexpr int M_WG = 16 * WM * NWM;
  constexpr int N_WG = 16 * WN * NWN;
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
  const int m_tile = L / ga.n_tile_cnt;
  const int n_tile = ga.n_tile0 + L % ga.n_tile_cnt;
  const int m0 = m_tile * M_WG;
  const int m1 = min(m0 + M_WG, ga.M);

  // input rows of the tile: flattened (stream, row) index q in [q0, q1]
  const int r0 = m0 / g.Wo, r1 = (m1 - 1) / g.Wo;
  const int b0 = r0 / g.Ho, i0 = r0 % g.Ho;
  const int b1 = r1 / g.Ho, i1 = r1 % g.Ho;
  const int q0 = b0 * g.H + max(0, i0 - g.pH);
  const int q1 = b1 * g.H + min(g.H - 1, i1 + KH - 1 - g.pH);
  const int nslots = q1 - q0 + 1;
  const int zero_slot = ga.max_slots;

  uint4* As = smem;                                      // [(slots+1) * cols][4]
  uint4* Bs = smem + (ga.max_slots + 1) * ga.cols * 4;   // [KHW * N_WG][4]
  const int a_units = (ga.max_slots + 1) * ga.cols * 4;
  for (int u = tid; u < a_units; u += NT) As[u] = make_uint4(0u, 0u, 0u, 0u);

  // LDS pixel index of each of this lane's A rows, per spatial tap row u
  int pixbase[WM][KH];
#pragma unroll
  for (int mf = 0; mf < WM; ++mf) {
    const int P = m0 + (wm * WM + mf) * 16 + lrow;
    const bool valid = P < ga.M;
    const int b = P / ga.So, p = P % ga.So;
    const int i = p / g.Wo, j = p % g.Wo;
#pragma unroll
    for (int u = 0; u < KH; ++u) {
      const int ih = i + u - g.pH;
      const int slot = (valid && ih >= 0 && ih < g.H) ? b * g.H + ih - q0 : zero_slot;
      pixbase[mf][u] = slot * ga.cols + j;
    }
  }

  v4f acc[WM][WN];
#pragma unroll
  for (int mf = 0; mf < WM; ++mf)
#pragma unroll
    for (int nf = 0; nf < WN; ++nf) acc[mf][nf] = v4f{0.f, 0.f, 0.f, 0.f};

  const int a_items = nslots * 4 * g.W;
  const int b_units = KHW * N_WG * 4;
  for (int ch = 0; ch < ga.n_chunks; ++ch) {
    __syncthreads();
    // stage A: item = (slot, channel group, column), column fastest so the
    // global reads of one channel row are coalesced across lanes
    for (int it = tid; it < a_items; it += NT) {
      const int xcol = it % g.W;
      const int rest = it / g.W;
      const int grp = rest & 3;
      const int s = rest >> 2;
      const int q = q0 + s;
      const int b = q / g.H, ih = q - b * g.H;
      const int c0 = ch * CK + grp * KL;
      union {
        T v[KL];
        uint4 u;
      } pk;
      const T* src = x + (int64_t(b) * g.Cin + c0) * x_bc + int64_t(ih) * g.W + xcol;
#pragma unroll
      for (int e = 0; e < KL; ++e) pk.v[e] = (c0 + e < g.Cin) ? src[int64_t(e) * x_bc] : T(0);
      const int pix = s * ga.cols + xcol + g.pW;
      As[pix * 4 + swz(pix, grp)] = pk.u;
    }
    // stage B: the pre-packed (already swizzled) weight block of (n_tile, ch)
    const uint4* wsrc = wp + (int64_t(n_tile) * ga.n_chunks + ch) * b_units;
    for (int u = tid; u < b_units; u += NT) Bs[u] = wsrc[u];
    __syncthreads();

#pragma unroll
    for (int uv = 0; uv < KHW; ++uv) {
      const int u = uv / KW, v = uv % KW;
      Frag af[WM], bf[WN];
#pragma unroll
      for (int mf = 0; mf < WM; ++mf) {
        const int pix = pixbase[mf][u] + v;
        const uint4 t = As[pix * 4 + swz(pix, lgrp)];
        af[mf] = __builtin_bit_cast(Frag, t);
      }
#pragma unroll
      for (int nf = 0; nf < WN; ++nf) {
        const int n = (wn * WN + nf) * 16 + lrow;
        const uint4 t = Bs[(uv * N_WG + n) * 4 + swz(n, lgrp)];
        bf[nf] = __builtin_bit_cast(Frag, t);
      }
#pragma unroll
      for (int mf = 0; mf < WM; ++mf)
#pragma unroll
        for (int nf = 0; nf < WN; ++nf) mma(acc[mf][nf], af[mf], bf[nf]);
    }
  }

  // Fused ring epilogue.  Lane (lrow, lgrp) of fragment (mf, nf) holds column
  // n = ... + lrow and the four consecutive pixels lgrp*4 .. lgrp*4+3.  The
  // ring is (slot, C_out, B*Ho*Wo), so those four pixels are contiguous.
  const bool vec = (ga.M % 4) == 0;
  const bool yvec = (ga.So % 4) == 0 && (y_bc % 4) == 0;
#pragma unroll
  for (int nf = 0; nf < WN; ++nf) {
    const int n = n_tile * N_WG + (wn * WN + nf) * 16 + lrow;
    if (n >= ga.N) continue;
    const int t = n / g.Cout, o = n - t * g.Cout;
    const int act = tt.action[t];
    if (act == CO_TAP_NONE) continue;
    const int slot = tt.slot[t] < 0 ? 0 : tt.slot[t];
    float* rrow = ring + int64_t(slot) * ring_slot + int64_t(o) * ga.M;
    const float bo = bias[o];
#pragma unroll
    for (int mf = 0; mf < WM; ++mf) {
      const int P0 = m0 + (wm * WM + mf) * 16 + lgrp * 4;
      if (P0 >= ga.M) continue;
      const v4f a = acc[mf][nf];
      float vals[4] = {a[0], a[1], a[2], a[3]};
      const bool full = vec && P0 + 3 < ga.M;
      if (act == CO_TAP_START) {
        if (full) {
          *reinterpret_cast<float4*>(rrow + P0) = make_float4(vals[0], vals[1], vals[2], vals[3]);
        } else {
          for (int r = 0; r < 4; ++r)
            if (P0 + r < ga.M) rrow[P0 + r] = vals[r];
        }
      } else if (act == CO_TAP_ACC) {
        if (full) {
          float4 cur = *reinterpret_cast<const float4*>(rrow + P0);
          cur.x += vals[0];
          cur.y += vals[1];
          cur.z += vals[2];
          cur.w += vals[3];
          *reinterpret_cast<float4*>(rrow + P0) = cur;
        } else {
          for (int r = 0; r < 4; ++r)
            if (P0 + r < ga.M) rrow[P0 + r] += vals[r];
        }
      } else {  // EMIT / EMIT_FRESH: complete the output frame
        if (act == CO_TAP_EMIT) {
          if (full) {
            const float4 cur = *reinterpret_cast<const float4*>(rrow + P0);
            vals[0] += cur.x;
            vals[1] += cur.y;
            vals[2] += cur.z;
            vals[3] += cur.w;
          } else {
            for (int r = 0; r < 4; ++r)
              if (P0 + r < ga.M) vals[r] += rrow[P0 + r];
          }
        }
        if (full && yvec) {
          const int b = P0 / ga.So, p = P0 - b * ga.So;
          T* yp = y + (int64_t(b) * g.Cout + o) * y_bc + p;
#pragma unroll
          for (int r = 0; r < 4; ++r) store_out<T>(yp, r, vals[r] + bo);
        } else {
          for (int r = 0; r < 4; ++r) {
            const int P = P0 + r;
            if (P >= ga.M) break;
            const int b = P / ga.So, p = P - b * ga.So;
            store_out<T>(y, (int64_t(b) * g.Cout + o) * y_bc + p, vals[r] + bo);
          }
        }
      }
    }
  }
}

// Pack W (C_out, C_in, kT, kH, kW) into [n_tile][chunk][uv][N_WG][4 units of
// KL channels], zero padded, units pre-swizzled exactly as the kernel reads.
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
  const int grp = phys ^ ((nl >> 1) & 3);
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

template <typename T, int KH, int KW, int WM, int WN, int NWM, int NWN>
hipError_t gemm_launch(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L, char* state,
                       const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  auto kern = conv_step_gemm_kernel<T, KH, KW, WM, WN, NWM, NWN>;
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
  hipLaunchKernelGGL(kern, dim3(unsigned(8 * ga.tiles_per_xcd)), dim3(64 * NWM * NWN),
                     size_t(c.lds_bytes), s, g, ga, static_cast<const T*>(io.x), io.x_bc,
                     static_cast<T*>(io.y), io.y_bc,
                     reinterpret_cast<const uint4*>(state + L.weight),
                     reinterpret_cast<const float*>(state + L.bias),
                     reinterpret_cast<float*>(state + L.ring), L.ring_slot_elems, tt);
  return hipGetLastError();
}

template <int KH, int KW>
hipError_t gemm_dispatch_taps(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L,
                              char* state, const StepIO& io, const co_step_plan& plan,
                              hipStream_t s) {
  switch (c.id) {
    case 0: return gemm_launch<bf16_t, KH, KW, 7, 4, 4, 1>(g, c, L, state, io, plan, s);
    case 1: return gemm_launch<bf16_t, KH, KW, 2, 2, 1, 4>(g, c, L, state, io, plan, s);
    case 2: return gemm_launch<float, KH, KW, 2, 2, 1, 4>(g, c, L, state, io, plan, s);
    case 3: return gemm_launch<float, KH, KW, 1, 1, 4, 1>(g, c, L, state, io, plan, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_conv_step_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                                 const StepIO& io, const co_step_plan& plan, hipStream_t s) {
  GemmConfig c;
  if (!gemm_config(g, g.cfg, &c)) return hipErrorInvalidValue;
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
