// Host-side scheduler: validation, delay, tap plans and state layouts.
#include "schedule.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>

namespace coinf {

namespace {

constexpr int32_t kMaxI32 = 0x7fffffff;

bool axis_unused_ok(const int32_t* in_size, const int32_t* kernel, const int32_t* stride,
                    const int32_t* padding, const int32_t* dilation, int spatial_dims) {
  for (int a = spatial_dims; a < 2; ++a) {
    if (in_size[a] != 1 || kernel[a + 1] != 1 || stride[a + 1] != 1 || padding[a + 1] != 0 ||
        dilation[a + 1] != 1)
      return false;
  }
  return true;
}

uint64_t fnv1a(uint64_t h, const void* p, size_t n) {
  const unsigned char* c = static_cast<const unsigned char*>(p);
  for (size_t i = 0; i < n; ++i) {
    h ^= c[i];
    h *= 1099511628211ull;
  }
  return h;
}

}  // namespace

bool depthwise_supported(const ConvGeom& g) {
  // stencil sizes the depthwise kernel is instantiated for
  const bool shape = (g.kH == 3 && g.kW == 3) || (g.kH == 1 && g.kW == 1) ||
                     (g.kH == 3 && g.kW == 1) || (g.kH == 5 && g.kW == 5);
  return g.G == g.Cin && g.G == g.Cout && shape && g.kT <= CO_MAX_TAPS;
}

namespace {

struct GemmShape {
  int32_t dtype, WM, WN, NWM, NWN, KL;
};

// Instantiated tile shapes (the kernel file instantiates the same table).
constexpr GemmShape kGemmShapes[kGemmConfigs] = {
    {CO_BF16, 7, 2, 4, 2, 8},  // 448 x 64, 8 waves: large M and N, many channels
    {CO_BF16, 2, 2, 1, 4, 8},  // 32 x 128: small K, wide N
    {CO_F32, 2, 2, 1, 4, 4},   // 32 x 128
    {CO_F32, 1, 1, 4, 1, 4},   // 64 x 16: small N, fills the chip with waves
    {CO_BF16, kWsWM, kWsWN, kWsWaves, 1, 8},  // 448 x 64, warp-specialized (3x3 only)
};

// Input rows a tile of output pixels [m0, m1) needs, over all of its images.
int64_t tile_slots(const ConvGeom& g, int64_t m0, int64_t m1) {
  const int64_t So = g.So();
  const int64_t r0 = m0 / g.Wo, r1 = (m1 - 1) / g.Wo;  // flattened output rows
  const int64_t b0 = r0 / g.Ho, i0 = r0 % g.Ho;
  const int64_t b1 = r1 / g.Ho, i1 = r1 % g.Ho;
  (void)So;
  int64_t q0 = b0 * g.H + std::max<int64_t>(0, i0 - g.pH);
  int64_t q1 = b1 * g.H + std::min<int64_t>(g.H - 1, i1 + g.kH - 1 - g.pH);
  return q1 >= q0 ? q1 - q0 + 1 : 1;
}

}  // namespace

int64_t ring_slot_elems(const ConvGeom& g) {
  // four floats past the frame keep a 16-byte read of the last four pixels
  // of a ragged frame inside the slot
  return round_up(g.out_frame_elems() + 4, kAlign / 4);
}

bool frame_offsets_fit(const ConvGeom& g) {
  const int64_t lim = int64_t(1) << 31;
  const int64_t esz = g.dtype == CO_BF16 ? 2 : 4;
  return int64_t(g.B) * g.Cin * g.S() * esz < lim && g.out_frame_elems() * esz < lim &&
         int64_t(g.R) * ring_slot_elems(g) * 4 < lim;
}

bool gemm_geometry_ok(const ConvGeom& g) {
  const bool taps = (g.kH == 3 && g.kW == 3) || (g.kH == 1 && g.kW == 1);
  return g.G == 1 && taps && g.sH == 1 && g.sW == 1 && g.dH == 1 && g.dW == 1 &&
         g.W + 2 * g.pW <= 256 && frame_offsets_fit(g);
}

// Staged rows of a warp-specialized tile [m0, m1): the images' rows with
// pH zero rows between consecutive images (one image's bottom halo is the
// next one's top halo), from the first row the tile's taps reach to the last.
int64_t ws_tile_rows(const ConvGeom& g, int64_t m0, int64_t m1) {
  const int64_t r0 = m0 / g.Wo, r1 = (m1 - 1) / g.Wo;
  const int64_t b0 = r0 / g.Ho, i0 = r0 % g.Ho;
  const int64_t b1 = r1 / g.Ho, i1 = r1 % g.Ho;
  return (b1 - b0) * (g.H + g.pH) + i1 - i0 + g.kH;
}

bool gemm_config(const ConvGeom& g, int id, GemmConfig* c) {
  if (id < 0 || id >= kGemmConfigs || !gemm_geometry_ok(g)) return false;
  // warp-specialized: 3x3 taps, at most one zero halo row between images
  // and frames of a multiple of 4 pixels (a lane's four outputs are one
  // 16-byte unit of a ring plane and one 8-byte unit of a y plane)
  if (id == kGemmWs && !(g.kH == 3 && g.kW == 3 && g.pH <= 1 && g.Ho == g.H + 2 * g.pH - 2 &&
                         g.So() % 4 == 0))
    return false;
  const GemmShape& s = kGemmShapes[id];
  if (s.dtype != g.dtype) return false;
  GemmConfig r{};
  r.id = id;
  r.dtype = s.dtype;
  r.WM = s.WM;
  r.WN = s.WN;
  r.NWM = s.NWM;
  r.NWN = s.NWN;
  r.KL = s.KL;
  r.CK = 4 * s.KL;
  r.M_WG = 16 * s.WM * s.NWM;
  r.N_WG = 16 * s.WN * s.NWN;
  const int64_t M = int64_t(g.B) * g.So();
  const int64_t N = int64_t(g.kT) * g.Cout;
  r.m_tiles = int32_t(ceil_div(M, r.M_WG));
  r.n_tiles = int32_t(ceil_div(N, r.N_WG));
  r.n_chunks = int32_t(ceil_div(g.Cin, r.CK));
  r.cols = g.W + g.pW;  // staged row pitch: rows share their zero halo column
  int64_t slots = 1;
  for (int64_t t = 0; t < r.m_tiles; ++t)
    slots = std::max(slots, tile_slots(g, t * r.M_WG, std::min<int64_t>(M, (t + 1) * r.M_WG)));
  r.max_slots = int32_t(slots);
  // LDS: two stages of A and two of B, in 16-byte units.  An A stage holds
  // (slots + zero row + halo spill) rows of `cols` pixels plus 2 trash pixels,
  // kGemmPixUnits units per pixel; a B stage kH*kW x N_WG columns x 4 units.
  // The kernel takes a_units from here, so allocation and layout agree.
  r.a_units = ((slots + 2) * r.cols + 2) * kGemmPixUnits;
  r.b_units = int64_t(g.kH) * g.kW * r.N_WG * 4;
  r.lds_bytes = 2 * (r.a_units + r.b_units) * 16;
  r.ws = id == kGemmWs ? 1 : 0;
  r.real_rows = int32_t(slots);
  if (r.ws) {
    // A stages only: every staged row (zero halo rows included), the first
    // pixel of one more row (the last row's right halo) and two trash pixels
    int64_t rows = 1;
    for (int64_t t = 0; t < r.m_tiles; ++t)
      rows = std::max(rows, ws_tile_rows(g, t * r.M_WG, std::min<int64_t>(M, (t + 1) * r.M_WG)));
    r.max_slots = int32_t(rows);
    r.a_units = (rows * r.cols + r.cols + 2) * kGemmPixUnits;
    r.b_units = 0;
    r.lds_bytes = 2 * r.a_units * 16;
  }
  if (r.lds_bytes > kLdsBytes) return false;
  // staging items (row, channel group, pixel pair) must fit the per-thread
  // register budget of the kernel
  const int64_t items = slots * 4 * (g.W % 2 == 0 ? g.W / 2 : g.W);
  if (items > int64_t(kGemmStageItems)) return false;
  *c = r;
  return true;
}

bool gemm_steps_config(const ConvGeom& g, GemmStepsConfig* c) {
  if (g.algo != CO_ALGO_GEMM || g.dtype != CO_BF16 || !gemm_geometry_ok(g) || g.sT != 1 ||
      g.dT != 1 || g.kT > kStepsKT)
    return false;
  GemmStepsConfig r{};
  r.M_WG = 16 * kStepsWM * kStepsNWM;
  r.O_WG = 16 * kStepsNWN;
  r.N_WG = kStepsKT * r.O_WG;
  const int64_t M = int64_t(g.B) * g.So();
  r.m_tiles = int32_t(ceil_div(M, r.M_WG));
  r.o_tiles = int32_t(ceil_div(g.Cout, r.O_WG));
  r.n_chunks = int32_t(ceil_div(g.Cin, 32));
  r.cols = g.W + g.pW;
  int64_t slots = 1;
  for (int64_t t = 0; t < r.m_tiles; ++t)
    slots = std::max(slots, tile_slots(g, t * r.M_WG, std::min<int64_t>(M, (t + 1) * r.M_WG)));
  r.max_slots = int32_t(slots);
  r.a_units = ((slots + 2) * r.cols + 2) * kGemmPixUnits;
  r.b_units = int64_t(g.kW) * r.N_WG * 4;
  r.lds_bytes = (2 * r.a_units + 3 * r.b_units) * 16;
  if (r.lds_bytes > kLdsBytes) return false;
  const int64_t items = slots * 4 * (g.W % 2 == 0 ? g.W / 2 : g.W);
  if (items > int64_t(kStepsStageItems)) return false;
  r.weight_bytes = int64_t(r.o_tiles) * r.n_chunks * g.kH * r.b_units * 16;
  if (r.weight_bytes >= (int64_t(1) << 31)) return false;
  *c = r;
  return true;
}

int gemm_pick(const ConvGeom& g) {
  // LDS-tiled configurations only: the warp-specialized one is its own
  // algorithm (CO_ALGO_GEMM_WS)
  int best = -1;
  double best_cost = 0;
  for (int id = 0; id < kGemmConfigs; ++id) {
    if (id == kGemmWs) continue;
    GemmConfig c;
    if (!gemm_config(g, id, &c)) continue;
    // Cycles of one wave: MFMA issue (bf16 16x16x32: 16 clk per fragment pair
    // per 32 channels; f32 16x16x4: 4 x 32 clk per 16 channels), plus staging
    // per chunk and the epilogue.  Workgroups resident per CU (LDS, 2048
    // threads) give the waves per SIMD; the SIMD's matrix unit completes one
    // instruction about every 30 cycles with one wave on it and every 21 with
    // two or more (bf16 16x16x32, measured), so the resident waves of a SIMD
    // take their turns: a round of workgroups lasts wps waves' worth.
    const int threads = 64 * c.NWM * c.NWN;
    const int64_t wg_cu = std::max<int64_t>(
        1, std::min<int64_t>(kLdsBytes / std::max<int64_t>(c.lds_bytes, 1), 2048 / threads));
    const double wps = double(wg_cu) * c.NWM * c.NWN / 4.0;
    const double mfma = (c.dtype == CO_BF16 ? 16.0 : 128.0) * (wps >= 2.0 ? 21.0 : 30.0) / 16.0;
    const double wave = double(c.WM) * c.WN * c.n_chunks * g.kH * g.kW * mfma +
                        300.0 * c.n_chunks + 100.0 * c.WM * c.WN;
    const double wgs = double(c.m_tiles) * c.n_tiles;
    const double rounds = std::ceil(wgs / (256.0 * double(wg_cu)));
    const double cost = rounds * wave * std::max(1.0, wps);
    if (best < 0 || cost < best_cost) {
      best = id;
      best_cost = cost;
    }
  }
  return best;
}

bool gemm_supported(const ConvGeom& g) { return gemm_pick(g) >= 0; }

namespace {

struct RegShape {
  int32_t dtype, WN, TAPS, CSMAX, KSPLIT;
};

// Instantiated register-GEMM shapes (the kernel file instantiates the same
// table): spatial taps x channel blocks held per tile (the matrix work covers
// all of them, so shapes are sized to common layers: 3x3 taps with up to 24
// fp32 channels, 1x1 with up to 64 or 128), operand registers per lane near
// or below 128 in every shape.  The split shape gives a 3x3 layer with few
// output tiles two waves per tile.
constexpr RegShape kRegShapes[kRegConfigs] = {
    {CO_F32, 4, 1, 16, 1}, {CO_F32, 2, 1, 32, 1}, {CO_F32, 1, 9, 6, 1},
    {CO_F32, 2, 9, 3, 1},  {CO_F32, 1, 10, 6, 2}, {CO_BF16, 4, 1, 2, 1},
    {CO_BF16, 2, 1, 4, 1}, {CO_BF16, 1, 1, 16, 1}, {CO_BF16, 1, 9, 2, 1},
    {CO_BF16, 2, 9, 1, 1},
};

}  // namespace

bool reg_config(const ConvGeom& g, int id, RegConfig* c) {
  // C_out >= 16 keeps every 16-column fragment within two temporal taps
  if (id < 0 || id >= kRegConfigs || g.G != 1 || g.Cout < 16 || !frame_offsets_fit(g))
    return false;
  const RegShape& s = kRegShapes[id];
  if (s.dtype != g.dtype) return false;
  RegConfig r{};
  r.id = id;
  r.dtype = s.dtype;
  r.WN = s.WN;
  r.TAPS = s.TAPS;
  r.KSPLIT = s.KSPLIT;
  r.CSMAX = s.CSMAX;
  r.CKS = g.dtype == CO_BF16 ? 32 : 4;
  r.CS = int32_t(ceil_div(g.Cin, r.CKS));
  const int taps = g.kH * g.kW;
  if (taps > s.TAPS || r.CS > s.CSMAX) return false;
  r.CSU = g.dtype == CO_BF16 ? r.CS : int32_t(ceil_div(r.CS, 4));
  r.KS = taps * r.CS;
  r.U = taps * r.CSU;
  r.m_frags = int32_t(ceil_div(int64_t(g.B) * g.So(), 16));
  r.n_frags = int32_t(ceil_div(int64_t(g.kT) * g.Cout, 16));
  // packed weights and the tile count are addressed with 32-bit offsets
  if (int64_t(r.n_frags) * r.U * 64 * 16 >= (int64_t(1) << 30) ||
      int64_t(r.m_frags) * r.n_frags >= (int64_t(1) << 30))
    return false;
  *c = r;
  return true;
}

int reg_pick(const ConvGeom& g) {
  // Waves (tiles x waves per tile) should cover the 1024 SIMDs; among shapes
  // that do, the widest wave tile (fewer re-reads of the input pixels), then
  // no split, then the smallest register footprint.  When none covers the
  // chip, the one with the most waves.
  int best = -1;
  int64_t best_waves = 0;
  int best_wn = 0, best_split = 0, best_k = 0;
  for (int id = 0; id < kRegConfigs; ++id) {
    RegConfig c;
    if (!reg_config(g, id, &c)) continue;
    const int64_t tiles = int64_t(c.m_frags) * ceil_div(c.n_frags, c.WN);
    const int64_t waves = tiles * c.KSPLIT;
    const bool fills = waves >= 1024;
    const int k = c.TAPS * c.CSMAX;
    bool better;
    if (best < 0) {
      better = true;
    } else {
      const bool best_fills = best_waves >= 1024;
      if (fills != best_fills)
        better = fills;
      else if (!fills && waves != best_waves)
        better = waves > best_waves;
      else if (c.WN != best_wn)
        better = c.WN > best_wn;
      else if (c.KSPLIT != best_split)
        better = c.KSPLIT < best_split;
      else
        better = k < best_k;
    }
    if (better) {
      best = id;
      best_waves = waves;
      best_wn = c.WN;
      best_split = c.KSPLIT;
      best_k = k;
    }
  }
  return best;
}

bool reg_supported(const ConvGeom& g) { return reg_pick(g) >= 0; }

int64_t packed_weight_bytes(const ConvGeom& g) {
  const int64_t n = int64_t(g.Cout) * g.Cg * g.kT * g.kH * g.kW;
  if (g.algo == CO_ALGO_GEMM) {
    // [n_tile][chunk][kH*kW][N_WG][CK] in the io dtype, zero padded
    GemmConfig c;
    if (!gemm_config(g, g.cfg, &c)) return 0;
    return int64_t(c.n_tiles) * c.n_chunks * g.kH * g.kW * c.N_WG * c.CK *
           (g.dtype == CO_BF16 ? 2 : 4);
  }
  if (g.algo == CO_ALGO_GEMM_REG) {
    // [fragment][unit][lane] of 16 bytes, in the matrix instruction's order
    RegConfig c;
    if (!reg_config(g, g.cfg, &c)) return 0;
    return int64_t(c.n_frags) * c.U * 64 * 16;
  }
  return n * 4;  // float32, PyTorch order
}

co_status conv_geom(const co_conv_desc* desc, ConvGeom* g) {
  if (!desc || !g) return CO_EINVAL;
  const co_conv_desc& d = *desc;
  if (d.spatial_dims < 0 || d.spatial_dims > 2) return CO_EINVAL;
  if (d.batch < 1 || d.in_channels < 1 || d.out_channels < 1 || d.groups < 1) return CO_EINVAL;
  if (d.in_channels % d.groups || d.out_channels % d.groups) return CO_EINVAL;
  if (d.dtype != CO_F32 && d.dtype != CO_BF16) return CO_EINVAL;
  if (d.has_bias != 0 && d.has_bias != 1) return CO_EINVAL;
  if (d.algo < CO_ALGO_AUTO || d.algo > CO_ALGO_GEMM_WS) return CO_EINVAL;
  for (int a = 0; a < 3; ++a) {
    if (d.kernel[a] < 1 || d.stride[a] < 1 || d.dilation[a] < 1 || d.padding[a] < 0)
      return CO_EINVAL;
  }
  for (int a = 0; a < 2; ++a)
    if (d.in_size[a] < 1) return CO_EINVAL;
  if (!axis_unused_ok(d.in_size, d.kernel, d.stride, d.padding, d.dilation, d.spatial_dims))
    return CO_EINVAL;
  if (d.kernel[0] > CO_MAX_TAPS) return CO_EINVAL;
  const int64_t f = int64_t(d.dilation[0]) * (d.kernel[0] - 1) + 1;
  if (f > kMaxI32 / 4) return CO_EINVAL;
  if (d.padding[0] > f - 1) return CO_EINVAL;  // negative delay (Principle 4)
  const int64_t Ho = axis_out_len(d.in_size[0], d.kernel[1], d.stride[1], d.padding[1], d.dilation[1]);
  const int64_t Wo = axis_out_len(d.in_size[1], d.kernel[2], d.stride[2], d.padding[2], d.dilation[2]);
  if (Ho < 1 || Wo < 1) return CO_EINVAL;
  // 32-bit element indexing inside a frame
  const int64_t in_frame = int64_t(d.batch) * d.in_channels * d.in_size[0] * d.in_size[1];
  const int64_t out_frame = int64_t(d.batch) * d.out_channels * Ho * Wo;
  const int64_t wcount = int64_t(d.out_channels) * (d.in_channels / d.groups) * d.kernel[0] *
                         d.kernel[1] * d.kernel[2];
  if (in_frame > kMaxI32 || out_frame > kMaxI32 || wcount > kMaxI32) return CO_EINVAL;

  ConvGeom r{};
  r.spatial_dims = d.spatial_dims;
  r.B = d.batch;
  r.Cin = d.in_channels;
  r.Cout = d.out_channels;
  r.G = d.groups;
  r.Cg = d.in_channels / d.groups;
  r.Og = d.out_channels / d.groups;
  r.H = d.in_size[0];
  r.W = d.in_size[1];
  r.Ho = int32_t(Ho);
  r.Wo = int32_t(Wo);
  r.kT = d.kernel[0];
  r.kH = d.kernel[1];
  r.kW = d.kernel[2];
  r.sT = d.stride[0];
  r.sH = d.stride[1];
  r.sW = d.stride[2];
  r.pT = d.padding[0];
  r.pH = d.padding[1];
  r.pW = d.padding[2];
  r.dT = d.dilation[0];
  r.dH = d.dilation[1];
  r.dW = d.dilation[2];
  r.f = int32_t(f);
  r.d = int32_t(f - d.padding[0] - 1);
  // Live partial outputs between steps: ceil((f-1)/sT); one more slot keeps
  // the output that starts and the output that completes in one step apart.
  r.R = int32_t(ceil_div(f - 1, d.stride[0]) + 1);
  r.has_bias = d.has_bias;
  r.dtype = d.dtype;

  r.cfg = -1;
  int32_t algo = d.algo;
  // multiply-accumulates of one step: tiny layers stay on the direct kernel,
  // whose single pass costs less than staging tiles through LDS
  const double macs = double(r.B) * r.So() * r.Cout * r.kT * r.Cg * r.kH * r.kW;
  if (algo == CO_ALGO_AUTO) {
    // Depthwise stencil; else matrix cores: operands in registers below
    // kRegMaxAutoMacs multiply-accumulates per step (one memory round trip
    // per step, which the LDS-staged kernels cannot amortize on small layers;
    // measured on bf16 3x3 and 3x1x1 layers from 14 to 1400 M), above it the
    // warp-specialized GEMM where it applies (faster than the LDS-tiled
    // configurations from 14 to 252 of its tiles), else the LDS-tiled GEMM;
    // tiny layers on the direct kernel.
    GemmConfig wc;
    if (depthwise_supported(r))
      algo = CO_ALGO_DEPTHWISE;
    else if (reg_supported(r) && macs < kRegMaxAutoMacs)
      algo = CO_ALGO_GEMM_REG;
    else if (macs >= 1.0e5 && gemm_config(r, kGemmWs, &wc))
      algo = CO_ALGO_GEMM_WS;
    else if (macs >= 1.0e5 && gemm_supported(r))
      algo = CO_ALGO_GEMM;
    else if (reg_supported(r))
      algo = CO_ALGO_GEMM_REG;
    else
      algo = CO_ALGO_DIRECT;
  } else if (algo == CO_ALGO_DEPTHWISE) {
    if (!depthwise_supported(r)) return CO_ENOTSUP;
  } else if (algo == CO_ALGO_GEMM) {
    if (!gemm_supported(r)) return CO_ENOTSUP;
  } else if (algo == CO_ALGO_GEMM_REG) {
    if (!reg_supported(r)) return CO_ENOTSUP;
  }
  if (algo == CO_ALGO_GEMM_WS) {
    GemmConfig wc;
    if (!gemm_config(r, kGemmWs, &wc)) return CO_ENOTSUP;
    algo = CO_ALGO_GEMM;  // the GEMM family with its warp-specialized configuration
    r.cfg = kGemmWs;
  } else if (algo == CO_ALGO_GEMM) {
    r.cfg = gemm_pick(r);
  }
  if (algo == CO_ALGO_GEMM_REG) r.cfg = reg_pick(r);
  r.algo = algo;
  *g = r;
  return CO_OK;
}

ConvLayout conv_layout(const ConvGeom& g) {
  ConvLayout L{};
  L.header = 0;
  L.bias = kHeaderBytes;
  L.weight = L.bias + round_up(int64_t(g.Cout) * 4, kAlign);
  L.weight_bytes = packed_weight_bytes(g);
  L.steps_weight = L.weight + round_up(L.weight_bytes, kAlign);
  GemmStepsConfig sc;
  L.steps_weight_bytes = gemm_steps_config(g, &sc) ? sc.weight_bytes : 0;
  L.ring = L.steps_weight + round_up(L.steps_weight_bytes, kAlign);
  L.ring_slot_elems = ring_slot_elems(g);
  L.total = L.ring + int64_t(g.R) * L.ring_slot_elems * 4;
  return L;
}

uint64_t conv_hash(const ConvGeom& g) {
  ConvGeom c = g;
  return fnv1a(1469598103934665603ull, &c, sizeof(c));
}

void conv_plan(const ConvGeom& g, int64_t n, bool update_state, co_step_plan* p) {
  std::memset(p, 0, sizeof(*p));
  p->n_taps = g.kT;
  const int64_t v = n + g.pT;  // virtual (padded) time of the arriving frame
  p->emit = (n >= g.d && (n - g.d) % g.sT == 0) ? 1 : 0;
  p->out_index = p->emit ? (n - g.d) / g.sT : -1;
  for (int j = 0; j < CO_MAX_TAPS; ++j) {
    p->slot[j] = -1;
    p->target[j] = -1;
  }
  for (int j = 0; j < g.kT; ++j) {
    const int64_t t = v - int64_t(j) * g.dT;
    if (t < 0 || t % g.sT != 0) continue;
    const int64_t tau = t / g.sT;  // output frame fed by tap j
    // first tap of output tau that falls on a real frame (earlier taps are
    // start padding, which contributes exactly zero)
    const int64_t start = tau * g.sT;
    const int64_t first = start >= g.pT ? 0 : ceil_div(g.pT - start, g.dT);
    int8_t act;
    if (j == g.kT - 1) {
      act = first == g.kT - 1 ? CO_TAP_EMIT_FRESH : CO_TAP_EMIT;
    } else if (!update_state) {
      continue;
    } else {
      act = j == first ? CO_TAP_START : CO_TAP_ACC;
    }
    p->action[j] = act;
    p->target[j] = tau;
    p->slot[j] = act == CO_TAP_EMIT_FRESH ? -1 : int32_t(tau % g.R);
  }
}

bool plan_table_fits(const ConvGeom& g) {
  return g.kT >= 1 && g.kT <= 10 && g.R <= kPlanMaxR && int64_t(g.sT) * g.R <= kPlanPeriod &&
         int64_t(g.kT - 1) * g.dT <= kPlanStart;
}

void plan_table(const ConvGeom& g, int64_t n0, int64_t count, PlanTable* t) {
  auto pack = [&](int64_t n) {
    co_step_plan plan;
    conv_plan(g, n, true, &plan);
    uint64_t code = 0;
    for (int j = 0; j < g.kT; ++j)
      code |= uint64_t(plan.action[j] | (std::max(plan.slot[j], 0) << 3)) << (6 * j);
    return code;
  };
  std::memset(t, 0, sizeof(*t));
  const int64_t n_steady = int64_t(g.kT - 1) * g.dT;
  t->n_start = int32_t(std::max<int64_t>(0, std::min<int64_t>(count, n_steady - n0)));
  t->period = g.sT * g.R;
  for (int i = 0; i < t->n_start; ++i) t->code_start[i] = pack(n0 + i);
  // the periodic table starts at the call's first steady frame
  for (int q = 0; q < t->period; ++q) t->code_period[q] = pack(n0 + t->n_start + q);
}

int64_t conv_emissions(const ConvGeom& g, int64_t n, int64_t count) {
  // emissions at steps m with m >= d and (m - d) % sT == 0, m in [n, n + count)
  const int64_t lo = n > g.d ? n : g.d;
  const int64_t hi = n + count;  // exclusive
  if (hi <= lo) return 0;
  const int64_t first = g.d + ceil_div(lo - g.d, g.sT) * g.sT;
  if (first >= hi) return 0;
  return (hi - 1 - first) / g.sT + 1;
}

co_status pool_geom(const co_pool_desc* desc, PoolGeom* g) {
  if (!desc || !g) return CO_EINVAL;
  const co_pool_desc& d = *desc;
  if (d.kind != CO_POOL_AVG && d.kind != CO_POOL_MAX) return CO_EINVAL;
  if (d.spatial_dims < 0 || d.spatial_dims > 2) return CO_EINVAL;
  if (d.batch < 1 || d.channels < 1) return CO_EINVAL;
  if (d.dtype != CO_F32 && d.dtype != CO_BF16) return CO_EINVAL;
  if (d.count_include_pad != 0 && d.count_include_pad != 1) return CO_EINVAL;
  for (int a = 0; a < 3; ++a) {
    if (d.kernel[a] < 1 || d.stride[a] < 1 || d.dilation[a] < 1 || d.padding[a] < 0)
      return CO_EINVAL;
    if (d.padding[a] > d.kernel[a] / 2) return CO_EINVAL;  // PyTorch's pool rule
    if (d.kind == CO_POOL_AVG && d.dilation[a] != 1) return CO_ENOTSUP;
  }
  for (int a = 0; a < 2; ++a)
    if (d.in_size[a] < 1) return CO_EINVAL;
  if (!axis_unused_ok(d.in_size, d.kernel, d.stride, d.padding, d.dilation, d.spatial_dims))
    return CO_EINVAL;
  if (d.kernel[0] > CO_MAX_TAPS) return CO_EINVAL;
  const int64_t f = int64_t(d.dilation[0]) * (d.kernel[0] - 1) + 1;
  if (f > 4096) return CO_EINVAL;
  const int64_t Ho = axis_out_len(d.in_size[0], d.kernel[1], d.stride[1], d.padding[1], d.dilation[1]);
  const int64_t Wo = axis_out_len(d.in_size[1], d.kernel[2], d.stride[2], d.padding[2], d.dilation[2]);
  if (Ho < 1 || Wo < 1) return CO_EINVAL;
  const int64_t in_frame = int64_t(d.batch) * d.channels * d.in_size[0] * d.in_size[1];
  if (in_frame > kMaxI32) return CO_EINVAL;
  // the step kernels address a frame with 32-bit buffer offsets
  if (in_frame * (d.dtype == CO_BF16 ? 2 : 4) >= (int64_t(1) << 31)) return CO_EINVAL;

  PoolGeom r{};
  r.kind = d.kind;
  r.spatial_dims = d.spatial_dims;
  r.B = d.batch;
  r.C = d.channels;
  r.H = d.in_size[0];
  r.W = d.in_size[1];
  r.Ho = int32_t(Ho);
  r.Wo = int32_t(Wo);
  r.kT = d.kernel[0];
  r.kH = d.kernel[1];
  r.kW = d.kernel[2];
  r.sT = d.stride[0];
  r.sH = d.stride[1];
  r.sW = d.stride[2];
  r.pT = d.padding[0];
  r.pH = d.padding[1];
  r.pW = d.padding[2];
  r.dT = d.dilation[0];
  r.dH = d.dilation[1];
  r.dW = d.dilation[2];
  r.f = int32_t(f);
  r.d = int32_t(f - d.padding[0] - 1);
  r.R = int32_t(f);  // the window's f frames: f - 1 kept plus the arriving one
  r.count_include_pad = d.count_include_pad;
  r.dtype = d.dtype;
  *g = r;
  return CO_OK;
}

PoolLayout pool_layout(const PoolGeom& g) {
  PoolLayout L{};
  L.header = 0;
  L.valid = kHeaderBytes;
  L.fifo = L.valid + round_up(int64_t(g.R) * 4, kAlign);
  L.fifo_slot_elems = round_up(g.out_frame_elems(), kAlign / 4);
  L.total = L.fifo + int64_t(g.R) * L.fifo_slot_elems * 4;
  return L;
}

uint64_t pool_hash(const PoolGeom& g) {
  PoolGeom c = g;
  return fnv1a(1469598103934665603ull ^ 0x5bd1e995ull, &c, sizeof(c));
}

void pool_plan(const PoolGeom& g, int64_t n, co_pool_plan* p) {
  std::memset(p, 0, sizeof(*p));
  p->n_taps = g.kT;
  p->write_slot = int32_t(n % g.R);
  p->emit = (n >= g.d && (n - g.d) % g.sT == 0) ? 1 : 0;
  p->out_index = p->emit ? (n - g.d) / g.sT : -1;
  for (int j = 0; j < CO_MAX_TAPS; ++j) p->src[j] = -1;
  if (!p->emit) return;
  const int64_t tau = p->out_index;
  for (int j = 0; j < g.kT; ++j) {
    const int64_t r = tau * g.sT + int64_t(j) * g.dT - g.pT;  // real frame index
    if (r < 0)
      p->src[j] = -1;
    else if (r == n)
      p->src[j] = -2;
    else
      p->src[j] = int32_t(r % g.R);
  }
}

int64_t pool_emissions(const PoolGeom& g, int64_t n, int64_t count) {
  const int64_t lo = n > g.d ? n : g.d;
  const int64_t hi = n + count;
  if (hi <= lo) return 0;
  const int64_t first = g.d + ceil_div(lo - g.d, g.sT) * g.sT;
  if (first >= hi) return 0;
  return (hi - 1 - first) / g.sT + 1;
}

co_status delay_geom(const co_delay_desc* desc, DelayGeom* g) {
  if (!desc || !g) return CO_EINVAL;
  const co_delay_desc& d = *desc;
  if (d.batch < 1 || d.channels < 1 || d.frame_elems < 1 || d.delay < 0) return CO_EINVAL;
  if (d.dtype != CO_F32 && d.dtype != CO_BF16) return CO_EINVAL;
  DelayGeom r{d.batch, d.channels, d.frame_elems, d.delay, d.dtype};
  if (r.frame() > kMaxI32 || int64_t(r.d) * r.frame() * r.esz() > (int64_t(1) << 40))
    return CO_EINVAL;
  *g = r;
  return CO_OK;
}

uint64_t delay_hash(const DelayGeom& g) {
  return fnv1a(1469598103934665603ull ^ 0x44454c59ull, &g, sizeof(g));
}

}  // namespace coinf
