// Host-side scheduler: validation, delay, tap plans and state layouts.
#include "schedule.hpp"

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

bool gemm_supported(const ConvGeom& g) {
  (void)g;
  return false;
}

int64_t packed_weight_bytes(const ConvGeom& g) {
  const int64_t n = int64_t(g.Cout) * g.Cg * g.kT * g.kH * g.kW;
  switch (g.algo) {
    case CO_ALGO_GEMM: {
      // [kT][C_out][K_pad] in the io dtype, K padded to the MFMA K step
      const int64_t K = int64_t(g.Cg) * g.kH * g.kW;
      const int64_t kstep = g.dtype == CO_BF16 ? 32 : 8;
      return int64_t(g.kT) * g.Cout * round_up(K, kstep) * (g.dtype == CO_BF16 ? 2 : 4);
    }
    default:
      return n * 4;  // float32, PyTorch order
  }
}

co_status conv_geom(const co_conv_desc* desc, ConvGeom* g) {
  if (!desc || !g) return CO_EINVAL;
  const co_conv_desc& d = *desc;
  if (d.spatial_dims < 0 || d.spatial_dims > 2) return CO_EINVAL;
  if (d.batch < 1 || d.in_channels < 1 || d.out_channels < 1 || d.groups < 1) return CO_EINVAL;
  if (d.in_channels % d.groups || d.out_channels % d.groups) return CO_EINVAL;
  if (d.dtype != CO_F32 && d.dtype != CO_BF16) return CO_EINVAL;
  if (d.has_bias != 0 && d.has_bias != 1) return CO_EINVAL;
  if (d.algo < CO_ALGO_AUTO || d.algo > CO_ALGO_DEPTHWISE) return CO_EINVAL;
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

  int32_t algo = d.algo;
  if (algo == CO_ALGO_AUTO) {
    if (depthwise_supported(r))
      algo = CO_ALGO_DEPTHWISE;
    else
      algo = gemm_supported(r) ? CO_ALGO_GEMM : CO_ALGO_DIRECT;
  } else if (algo == CO_ALGO_DEPTHWISE) {
    if (!depthwise_supported(r)) return CO_ENOTSUP;
  } else if (algo == CO_ALGO_GEMM) {
    if (!gemm_supported(r)) return CO_ENOTSUP;
  }
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
  L.ring = L.weight + round_up(L.weight_bytes, kAlign);
  L.ring_slot_elems = round_up(g.out_frame_elems(), kAlign / 4);
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

}  // namespace coinf
