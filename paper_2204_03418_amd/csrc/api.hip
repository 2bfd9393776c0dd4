// C ABI of libcoinf: validation, handle bookkeeping and the step loops.
// Every entry point validates on the host before it enqueues anything, so a
// negative status means nothing ran and the handle is unchanged.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <new>
#include <unordered_map>

#include "device.hpp"
#include "launch.hpp"

using namespace coinf;

// Device scratch of co_conv_forward_steps_noalloc: each GPU the library runs
// on holds its own copy until the process ends.  Host code never uses the
// array's name as an address; it asks the runtime for the copy on the
// current device (scratch_address below).
constexpr int64_t kScratchBytes = int64_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct co_conv_handle {
  ConvGeom g;
  ConvLayout L;
  char* state;
  int64_t n;  // frames consumed since the last clean state
};

struct co_pool_handle {
  PoolGeom g;
  PoolLayout L;
  char* state;
  int64_t n;
};

struct co_convpool_handle {
  co_conv_handle* conv;
  co_pool_handle* pool;
};

struct co_bneck_handle {
  co_conv_handle* pw;   // pointwise convolution (1x1x1, delay 0)
  int32_t act1;
  co_conv_handle* dw;   // depthwise convolution
  int32_t act2;
  co_pool_handle* pool;
};

struct co_delay_handle {
  DelayGeom g;
  char* state;
  int64_t n;  // frames consumed since the last clean state
};

namespace {

constexpr int64_t kMaxLaunchElems = int64_t(1) << 38;  // grid limit at 256 threads

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// The persistent direct kernel indexes y with 64-bit offsets; its element
// index per (stream, channel) plane stays 32-bit.
co_status hip_status(hipError_t e) { return e == hipSuccess ? CO_OK : CO_EHIP; }

// Live handles, by kind.  Every entry point checks its handle here, so a
// destroyed handle, a second destroy, or a handle of another kind returns
// CO_EINVAL without touching freed memory.
enum class HKind : uint8_t { Conv, Pool, ConvPool, Delay, Bneck };
std::mutex g_live_mu;
std::unordered_map<const void*, HKind>& live_map() {
  static auto* m = new std::unordered_map<const void*, HKind>();  // kept past exit
  return *m;
}

bool live(const void* h, HKind k) {
  if (!h) return false;
  std::lock_guard<std::mutex> lock(g_live_mu);
  const auto it = live_map().find(h);
  return it != live_map().end() && it->second == k;
}

template <typename H>
co_status publish(H* h, HKind k, H** out) {
  std::lock_guard<std::mutex> lock(g_live_mu);
  live_map()[h] = k;
  *out = h;
  return CO_OK;
}

// Removes a live handle; false when it was not live (already destroyed).
bool retire(const void* h, HKind k) {
  std::lock_guard<std::mutex> lock(g_live_mu);
  const auto it = live_map().find(h);
  if (h == nullptr || it == live_map().end() || it->second != k) return false;
  live_map().erase(it);
  return true;
}

bool any_tap(const co_step_plan& p) {
  for (int j = 0; j < p.n_taps; ++j)
    if (p.action[j] != CO_TAP_NONE) return true;
  return false;
}

co_status read_header(const void* state, hipStream_t s, StateHeader* h) {
  if (hipMemcpyAsync(h, state, sizeof(*h), hipMemcpyDeviceToHost, s) != hipSuccess)
    return CO_EHIP;
  if (hipStreamSynchronize(s) != hipSuccess) return CO_EHIP;
  return CO_OK;
}

// Stream-ordered backup of a byte range, restored by restore_range.
struct Backup {
  void* tmp = nullptr;
  int64_t bytes = 0;
};

co_status backup_range(char* src, int64_t bytes, hipStream_t s, Backup* b) {
  b->bytes = bytes;
  if (bytes == 0) return CO_OK;
  if (hipMallocAsync(&b->tmp, size_t(bytes), s) != hipSuccess) return CO_EHIP;
  if (hipMemcpyAsync(b->tmp, src, size_t(bytes), hipMemcpyDeviceToDevice, s) != hipSuccess)
    return CO_EHIP;
  return CO_OK;
}

co_status restore_range(char* dst, hipStream_t s, Backup* b) {
  if (b->bytes == 0) return CO_OK;
  co_status st = CO_OK;
  if (hipMemcpyAsync(dst, b->tmp, size_t(b->bytes), hipMemcpyDeviceToDevice, s) != hipSuccess)
    st = CO_EHIP;
  if (hipFreeAsync(b->tmp, s) != hipSuccess) st = CO_EHIP;
  b->tmp = nullptr;
  return st;
}

// Device address of `scratch` on the device that runs `stream` (the current
// device for the null stream), looked up once per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

co_status scratch_address(hipStream_t stream, void** out) {
  int cur = 0, dev = 0;
  if (hipGetDevice(&cur) != hipSuccess) return CO_EHIP;
  dev = cur;
  if (stream && hipStreamGetDevice(stream, &dev) != hipSuccess) return CO_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return CO_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return CO_EHIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) return CO_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return CO_OK;
}

int64_t round256(int64_t n) { return (n + 255) & ~int64_t(255); }

// Caller-side device workspace of a forward_steps call (null: the call makes
// stream-ordered allocations instead).
struct Scratch {
  char* p;
  int64_t bytes;
};

co_status conv_forward_steps(co_conv_handle* h, const void* x, int32_t T, void* y,
                             int32_t y_cap_frames, int32_t pad_end, int32_t update_state,
                             hipStream_t s, int32_t* n_out, const Scratch* sc) {
  if (!live(h, HKind::Conv) || T < 0 || y_cap_frames < 0 || !n_out) return CO_EINVAL;
  if (T > 0 && !x) return CO_EINVAL;
  const ConvGeom& g = h->g;
  const int64_t count = int64_t(T) + (pad_end ? g.pT : 0);
  if (count > kMaxSteps - h->n) return CO_EINVAL;
  const int64_t n_emit = conv_emissions(g, h->n, count);
  if (n_emit > y_cap_frames) return CO_EINVAL;
  if (n_emit > 0 && !y) return CO_EINVAL;
  const int64_t n0 = h->n;
  const bool dw = dw_steps_supported(g, T, y_cap_frames);
  const bool dir = direct_steps_supported(g, T, y_cap_frames);
  const bool gem = gemm_steps_supported(g, T, y_cap_frames, x);
  if (count > 0 && (dw || dir || gem || reg_steps_supported(g, T, y_cap_frames))) {
    // one persistent launch: partial sums stay on chip across frames; with
    // update_state = 0 the state is simply not written back
    const auto launch = dw    ? launch_conv_steps_depthwise
                        : dir ? launch_conv_steps_direct
                        : gem ? launch_conv_steps_gemm
                              : launch_conv_steps_reg;
    const co_status st = hip_status(launch(g, h->L, h->state, x, int64_t(T) * g.S(), T,
                                           int32_t(count), y, int64_t(y_cap_frames) * g.So(),
                                           n0, update_state != 0, s));
    if (st != CO_OK) return st;
    if (update_state) h->n += count;
    *n_out = int32_t(n_emit);
    return CO_OK;
  }
  const int64_t S = g.S(), So = g.So();
  const size_t esz = g.dtype == CO_BF16 ? 2 : 4;
  const int64_t ring_bytes = int64_t(g.R) * h->L.ring_slot_elems * 4;
  // With a caller workspace: the ring's backup first, then the staged copies
  // of a frame the step kernel cannot read in place.  Whether a frame is
  // staged depends on its pointer's alignment, which repeats every two
  // frames, and on the plane strides, which every frame shares.
  const int64_t backup = update_state ? 0 : round256(ring_bytes);
  if (sc) {
    int64_t stage = 0;
    for (int64_t t = 0; t < std::min<int64_t>(T, 2); ++t) {
      const StepIO io{static_cast<const char*>(x) + size_t(t * S) * esz, int64_t(T) * S,
                      n_emit > 0 ? y : nullptr, int64_t(y_cap_frames) * So};
      stage = std::max(stage, conv_step_staging_bytes(g, io));
    }
    if (backup + stage > sc->bytes) return CO_ESCRATCH;
  }
  Backup bk;
  if (!update_state) {
    if (sc) {
      if (hipMemcpyAsync(sc->p, h->state + h->L.ring, size_t(ring_bytes),
                         hipMemcpyDeviceToDevice, s) != hipSuccess)
        return CO_EHIP;
    } else {
      const co_status st = backup_range(h->state + h->L.ring, ring_bytes, s, &bk);
      if (st != CO_OK) return st;
    }
  }
  int64_t k = 0;
  co_status st = CO_OK;
  for (int64_t t = 0; t < count; ++t) {
    co_step_plan plan;
    conv_plan(g, h->n, true, &plan);
    const bool pad = t >= T;
    if (any_tap(plan)) {
      StepIO io{pad ? nullptr : static_cast<const char*>(x) + size_t(t * S) * esz,
                int64_t(T) * S,
                plan.emit ? static_cast<char*>(y) + size_t(k * So) * esz : nullptr,
                int64_t(y_cap_frames) * So};
      if (sc) {
        io.ws = sc->p + backup;
        io.ws_bytes = sc->bytes - backup;
      }
      st = hip_status(launch_conv_step(g, h->L, h->state, io, plan, pad, s));
      if (st != CO_OK) break;
    }
    if (plan.emit) ++k;
    ++h->n;
  }
  if (!update_state) {
    co_status r = CO_OK;
    if (sc) {
      if (hipMemcpyAsync(h->state + h->L.ring, sc->p, size_t(ring_bytes),
                         hipMemcpyDeviceToDevice, s) != hipSuccess)
        r = CO_EHIP;
    } else {
      r = restore_range(h->state + h->L.ring, s, &bk);
    }
    if (st == CO_OK) st = r;
    h->n = n0;
  }
  *n_out = int32_t(k);
  return st;
}

}  // namespace

extern "C" {

const char* co_status_str(co_status s) {
  switch (s) {
    case CO_OK: return "CO_OK";
    case CO_EMPTY: return "CO_EMPTY";
    case CO_EINVAL: return "CO_EINVAL: invalid argument";
    case CO_ENOTSUP: return "CO_ENOTSUP: unsupported configuration";
    case CO_ESTATE: return "CO_ESTATE: state buffer too small or made for another descriptor";
    case CO_EHIP: return "CO_EHIP: HIP runtime error";
    case CO_ESCRATCH:
      return "CO_ESCRATCH: the call needs more device scratch than the no-allocation entry "
             "point holds";
    default: return "unknown status";
  }
}

// ---------------------------------------------------------------- convolution

co_status co_conv_query(const co_conv_desc* desc, co_conv_info* info) {
  if (!info) return CO_EINVAL;
  ConvGeom g;
  const co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  const ConvLayout L = conv_layout(g);
  info->receptive_field = g.f;
  info->delay = g.d;
  info->out_size[0] = g.Ho;
  info->out_size[1] = g.Wo;
  info->ring_slots = g.R;
  info->algo = g.algo;
  info->state_bytes = L.total;
  return CO_OK;
}

co_status co_conv_plan_step(const co_conv_desc* desc, int64_t n, int32_t update_state,
                            co_step_plan* plan) {
  if (!plan || n < 0 || n >= kMaxSteps) return CO_EINVAL;
  ConvGeom g;
  const co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  conv_plan(g, n, update_state != 0, plan);
  return CO_OK;
}

co_status co_conv_init_state(const co_conv_desc* desc, const void* weight, const void* bias,
                             void* state, int64_t state_bytes, void* stream,
                             co_conv_handle** out) {
  if (!out || !state || !weight) return CO_EINVAL;
  ConvGeom g;
  co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  if (g.has_bias && !bias) return CO_EINVAL;
  const ConvLayout L = conv_layout(g);
  if (state_bytes < L.total) return CO_ESTATE;
  StateHeader hdr{kConvMagic, kStateVersion, conv_hash(g), L.total, g.algo, g.R};
  co_conv_handle* h = new (std::nothrow) co_conv_handle{g, L, static_cast<char*>(state), 0};
  if (!h) return CO_EINVAL;
  st = hip_status(launch_conv_init(g, L, h->state, weight, bias, hdr, as_stream(stream)));
  if (st != CO_OK) {
    delete h;
    return st;
  }
  return publish(h, HKind::Conv, out);
}

co_status co_conv_init_state_bn(const co_conv_desc* desc, const void* weight, const void* bias,
                                const float* gamma, const float* beta, const float* mean,
                                const float* var, float eps, void* state, int64_t state_bytes,
                                void* stream, co_conv_handle** out) {
  if (!out || !state || !weight || !gamma || !beta || !mean || !var) return CO_EINVAL;
  if (!(eps >= 0.f) || !std::isfinite(eps)) return CO_EINVAL;
  ConvGeom g;
  co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  if (g.has_bias && !bias) return CO_EINVAL;
  const ConvLayout L = conv_layout(g);
  if (state_bytes < L.total) return CO_ESTATE;
  StateHeader hdr{kConvMagic, kStateVersion, conv_hash(g), L.total, g.algo, g.R};
  co_conv_handle* h = new (std::nothrow) co_conv_handle{g, L, static_cast<char*>(state), 0};
  if (!h) return CO_EINVAL;
  st = hip_status(launch_conv_init_bn(g, L, h->state, weight, bias, gamma, beta, mean, var, eps,
                                      hdr, as_stream(stream)));
  if (st != CO_OK) {
    delete h;
    return st;
  }
  return publish(h, HKind::Conv, out);
}

co_status co_conv_fold_bn(const co_conv_desc* desc, const void* weight, const void* bias,
                          const float* gamma, const float* beta, const float* mean,
                          const float* var, float eps, void* w_out, void* b_out, void* stream) {
  if (!weight || !gamma || !beta || !mean || !var || !w_out || !b_out) return CO_EINVAL;
  if (!(eps >= 0.f) || !std::isfinite(eps)) return CO_EINVAL;
  ConvGeom g;
  const co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  if (g.has_bias && !bias) return CO_EINVAL;
  if (int64_t(g.Cg) * g.kT * g.kH * g.kW * g.Cout > kMaxLaunchElems) return CO_EINVAL;
  return hip_status(launch_bn_fold(g, weight, bias, gamma, beta, mean, var, eps, w_out, b_out,
                                   as_stream(stream)));
}

co_status co_conv_forward_step(co_conv_handle* h, const void* x_t, void* y_t,
                               int32_t update_state, void* stream) {
  if (!live(h, HKind::Conv) || !x_t || h->n >= kMaxSteps) return CO_EINVAL;
  co_step_plan plan;
  conv_plan(h->g, h->n, update_state != 0, &plan);
  if (plan.emit && !y_t) return CO_EINVAL;
  if (any_tap(plan)) {
    const StepIO io{x_t, h->g.S(), y_t, h->g.So()};
    const co_status st =
        hip_status(launch_conv_step(h->g, h->L, h->state, io, plan, false, as_stream(stream)));
    if (st != CO_OK) return st;
  }
  if (update_state) ++h->n;
  return plan.emit ? CO_OK : CO_EMPTY;
}

co_status co_conv_forward_steps(co_conv_handle* h, const void* x, int32_t T, void* y,
                                int32_t y_cap_frames, int32_t pad_end, int32_t update_state,
                                void* stream, int32_t* n_out) {
  return conv_forward_steps(h, x, T, y, y_cap_frames, pad_end, update_state, as_stream(stream),
                            n_out, nullptr);
}

co_status co_conv_forward_steps_noalloc(co_conv_handle* h, const void* x, int32_t T, void* y,
                                        int32_t y_cap_frames, int32_t pad_end,
                                        int32_t update_state, void* stream, int32_t* n_out) {
  if (!live(h, HKind::Conv)) return CO_EINVAL;
  void* p = nullptr;
  const co_status st = scratch_address(as_stream(stream), &p);
  if (st != CO_OK) return st;
  const Scratch sc{static_cast<char*>(p), kScratchBytes};
  return conv_forward_steps(h, x, T, y, y_cap_frames, pad_end, update_state, as_stream(stream),
                            n_out, &sc);
}

co_status co_conv_scratch_bytes(int64_t* bytes) {
  if (!bytes) return CO_EINVAL;
  *bytes = kScratchBytes;
  return CO_OK;
}

co_status co_conv_steps_fused(const co_conv_handle* h, int32_t T, int32_t y_cap_frames,
                              int32_t* fused) {
  if (!live(h, HKind::Conv) || !fused || T < 0 || y_cap_frames < 0) return CO_EINVAL;
  const ConvGeom& g = h->g;
  // (the GEMM family also needs 4-byte aligned pixel pairs in x; an
  // allocation from the caching allocator always is)
  static const uint32_t aligned_probe = 0;
  *fused = dw_steps_supported(g, T, y_cap_frames) ||
                   direct_steps_supported(g, T, y_cap_frames) ||
                   gemm_steps_supported(g, T, y_cap_frames, &aligned_probe) ||
                   reg_steps_supported(g, T, y_cap_frames)
               ? 1
               : 0;
  return CO_OK;
}

co_status co_conv_clip_frames(const co_conv_desc* desc, int32_t T, int32_t* t_out) {
  if (!t_out || T < 0) return CO_EINVAL;
  ConvGeom g;
  const co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  *t_out = int32_t(axis_out_len(T, g.kT, g.sT, g.pT, g.dT));
  return CO_OK;
}

co_status co_conv_forward(const co_conv_desc* desc, const void* weight, const void* bias,
                          const void* x, int32_t T, void* y, void* stream) {
  ConvGeom g;
  co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  if (T < 0 || !weight || (g.has_bias && !bias)) return CO_EINVAL;
  const int64_t T_out = axis_out_len(T, g.kT, g.sT, g.pT, g.dT);
  if (T_out == 0) return CO_OK;
  if (!x || !y) return CO_EINVAL;
  if (int64_t(g.B) * g.Cout * T_out * g.So() > (int64_t(1) << 40)) return CO_EINVAL;
  return hip_status(launch_conv_clip(g, T, int32_t(T_out), weight, bias, x, y, as_stream(stream)));
}

co_status co_conv_forward_ws(const co_conv_desc* desc, const void* weight, const void* bias,
                             const co_bn_params* bn, const void* x, int32_t T, void* y,
                             void* workspace, int64_t workspace_bytes, void* stream) {
  ConvGeom g;
  co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  if (T < 0 || !weight || (g.has_bias && !bias)) return CO_EINVAL;
  const int64_t T_out = axis_out_len(T, g.kT, g.sT, g.pT, g.dT);
  if (T_out == 0) return CO_OK;
  if (!x || !y || !workspace || T_out > INT32_MAX) return CO_EINVAL;
  // a clean state in the workspace, then the clip with its end padding: the
  // steps emit exactly the clip's T_out frames, written in place into y
  co_conv_handle* h = nullptr;
  st = bn ? co_conv_init_state_bn(desc, weight, bias, bn->gamma, bn->beta, bn->mean, bn->var,
                                  bn->eps, workspace, workspace_bytes, stream, &h)
          : co_conv_init_state(desc, weight, bias, workspace, workspace_bytes, stream, &h);
  if (st != CO_OK) return st;
  int32_t n = 0;
  st = conv_forward_steps(h, x, T, y, int32_t(T_out), 1, 1, as_stream(stream), &n, nullptr);
  co_conv_destroy(h);
  if (st == CO_OK && n != T_out) return CO_EINVAL;  // (Principle 4: cannot happen)
  return st;
}

co_status co_conv_clean_state(co_conv_handle* h, void* stream) {
  (void)stream;
  if (!live(h, HKind::Conv)) return CO_EINVAL;
  // Every partial sum is started by the first real tap of its output before
  // anything reads it, so a clean state needs no device work.
  h->n = 0;
  return CO_OK;
}

co_status co_conv_get_steps(const co_conv_handle* h, int64_t* n) {
  if (!live(h, HKind::Conv) || !n) return CO_EINVAL;
  *n = h->n;
  return CO_OK;
}

co_status co_conv_out_frames(const co_conv_desc* desc, int64_t n0, int32_t T, int32_t pad_end,
                             int32_t* n_out) {
  if (!n_out || n0 < 0 || T < 0) return CO_EINVAL;
  ConvGeom g;
  const co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  const int64_t count = int64_t(T) + (pad_end ? g.pT : 0);
  if (n0 > kMaxSteps - count) return CO_EINVAL;
  *n_out = int32_t(conv_emissions(g, n0, count));
  return CO_OK;
}

co_status co_conv_attach_state(const co_conv_desc* desc, void* state, int64_t state_bytes,
                               int64_t n, void* stream, co_conv_handle** out) {
  if (!out || !state || n < 0 || n > kMaxSteps) return CO_EINVAL;
  ConvGeom g;
  co_status st = conv_geom(desc, &g);
  if (st != CO_OK) return st;
  const ConvLayout L = conv_layout(g);
  if (state_bytes < L.total) return CO_ESTATE;
  StateHeader hdr;
  st = read_header(state, as_stream(stream), &hdr);
  if (st != CO_OK) return st;
  if (hdr.magic != kConvMagic || hdr.version != kStateVersion || hdr.desc_hash != conv_hash(g) ||
      hdr.bytes != L.total || hdr.algo != g.algo || hdr.slots != g.R)
    return CO_ESTATE;
  co_conv_handle* h = new (std::nothrow) co_conv_handle{g, L, static_cast<char*>(state), n};
  if (!h) return CO_EINVAL;
  return publish(h, HKind::Conv, out);
}

co_status co_conv_destroy(co_conv_handle* h) {
  if (!retire(h, HKind::Conv)) return CO_EINVAL;
  delete h;
  return CO_OK;
}

const char* co_conv_algo_name(const co_conv_handle* h) {
  if (!live(h, HKind::Conv)) return "none";
  switch (h->g.algo) {
    case CO_ALGO_DEPTHWISE: return "depthwise";
    case CO_ALGO_GEMM:
      if (h->g.cfg == kGemmWs) return "gemm_ws_bf16";
      return h->g.dtype == CO_BF16 ? "gemm_bf16" : "gemm_f32";
    case CO_ALGO_GEMM_REG: return h->g.dtype == CO_BF16 ? "gemm_reg_bf16" : "gemm_reg_f32";
    default: return "direct";
  }
}

// -------------------------------------------------------------------- pooling

co_status co_pool_query(const co_pool_desc* desc, co_pool_info* info) {
  if (!info) return CO_EINVAL;
  PoolGeom g;
  const co_status st = pool_geom(desc, &g);
  if (st != CO_OK) return st;
  const PoolLayout L = pool_layout(g);
  info->receptive_field = g.f;
  info->delay = g.d;
  info->out_size[0] = g.Ho;
  info->out_size[1] = g.Wo;
  info->fifo_slots = g.R;
  info->reserved = 0;
  info->state_bytes = L.total;
  return CO_OK;
}

co_status co_pool_plan_step(const co_pool_desc* desc, int64_t n, co_pool_plan* plan) {
  if (!plan || n < 0 || n >= kMaxSteps) return CO_EINVAL;
  PoolGeom g;
  const co_status st = pool_geom(desc, &g);
  if (st != CO_OK) return st;
  pool_plan(g, n, plan);
  return CO_OK;
}

co_status co_pool_init_state(const co_pool_desc* desc, void* state, int64_t state_bytes,
                             void* stream, co_pool_handle** out) {
  if (!out || !state) return CO_EINVAL;
  PoolGeom g;
  co_status st = pool_geom(desc, &g);
  if (st != CO_OK) return st;
  const PoolLayout L = pool_layout(g);
  if (state_bytes < L.total) return CO_ESTATE;
  StateHeader hdr{kPoolMagic, kStateVersion, pool_hash(g), L.total, 0, g.R};
  co_pool_handle* h = new (std::nothrow) co_pool_handle{g, L, static_cast<char*>(state), 0};
  if (!h) return CO_EINVAL;
  st = hip_status(launch_pool_init(g, L, h->state, hdr, as_stream(stream)));
  if (st != CO_OK) {
    delete h;
    return st;
  }
  return publish(h, HKind::Pool, out);
}

co_status co_pool_forward_step(co_pool_handle* h, const void* x_t, void* y_t,
                               int32_t update_state, void* stream) {
  if (!live(h, HKind::Pool) || !x_t || h->n >= kMaxSteps) return CO_EINVAL;
  co_pool_plan plan;
  pool_plan(h->g, h->n, &plan);
  if (plan.emit && !y_t) return CO_EINVAL;
  if (plan.emit || update_state) {
    const StepIO io{x_t, h->g.S(), y_t, h->g.So()};
    const co_status st = hip_status(launch_pool_step(h->g, h->L, h->state, io, plan,
                                                     update_state != 0, false, as_stream(stream)));
    if (st != CO_OK) return st;
  }
  if (update_state) ++h->n;
  return plan.emit ? CO_OK : CO_EMPTY;
}

co_status co_pool_steps_fused(const co_pool_handle* h, int32_t T, int32_t y_cap_frames,
                              int32_t* fused) {
  if (!live(h, HKind::Pool) || !fused || T < 0 || y_cap_frames < 0) return CO_EINVAL;
  *fused = pool_steps_supported(h->g, T, y_cap_frames) ? 1 : 0;
  return CO_OK;
}

co_status co_pool_forward_steps(co_pool_handle* h, const void* x, int32_t T, void* y,
                                int32_t y_cap_frames, int32_t pad_end, int32_t update_state,
                                void* stream, int32_t* n_out) {
  if (!live(h, HKind::Pool) || T < 0 || y_cap_frames < 0 || !n_out) return CO_EINVAL;
  if (T > 0 && !x) return CO_EINVAL;
  const PoolGeom& g = h->g;
  const int64_t count = int64_t(T) + (pad_end ? g.pT : 0);
  if (count > kMaxSteps - h->n) return CO_EINVAL;
  const int64_t n_emit = pool_emissions(g, h->n, count);
  if (n_emit > y_cap_frames) return CO_EINVAL;
  if (n_emit > 0 && !y) return CO_EINVAL;
  hipStream_t s = as_stream(stream);
  const int64_t n0 = h->n;
  if (count > 0 && pool_steps_supported(g, T, y_cap_frames)) {
    // one persistent launch: the FIFO stays in registers across frames; with
    // update_state = 0 the state is simply not written back
    const co_status st = hip_status(launch_pool_steps(
        g, h->L, h->state, x, int64_t(T) * g.S(), T, int32_t(count), y,
        int64_t(y_cap_frames) * g.So(), n0, update_state != 0, s));
    if (st != CO_OK) return st;
    if (update_state) h->n += count;
    *n_out = int32_t(n_emit);
    return CO_OK;
  }
  Backup bk;
  // FIFO and validity flags are contiguous from L.valid to the end
  const int64_t bytes = h->L.total - h->L.valid;
  if (!update_state) {
    const co_status st = backup_range(h->state + h->L.valid, bytes, s, &bk);
    if (st != CO_OK) return st;
  }
  const int64_t S = g.S(), So = g.So();
  const size_t esz = g.dtype == CO_BF16 ? 2 : 4;
  // The pool step addresses a frame with 32-bit buffer offsets over
  // everything reachable from the frame pointer.  A clip whose planes lie
  // 2^31 bytes or more apart is stepped through a contiguous copy of each
  // frame (B*C rows of S elements).
  const bool staged =
      T > 0 && ((int64_t(g.B) * g.C - 1) * T * S + S) * int64_t(esz) >= (int64_t(1) << 31);
  void* frame = nullptr;
  co_status st = CO_OK;
  if (staged && hipMallocAsync(&frame, size_t(g.B) * g.C * S * esz, s) != hipSuccess)
    st = CO_EHIP;
  int64_t k = 0;
  for (int64_t t = 0; t < count && st == CO_OK; ++t) {
    co_pool_plan plan;
    pool_plan(g, h->n, &plan);
    const bool pad = t >= T;
    const char* xt = pad ? nullptr : static_cast<const char*>(x) + size_t(t * S) * esz;
    int64_t x_bc = int64_t(T) * S;
    if (staged && !pad) {
      if (hipMemcpy2DAsync(frame, size_t(S) * esz, xt, size_t(T) * S * esz, size_t(S) * esz,
                           size_t(g.B) * g.C, hipMemcpyDeviceToDevice, s) != hipSuccess) {
        st = CO_EHIP;
        break;
      }
      xt = static_cast<const char*>(frame);
      x_bc = S;
    }
    const StepIO io{xt, x_bc, plan.emit ? static_cast<char*>(y) + size_t(k * So) * esz : nullptr,
                    int64_t(y_cap_frames) * So};
    st = hip_status(launch_pool_step(g, h->L, h->state, io, plan, true, pad, s));
    if (st != CO_OK) break;
    if (plan.emit) ++k;
    ++h->n;
  }
  if (frame && hipFreeAsync(frame, s) != hipSuccess && st == CO_OK) st = CO_EHIP;
  if (!update_state) {
    const co_status r = restore_range(h->state + h->L.valid, s, &bk);
    if (st == CO_OK) st = r;
    h->n = n0;
  }
  *n_out = int32_t(k);
  return st;
}

co_status co_pool_clip_frames(const co_pool_desc* desc, int32_t T, int32_t* t_out) {
  if (!t_out || T < 0) return CO_EINVAL;
  PoolGeom g;
  const co_status st = pool_geom(desc, &g);
  if (st != CO_OK) return st;
  *t_out = int32_t(axis_out_len(T, g.kT, g.sT, g.pT, g.dT));
  return CO_OK;
}

co_status co_pool_forward(const co_pool_desc* desc, const void* x, int32_t T, void* y,
                          void* stream) {
  PoolGeom g;
  co_status st = pool_geom(desc, &g);
  if (st != CO_OK) return st;
  if (T < 0) return CO_EINVAL;
  const int64_t T_out = axis_out_len(T, g.kT, g.sT, g.pT, g.dT);
  if (T_out == 0) return CO_OK;
  if (!x || !y) return CO_EINVAL;
  return hip_status(launch_pool_clip(g, T, int32_t(T_out), x, y, as_stream(stream)));
}

co_status co_pool_clean_state(co_pool_handle* h, void* stream) {
  (void)stream;
  if (!live(h, HKind::Pool)) return CO_EINVAL;
  // The FIFO is only read for frames written since the last clean state.
  h->n = 0;
  return CO_OK;
}

co_status co_pool_get_steps(const co_pool_handle* h, int64_t* n) {
  if (!live(h, HKind::Pool) || !n) return CO_EINVAL;
  *n = h->n;
  return CO_OK;
}

co_status co_pool_out_frames(const co_pool_desc* desc, int64_t n0, int32_t T, int32_t pad_end,
                             int32_t* n_out) {
  if (!n_out || n0 < 0 || T < 0) return CO_EINVAL;
  PoolGeom g;
  const co_status st = pool_geom(desc, &g);
  if (st != CO_OK) return st;
  const int64_t count = int64_t(T) + (pad_end ? g.pT : 0);
  if (n0 > kMaxSteps - count) return CO_EINVAL;
  *n_out = int32_t(pool_emissions(g, n0, count));
  return CO_OK;
}

co_status co_pool_attach_state(const co_pool_desc* desc, void* state, int64_t state_bytes,
                               int64_t n, void* stream, co_pool_handle** out) {
  if (!out || !state || n < 0 || n > kMaxSteps) return CO_EINVAL;
  PoolGeom g;
  co_status st = pool_geom(desc, &g);
  if (st != CO_OK) return st;
  const PoolLayout L = pool_layout(g);
  if (state_bytes < L.total) return CO_ESTATE;
  StateHeader hdr;
  st = read_header(state, as_stream(stream), &hdr);
  if (st != CO_OK) return st;
  if (hdr.magic != kPoolMagic || hdr.version != kStateVersion || hdr.desc_hash != pool_hash(g) ||
      hdr.bytes != L.total || hdr.slots != g.R)
    return CO_ESTATE;
  co_pool_handle* h = new (std::nothrow) co_pool_handle{g, L, static_cast<char*>(state), n};
  if (!h) return CO_EINVAL;
  return publish(h, HKind::Pool, out);
}

co_status co_pool_destroy(co_pool_handle* h) {
  if (!retire(h, HKind::Pool)) return CO_EINVAL;
  delete h;
  return CO_OK;
}


// ------------------------------------------------------------ delay, merges

co_status co_delay_query(const co_delay_desc* desc, int64_t* state_bytes) {
  if (!state_bytes) return CO_EINVAL;
  DelayGeom g;
  const co_status st = delay_geom(desc, &g);
  if (st != CO_OK) return st;
  *state_bytes = g.state_bytes();
  return CO_OK;
}

co_status co_delay_init_state(const co_delay_desc* desc, void* state, int64_t state_bytes,
                              void* stream, co_delay_handle** out) {
  if (!out || !state) return CO_EINVAL;
  DelayGeom g;
  co_status st = delay_geom(desc, &g);
  if (st != CO_OK) return st;
  if (state_bytes < g.state_bytes()) return CO_ESTATE;
  const uint64_t hash = delay_hash(g);
  StateHeader hdr{kDelayMagic, kStateVersion, hash, g.state_bytes(), 0, g.d};
  co_delay_handle* h = new (std::nothrow) co_delay_handle{g, static_cast<char*>(state), 0};
  if (!h) return CO_EINVAL;
  st = hip_status(launch_delay_init(g, h->state, hdr, as_stream(stream)));
  if (st != CO_OK) {
    delete h;
    return st;
  }
  return publish(h, HKind::Delay, out);
}

co_status co_delay_forward_step(co_delay_handle* h, const void* x_t, void* y_t,
                                int32_t update_state, void* stream) {
  if (!live(h, HKind::Delay) || !x_t || h->n >= kMaxSteps) return CO_EINVAL;
  const bool emit = h->n >= h->g.d && y_t;
  if (emit || (update_state && h->g.d > 0)) {
    const co_status st = hip_status(launch_delay_step(h->g, h->state, x_t, nullptr, y_t, h->n,
                                                      emit, update_state != 0,
                                                      as_stream(stream)));
    if (st != CO_OK) return st;
  }
  const bool nonempty = h->n >= h->g.d;
  if (update_state) ++h->n;
  return nonempty ? CO_OK : CO_EMPTY;
}

co_status co_delay_add_step(co_delay_handle* h, const void* x_t, const void* a_t, void* y_t,
                            int32_t update_state, void* stream) {
  if (!live(h, HKind::Delay) || !x_t || h->n >= kMaxSteps) return CO_EINVAL;
  const bool emit = h->n >= h->g.d;
  if (emit && (!a_t || !y_t)) return CO_EINVAL;
  if (emit || (update_state && h->g.d > 0)) {
    const co_status st = hip_status(launch_delay_step(h->g, h->state, x_t, emit ? a_t : nullptr,
                                                      emit ? y_t : nullptr, h->n, emit,
                                                      update_state != 0, as_stream(stream)));
    if (st != CO_OK) return st;
  }
  if (update_state) ++h->n;
  return emit ? CO_OK : CO_EMPTY;
}

co_status co_delay_forward_steps(co_delay_handle* h, const void* x, int32_t T, void* y,
                                 int32_t y_cap_frames, int32_t update_state, void* stream,
                                 int32_t* n_out) {
  if (!live(h, HKind::Delay) || T < 0 || y_cap_frames < 0 || !n_out) return CO_EINVAL;
  if (T > 0 && !x) return CO_EINVAL;
  if (T > kMaxSteps - h->n) return CO_EINVAL;
  const DelayGeom& g = h->g;
  const int64_t first = std::min<int64_t>(T, std::max<int64_t>(0, g.d - h->n));
  const int32_t nout = int32_t(T - first);
  if (nout > y_cap_frames || (nout > 0 && !y)) return CO_EINVAL;
  if (g.frame() * std::max<int64_t>(T, 1) > kMaxLaunchElems) return CO_EINVAL;
  const co_status st = hip_status(launch_delay_steps(g, h->state, x, T, nullptr, y, y_cap_frames,
                                                     h->n, int32_t(first), nout,
                                                     update_state != 0, as_stream(stream)));
  if (st != CO_OK) return st;
  if (update_state) h->n += T;
  *n_out = nout;
  return CO_OK;
}

co_status co_delay_add_steps(co_delay_handle* h, const void* x, int32_t T, const void* a,
                             int32_t a_frames, void* y, int32_t update_state, void* stream) {
  if (!live(h, HKind::Delay) || T < 0 || a_frames < 0 || a_frames > T) return CO_EINVAL;
  if (T > 0 && !x) return CO_EINVAL;
  if (T > kMaxSteps - h->n) return CO_EINVAL;
  if (a_frames > 0 && (!a || !y)) return CO_EINVAL;
  const DelayGeom& g = h->g;
  const int64_t first = int64_t(T) - a_frames;  // step of a's first frame in this call
  if (a_frames > 0 && h->n + first < g.d) return CO_EINVAL;  // residual precedes the stream
  if (g.frame() * std::max<int64_t>(T, 1) > kMaxLaunchElems) return CO_EINVAL;
  const co_status st = hip_status(launch_delay_steps(g, h->state, x, T, a, y, a_frames, h->n,
                                                     int32_t(first), a_frames,
                                                     update_state != 0, as_stream(stream)));
  if (st != CO_OK) return st;
  if (update_state) h->n += T;
  return CO_OK;
}

co_status co_add_frames(const void* a, const void* x, void* y, int32_t rows, int32_t frame_elems,
                        int32_t a_frames, int32_t x_frames, int32_t x_offset, int32_t dtype,
                        void* stream) {
  if (rows < 0 || frame_elems < 1 || a_frames < 0 || x_frames < 0 || x_offset < 0) return CO_EINVAL;
  if (dtype != CO_F32 && dtype != CO_BF16) return CO_EINVAL;
  if (int64_t(x_offset) + a_frames > x_frames) return CO_EINVAL;
  const int64_t total = int64_t(rows) * a_frames * frame_elems;
  if (total == 0) return CO_OK;
  if (!a || !x || !y || total > kMaxLaunchElems) return CO_EINVAL;
  return hip_status(launch_add_frames(a, x, y, rows, frame_elems, a_frames, x_frames, x_offset,
                                      dtype, as_stream(stream)));
}

co_status co_act_forward(const void* x, void* y, int64_t n, int32_t dtype, int32_t act,
                         void* stream) {
  if (n < 0 || (dtype != CO_F32 && dtype != CO_BF16)) return CO_EINVAL;
  if (act != CO_ACT_NONE && act != CO_ACT_RELU) return CO_EINVAL;
  if (n == 0) return CO_OK;
  if (!x || !y || n > kMaxLaunchElems) return CO_EINVAL;
  return hip_status(launch_act(x, y, n, dtype, act, as_stream(stream)));
}

co_status co_delay_clean_state(co_delay_handle* h, void* stream) {
  (void)stream;
  if (!live(h, HKind::Delay)) return CO_EINVAL;
  // every ring slot is written before it is read again
  h->n = 0;
  return CO_OK;
}

co_status co_delay_get_steps(const co_delay_handle* h, int64_t* n) {
  if (!live(h, HKind::Delay) || !n) return CO_EINVAL;
  *n = h->n;
  return CO_OK;
}

co_status co_delay_destroy(co_delay_handle* h) {
  if (!retire(h, HKind::Delay)) return CO_EINVAL;
  delete h;
  return CO_OK;
}

co_status co_chain_delay(int32_t n, const int32_t* f, const int32_t* s, const int32_t* p,
                         int64_t* f_acc, int64_t* p_acc, int64_t* s_acc, int64_t* delay) {
  if (n < 1 || !f || !s || !p || !f_acc || !p_acc || !s_acc || !delay) return CO_EINVAL;
  // Principle 6 in the form its worked example evaluates: layer i's
  // receptive field and padding count in units of the accumulated stride of
  // the layers before it.
  int64_t fa = 0, pa = 0, sa = 1;
  for (int32_t i = 0; i < n; ++i) {
    if (f[i] < 1 || s[i] < 1 || p[i] < 0) return CO_EINVAL;
    if (i == 0) {
      fa = f[0];
      pa = p[0];
      sa = s[0];
    } else {
      fa = fa + int64_t(f[i] - 1) * sa;
      pa = pa + int64_t(p[i]) * sa;
      sa = sa * s[i];
    }
    if (fa > (int64_t(1) << 40) || sa > (int64_t(1) << 40)) return CO_EINVAL;
  }
  *f_acc = fa;
  *p_acc = pa;
  *s_acc = sa;
  *delay = fa - pa - 1;
  return CO_OK;
}

co_status co_residual_align(int64_t f, int64_t s, int64_t p, int64_t module_delay,
                            int64_t* res_delay, int64_t* shrink, int64_t* delay) {
  if (!res_delay || !shrink || !delay) return CO_EINVAL;
  if (f < 1 || s != 1 || p < 0 || 2 * p > f - 1 || module_delay < 0) return CO_EINVAL;
  // the input joins the module's output on the centre of its receptive
  // field: the residual branch waits (f - 1) / 2 frames (rounded down), clip
  // mode drops the frames the module's padding does not restore, and the
  // whole is empty while either branch is (Principle 7)
  const int64_t c = (f - 1) / 2;
  *res_delay = c;
  *shrink = c - p;
  *delay = std::max(module_delay, c);
  return CO_OK;
}


// -------------------------------------------------- fused depthwise + pool

co_status co_convpool_bind(co_conv_handle* conv, co_pool_handle* pool, co_convpool_handle** out) {
  if (!live(conv, HKind::Conv) || !live(pool, HKind::Pool) || !out) return CO_EINVAL;
  if (!convpool_supported(conv->g, pool->g)) return CO_ENOTSUP;
  co_convpool_handle* h = new (std::nothrow) co_convpool_handle{conv, pool};
  if (!h) return CO_EINVAL;
  return publish(h, HKind::ConvPool, out);
}

namespace {

// A fused pair whose two handles are both still live.
static bool live_pair(const co_convpool_handle* h) {
  return live(h, HKind::ConvPool) && live(h->conv, HKind::Conv) && live(h->pool, HKind::Pool);
}

// One fused step at the handles' counters, reading frame planes x_bc
// elements apart; *emitted says whether z was written.
static co_status convpool_step(co_convpool_handle* h, const void* x_t, int64_t x_bc, void* z,
                               int64_t z_bc, bool update, hipStream_t s, bool* emitted) {
  co_conv_handle* c = h->conv;
  co_pool_handle* p = h->pool;
  co_step_plan cplan;
  conv_plan(c->g, c->n, update, &cplan);
  co_pool_plan pplan;
  if (cplan.emit) pool_plan(p->g, p->n, &pplan);
  const bool pemit = cplan.emit && pplan.emit;
  if (pemit && !z) return CO_EINVAL;
  if (any_tap(cplan) || cplan.emit) {
    const co_status st = hip_status(launch_convpool_step(c->g, c->L, c->state, p->g, p->L,
                                                         p->state, x_t, x_bc, z, z_bc, cplan,
                                                         cplan.emit ? &pplan : nullptr, update, s));
    if (st != CO_OK) return st;
  }
  if (update) {
    ++c->n;
    if (cplan.emit) ++p->n;
  }
  *emitted = pemit;
  return CO_OK;
}

}  // namespace

co_status co_convpool_forward_step(co_convpool_handle* h, const void* x_t, void* z_t,
                                   int32_t update_state, void* stream) {
  if (!live_pair(h) || !x_t || h->conv->n >= kMaxSteps) return CO_EINVAL;
  bool emitted = false;
  const co_status st = convpool_step(h, x_t, h->conv->g.S(), z_t, 1, update_state != 0,
                                     as_stream(stream), &emitted);
  if (st != CO_OK) return st;
  return emitted ? CO_OK : CO_EMPTY;
}

co_status co_convpool_forward_steps(co_convpool_handle* h, const void* x, int32_t T, void* z,
                                    int32_t z_cap_frames, int32_t update_state, void* stream,
                                    int32_t* n_out) {
  if (!live_pair(h) || T < 0 || z_cap_frames < 0 || !n_out) return CO_EINVAL;
  if (T > 0 && !x) return CO_EINVAL;
  co_conv_handle* c = h->conv;
  co_pool_handle* p = h->pool;
  if (T > kMaxSteps - c->n) return CO_EINVAL;
  // the pool steps once per emitted convolution frame
  const int64_t conv_out = conv_emissions(c->g, c->n, T);
  const int64_t n_emit = pool_emissions(p->g, p->n, conv_out);
  if (n_emit > z_cap_frames || (n_emit > 0 && !z)) return CO_EINVAL;
  const int64_t x_bc = int64_t(T) * c->g.S();
  const size_t esz = c->g.dtype == CO_BF16 ? 2 : 4;
  if ((int64_t(c->g.B) * c->g.Cin * x_bc) * int64_t(esz) >= (int64_t(1) << 31)) return CO_EINVAL;
  hipStream_t s = as_stream(stream);
  const int64_t n0c = c->n, n0p = p->n;
  if (T > 0 && convpool_steps_supported(c->g, p->g, T)) {
    // one persistent launch; with update_state = 0 it writes no state
    const co_status st = hip_status(launch_convpool_steps(c->g, c->L, c->state, p->g, p->L,
                                                          p->state, x, T, z, z_cap_frames, n0c,
                                                          n0p, update_state != 0, s));
    if (st != CO_OK) return st;
    if (update_state) {
      c->n += T;
      p->n += conv_out;
    }
    *n_out = int32_t(n_emit);
    return CO_OK;
  }
  Backup bk_ring, bk_fifo;
  if (!update_state) {
    co_status st = backup_range(c->state + c->L.ring, int64_t(c->g.R) * c->L.ring_slot_elems * 4,
                                s, &bk_ring);
    if (st == CO_OK)
      st = backup_range(p->state + p->L.valid, p->L.total - p->L.valid, s, &bk_fifo);
    if (st != CO_OK) return st;
  }
  co_status st = CO_OK;
  int64_t k = 0;
  for (int32_t t = 0; t < T && st == CO_OK; ++t) {
    bool emitted = false;
    st = convpool_step(h, static_cast<const char*>(x) + size_t(t) * c->g.S() * esz, x_bc,
                       static_cast<char*>(z) + size_t(k) * esz, z_cap_frames, true, s, &emitted);
    if (emitted) ++k;
  }
  if (!update_state) {
    const co_status r1 = restore_range(c->state + c->L.ring, s, &bk_ring);
    const co_status r2 = restore_range(p->state + p->L.valid, s, &bk_fifo);
    if (st == CO_OK) st = r1 != CO_OK ? r1 : r2;
    c->n = n0c;
    p->n = n0p;
  }
  *n_out = int32_t(k);
  return st;
}

// ------------------------------------------------------- fused bottleneck

co_status co_bneck_bind(co_conv_handle* pw, int32_t act1, co_conv_handle* dw, int32_t act2,
                        co_pool_handle* pool, co_bneck_handle** out) {
  if (!live(pw, HKind::Conv) || !live(dw, HKind::Conv) || !live(pool, HKind::Pool) || !out)
    return CO_EINVAL;
  for (const int32_t a : {act1, act2})
    if (a != CO_ACT_NONE && a != CO_ACT_RELU) return CO_EINVAL;
  if (!bneck_supported(pw->g, dw->g, pool->g)) return CO_ENOTSUP;
  co_bneck_handle* h = new (std::nothrow) co_bneck_handle{pw, act1, dw, act2, pool};
  if (!h) return CO_EINVAL;
  return publish(h, HKind::Bneck, out);
}

namespace {

static bool live_bneck(const co_bneck_handle* h) {
  return live(h, HKind::Bneck) && live(h->pw, HKind::Conv) && live(h->dw, HKind::Conv) &&
         live(h->pool, HKind::Pool);
}

// One fused bottleneck step at the handles' counters, reading input planes
// x_bc elements apart; *emitted says whether z was written.
static co_status bneck_step(co_bneck_handle* h, const void* x_t, int64_t x_bc, void* z,
                            int64_t z_bc, bool update, hipStream_t s, bool* emitted) {
  co_conv_handle* pw = h->pw;
  co_conv_handle* c = h->dw;
  co_pool_handle* p = h->pool;
  co_step_plan cplan;
  conv_plan(c->g, c->n, update, &cplan);
  co_pool_plan pplan;
  if (cplan.emit) pool_plan(p->g, p->n, &pplan);
  const bool pemit = cplan.emit && pplan.emit;
  if (pemit && !z) return CO_EINVAL;
  if (any_tap(cplan) || cplan.emit) {
    const co_status st = hip_status(launch_bneck_step(
        pw->g, pw->L, pw->state, h->act1, c->g, c->L, c->state, h->act2, p->g, p->L, p->state,
        x_t, x_bc, z, z_bc, cplan, cplan.emit ? &pplan : nullptr, update, s));
    if (st != CO_OK) return st;
  }
  if (update) {
    ++pw->n;  // the pointwise convolution emits every frame (delay 0)
    ++c->n;
    if (cplan.emit) ++p->n;
  }
  *emitted = pemit;
  return CO_OK;
}

}  // namespace

co_status co_bneck_forward_step(co_bneck_handle* h, const void* x_t, void* z_t,
                                int32_t update_state, void* stream) {
  if (!live_bneck(h) || !x_t) return CO_EINVAL;
  if (h->pw->n >= kMaxSteps || h->dw->n >= kMaxSteps) return CO_EINVAL;
  bool emitted = false;
  const co_status st = bneck_step(h, x_t, h->pw->g.S(), z_t, 1, update_state != 0,
                                  as_stream(stream), &emitted);
  if (st != CO_OK) return st;
  return emitted ? CO_OK : CO_EMPTY;
}

co_status co_bneck_forward_steps(co_bneck_handle* h, const void* x, int32_t T, void* z,
                                 int32_t z_cap_frames, int32_t update_state, void* stream,
                                 int32_t* n_out) {
  if (!live_bneck(h) || T < 0 || z_cap_frames < 0 || !n_out) return CO_EINVAL;
  if (T > 0 && !x) return CO_EINVAL;
  co_conv_handle* pw = h->pw;
  co_conv_handle* c = h->dw;
  co_pool_handle* p = h->pool;
  if (T > kMaxSteps - pw->n || T > kMaxSteps - c->n) return CO_EINVAL;
  const int64_t S = pw->g.S();
  const int64_t esz = pw->g.dtype == CO_BF16 ? 2 : 4;
  // frames are read in place from the clip with 32-bit buffer offsets
  if (int64_t(pw->g.B) * pw->g.Cin * int64_t(T) * S * esz >= (int64_t(1) << 31)) return CO_EINVAL;
  // the pool steps once per emitted depthwise frame
  const int64_t conv_out = conv_emissions(c->g, c->n, T);
  const int64_t n_emit = pool_emissions(p->g, p->n, conv_out);
  if (n_emit > z_cap_frames || (n_emit > 0 && !z)) return CO_EINVAL;
  hipStream_t s = as_stream(stream);
  const int64_t n0w = pw->n, n0c = c->n, n0p = p->n;
  Backup bk_ring, bk_fifo;
  if (!update_state) {
    co_status st = backup_range(c->state + c->L.ring, int64_t(c->g.R) * c->L.ring_slot_elems * 4,
                                s, &bk_ring);
    if (st == CO_OK)
      st = backup_range(p->state + p->L.valid, p->L.total - p->L.valid, s, &bk_fifo);
    if (st != CO_OK) return st;
  }
  co_status st = CO_OK;
  int64_t k = 0;
  for (int32_t t = 0; t < T && st == CO_OK; ++t) {
    bool emitted = false;
    st = bneck_step(h, static_cast<const char*>(x) + size_t(t) * S * esz, int64_t(T) * S,
                    static_cast<char*>(z) + size_t(k) * esz, z_cap_frames, true, s, &emitted);
    if (emitted) ++k;
  }
  if (!update_state) {
    const co_status r1 = restore_range(c->state + c->L.ring, s, &bk_ring);
    const co_status r2 = restore_range(p->state + p->L.valid, s, &bk_fifo);
    if (st == CO_OK) st = r1 != CO_OK ? r1 : r2;
    pw->n = n0w;
    c->n = n0c;
    p->n = n0p;
  }
  *n_out = int32_t(k);
  return st;
}

co_status co_bneck_destroy(co_bneck_handle* h) {
  if (!retire(h, HKind::Bneck)) return CO_EINVAL;
  delete h;
  return CO_OK;
}

co_status co_convpool_destroy(co_convpool_handle* h) {
  if (!retire(h, HKind::ConvPool)) return CO_EINVAL;
  delete h;
  return CO_OK;
}

}  // extern "C"
