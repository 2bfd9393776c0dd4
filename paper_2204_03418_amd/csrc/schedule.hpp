// Host-side scheduler of the continual convolution / pooling steps.
//
// Pure C++ (no HIP): descriptor validation, receptive field and delay
// (Principle 4), the per-step tap schedule (Principles 3-5) and the layout of
// the caller-owned state buffer.  The device code consumes what this file
// decides; nothing here touches the GPU.
#pragma once

#include <cstdint>

#include "../../include/coinf.h"

namespace coinf {

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t m) { return ceil_div(a, m) * m; }

// floor((L + 2p - d(k-1) - 1)/s) + 1, or 0 when no window fits.
inline int64_t axis_out_len(int64_t L, int64_t k, int64_t s, int64_t p, int64_t d) {
  const int64_t span = L + 2 * p - d * (k - 1) - 1;
  return span < 0 ? 0 : span / s + 1;
}

// Everything a convolution kernel needs to know about the layer, resolved
// once from the descriptor.  Spatial axes are always two (unused ones are 1).
// Division by a divisor known on the host: for 0 <= n < 2^31 and
// 1 <= d < 2^31, n / d == (n * m) >> s with l = ceil(log2 d), s = 31 + l and
// m = ceil(2^s / d) (< 2^32).  The product's error n*(m - 2^s/d)/2^s is below
// 2^-l <= 1/d, which cannot carry past the next multiple of d.  Kernels take
// index decompositions this way instead of emulating integer division.
struct FastDiv {
  uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((uint64_t(1) << l) < d) ++l;
  const uint64_t m = ((uint64_t(1) << (31 + l)) + d - 1) / d;
  return FastDiv{d, uint32_t(m), 31 + l};
}

struct ConvGeom {
  int32_t spatial_dims;
  int32_t B, Cin, Cout, G, Cg, Og;
  int32_t H, W, Ho, Wo;
  int32_t kT, kH, kW;
  int32_t sT, sH, sW;
  int32_t pT, pH, pW;
  int32_t dT, dH, dW;
  int32_t f, d, R;          // receptive field, delay, ring slots
  int32_t has_bias, dtype, algo;
  int32_t cfg;              // GEMM / register-GEMM instantiation (-1: none)
  int64_t S() const { return int64_t(H) * W; }
  int64_t So() const { return int64_t(Ho) * Wo; }
  int64_t out_frame_elems() const { return int64_t(B) * Cout * So(); }
};

// Tile configuration of the implicit-GEMM step kernel.  The GEMM is
// C[M = B*Ho*Wo output pixels][N = kT*C_out (tap, channel)] over
// K = kH*kW*C_in (spatial tap, channel; channels innermost).  Each wave owns
// WM x WN fragments of 16x16; a workgroup has NWM x NWN waves.
struct GemmConfig {
  int32_t id;          // kernel instantiation
  int32_t dtype;       // CO_F32 | CO_BF16
  int32_t WM, WN;      // fragments per wave along M and N
  int32_t NWM, NWN;    // waves per workgroup along M and N
  int32_t KL;          // elements per lane per 16-byte operand read
  int32_t CK;          // input channels per LDS chunk (= 4 * KL)
  int32_t M_WG, N_WG;  // workgroup tile
  int32_t m_tiles, n_tiles, n_chunks;
  int32_t cols;        // staged row pitch in pixels (W + pW: shared halo)
  int32_t max_slots;   // staged input rows per tile (one zero row follows)
  int64_t a_units;     // 16-byte units of one A stage in LDS
  int64_t b_units;     // 16-byte units of one B stage in LDS
  int64_t lds_bytes;   // 2 * (a_units + b_units) * 16
  int32_t ws;          // warp-specialized kernel (conv_gemm_ws.hip): producer waves
                       // stage A, consumer waves stream B from L2 (b_units = 0)
  int32_t real_rows;   // ws: most input rows a tile stages (the rest are zero halo rows)
};

// Register-operand implicit GEMM (small K): one wave per 16-pixel x
// 16*WN-column tile holds every k-step's operands in registers.  A k-step is
// one spatial tap (u, v) and one block of CKS input channels: 4 for fp32
// (v_mfma_f32_16x16x4_f32, one channel per lane) and 32 for bf16
// (v_mfma_f32_16x16x32_bf16, eight channels per lane).
struct RegConfig {
  int32_t id;       // kernel instantiation
  int32_t dtype;    // CO_F32 | CO_BF16
  int32_t WN;       // 16-column fragments per wave
  int32_t TAPS;     // spatial taps (kH*kW) the instantiation holds (all waves of a tile)
  int32_t KSPLIT;   // waves sharing one tile (each takes TAPS / KSPLIT taps)
  int32_t CSMAX;    // channel blocks per tap the instantiation holds
  int32_t CKS;      // input channels per k-step (channel block)
  int32_t CS;       // channel blocks per spatial tap, ceil(C_in / CKS)
  int32_t CSU;      // 16-byte weight units per lane, fragment and tap
  int32_t KS;       // k-steps: kH * kW * CS
  int32_t U;        // 16-byte weight units per lane and fragment: kH * kW * CSU
  int32_t m_frags;  // 16-pixel fragments, ceil(B*Ho*Wo / 16)
  int32_t n_frags;  // 16-column fragments, ceil(kT*C_out / 16)
};

constexpr int kRegConfigs = 10;

constexpr int kGemmConfigs = 5;
constexpr int kGemmWs = 4;             // the warp-specialized bf16 3x3 configuration
constexpr int kWsWM = 7;               // consumer wave: 7 pixel fragments ...
constexpr int kWsWN = 4;               // ... x 4 column fragments of 16x16
constexpr int kWsWaves = 4;            // consumer waves (and as many producer waves)
// Multiply-accumulates per step above which AUTO takes the LDS-staged GEMM
// family over the register GEMM.
constexpr double kRegMaxAutoMacs = 3.0e8;
constexpr int kGemmPixUnits = 5;  // 16-byte units per staged pixel (4 + 1 pad)
constexpr int kGemmStageItems = 1024;  // staging items per workgroup and chunk
constexpr int64_t kLdsBytes = 160 * 1024;
// Largest step counter a handle accepts: the schedule's virtual time n + pT
// and the end n + count of a forward_steps call stay far from overflow.
constexpr int64_t kMaxSteps = int64_t(1) << 62;

// Persistent forward_steps of the LDS-tiled GEMM (bf16, temporal stride and
// dilation 1, kT <= kStepsKT): a workgroup of kStepsNWM x kStepsNWN waves
// owns M_WG = 16 * kStepsWM * kStepsNWM output pixels x O_WG = 16 * kStepsNWN
// output channels for every temporal tap (N_WG = kStepsKT * O_WG columns),
// so the partial sums its outputs continue stay in its registers across
// frames.  Per frame it stages the input in chunks of 32 channels (double
// buffered) and streams the weights in stages of one chunk x one kernel row
// (triple buffered).
struct GemmStepsConfig {
  int32_t M_WG, O_WG, N_WG;
  int32_t m_tiles, o_tiles, n_chunks;
  int32_t cols, max_slots;
  int64_t a_units;       // 16-byte units of one input stage
  int64_t b_units;       // 16-byte units of one weight stage (kW x N_WG x 4)
  int64_t lds_bytes;     // (2 * a_units + 3 * b_units) * 16
  int64_t weight_bytes;  // packed weights: o_tiles x n_chunks x kH stages
};
constexpr int kStepsWM = 5, kStepsNWM = 2, kStepsNWN = 4, kStepsKT = 3;
constexpr int kStepsStageItems = 512;  // input staging items per workgroup and chunk

// Layout of a convolution state buffer (byte offsets).
struct ConvLayout {
  int64_t header, bias, weight, ring;
  int64_t weight_bytes;
  int64_t steps_weight, steps_weight_bytes;  // second packing for persistent forward_steps (0: none)
  int64_t ring_slot_elems;  // floats between consecutive ring slots
  int64_t total;
};

struct PoolGeom {
  int32_t kind, spatial_dims;
  int32_t B, C;
  int32_t H, W, Ho, Wo;
  int32_t kT, kH, kW;
  int32_t sT, sH, sW;
  int32_t pT, pH, pW;
  int32_t dT, dH, dW;
  int32_t f, d, R;          // receptive field, delay, FIFO slots
  int32_t count_include_pad, dtype;
  int64_t S() const { return int64_t(H) * W; }
  int64_t So() const { return int64_t(Ho) * Wo; }
  int64_t out_frame_elems() const { return int64_t(B) * C * So(); }
};

struct PoolLayout {
  int64_t header, valid, fifo;
  int64_t fifo_slot_elems;
  int64_t total;
};

constexpr int64_t kHeaderBytes = 256;
constexpr int64_t kAlign = 256;
constexpr uint32_t kConvMagic = 0x564E4F43u;  // "CONV"
constexpr uint32_t kPoolMagic = 0x4C4F4F50u;  // "POOL"
constexpr uint32_t kStateVersion = 1;

constexpr uint32_t kDelayMagic = 0x594C4544u;  // "DELY"

// Delay geometry: frames of B x C x E elements, a ring of d input frames
// laid out (slot, B, C, E) in the io dtype after the header.
struct DelayGeom {
  int32_t B, C, E, d, dtype;
  int64_t frame() const { return int64_t(B) * C * E; }
  int64_t esz() const { return dtype == CO_BF16 ? 2 : 4; }
  int64_t ring_offset() const { return kHeaderBytes; }
  int64_t state_bytes() const { return kHeaderBytes + int64_t(d) * frame() * esz(); }
};
co_status delay_geom(const co_delay_desc* desc, DelayGeom* g);
uint64_t delay_hash(const DelayGeom& g);

// State header, written at init and checked on attach.
struct StateHeader {
  uint32_t magic;
  uint32_t version;
  uint64_t desc_hash;
  int64_t bytes;
  int32_t algo;
  int32_t slots;
};

// Floats in one ring slot: the output frame, padded.
int64_t ring_slot_elems(const ConvGeom& g);
// Whether one input frame, one output frame (in the io dtype) and the whole
// fp32 ring each stay below 2^31 bytes: the GEMM-family kernels address them
// through 32-bit buffer offsets.
bool frame_offsets_fit(const ConvGeom& g);

// Validate a convolution descriptor, resolve the algorithm and fill g.
co_status conv_geom(const co_conv_desc* desc, ConvGeom* g);
ConvLayout conv_layout(const ConvGeom& g);
// Hash of the validated descriptor and resolved algorithm (FNV-1a).
uint64_t conv_hash(const ConvGeom& g);
// Tap plan of step n (see co_conv_plan_step).
void conv_plan(const ConvGeom& g, int64_t n, bool update_state, co_step_plan* plan);

// Step plans of a forward_steps call for the plan-driven persistent kernels
// (temporal stride or dilation above 1), packed per frame as 6 bits a tap:
// the CO_TAP_ action (3 bits) and the ring slot (3 bits).  Explicit for the
// call's frames within a stream's first (kT - 1) dT steps, where start
// padding and missing outputs matter; after those the plan of step n + sT R
// equals that of step n (slots cycle with the output index mod R), so one
// period covers the rest of the call.
constexpr int kPlanStart = 32;   // explicit plans
constexpr int kPlanPeriod = 64;  // periodic plans: sT R steps
constexpr int kPlanMaxR = 8;     // ring slots a 3-bit field addresses
struct PlanTable {
  int32_t n_start;  // frames of the call that take explicit plans
  int32_t period;   // sT * R
  uint64_t code_start[kPlanStart];
  uint64_t code_period[kPlanPeriod];
};
// Whether a layer's plans fit a PlanTable (kT <= 10 taps of 6 bits, R <= 8,
// a period of at most kPlanPeriod steps).
bool plan_table_fits(const ConvGeom& g);
void plan_table(const ConvGeom& g, int64_t n0, int64_t count, PlanTable* t);
// Number of non-empty outputs of steps n .. n + count - 1.
int64_t conv_emissions(const ConvGeom& g, int64_t n, int64_t count);

co_status pool_geom(const co_pool_desc* desc, PoolGeom* g);
PoolLayout pool_layout(const PoolGeom& g);
uint64_t pool_hash(const PoolGeom& g);
void pool_plan(const PoolGeom& g, int64_t n, co_pool_plan* plan);
int64_t pool_emissions(const PoolGeom& g, int64_t n, int64_t count);

// Fill the derived sizes of tile configuration `id` for a geometry; false
// when it does not apply (dtype, LDS) .
bool gemm_config(const ConvGeom& g, int id, GemmConfig* c);
// The configuration the library picks for a geometry (-1: none fits).
int gemm_pick(const ConvGeom& g);

// Register-operand GEMM: derived sizes of instantiation `id` (false when it
// does not apply) and the one the library picks (-1: none holds K).
bool reg_config(const ConvGeom& g, int id, RegConfig* c);
int reg_pick(const ConvGeom& g);
bool reg_supported(const ConvGeom& g);

// Whether the implicit-GEMM / depthwise kernels accept a geometry.
bool gemm_supported(const ConvGeom& g);
bool gemm_geometry_ok(const ConvGeom& g);
bool gemm_steps_config(const ConvGeom& g, GemmStepsConfig* c);
bool depthwise_supported(const ConvGeom& g);

// Bytes of packed weights for an algorithm.
int64_t packed_weight_bytes(const ConvGeom& g);

}  // namespace coinf
