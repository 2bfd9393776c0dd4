// Kernel launchers of libcoinf (host side of the HIP kernels).
#pragma once

#include <hip/hip_runtime.h>

#include "schedule.hpp"

namespace coinf {

// Where one step reads its frame and writes its output.  x_bc / y_bc are the
// element strides between consecutive (batch, channel) planes: S for a single
// frame (B, C, S1, S2), T*S when the frame is read in place from a clip
// (B, C, T, S1, S2).
// ws / ws_bytes: caller-provided device scratch for a step that has to stage
// its frame (see launch_conv_step_staged); null lets the step allocate.
struct StepIO {
  const void* x;
  int64_t x_bc;
  void* y;
  int64_t y_bc;
  void* ws = nullptr;
  int64_t ws_bytes = 0;
};

// One convolution step with the handle's algorithm.  zero_frame runs an
// end-padding frame, which contributes exactly zero (no contraction).
hipError_t launch_conv_step(const ConvGeom& g, const ConvLayout& L, char* state,
                            const StepIO& io, const co_step_plan& plan, bool zero_frame,
                            hipStream_t stream);

// Pack bias and weights into the state and write its header.
hipError_t launch_conv_init(const ConvGeom& g, const ConvLayout& L, char* state,
                            const void* weight, const void* bias, const StateHeader& hdr,
                            hipStream_t stream);
// The same with an evaluation-mode batch normalisation folded in: per output
// channel o, scale = gamma / sqrt(var + eps) multiplies the weights and the
// bias becomes bias * scale + beta - mean * scale (gamma, beta, mean, var:
// float32, C_out each).
hipError_t launch_conv_init_bn(const ConvGeom& g, const ConvLayout& L, char* state,
                               const void* weight, const void* bias, const float* gamma,
                               const float* beta, const float* mean, const float* var, float eps,
                               const StateHeader& hdr, hipStream_t stream);
// Folded weights (C_out, C_in/G, kT, kH, kW) and bias (C_out) in the io dtype.
hipError_t launch_bn_fold(const ConvGeom& g, const void* weight, const void* bias,
                          const float* gamma, const float* beta, const float* mean,
                          const float* var, float eps, void* w_out, void* b_out, hipStream_t s);

// Clip-mode regular convolution (symmetric temporal padding).
hipError_t launch_conv_clip(const ConvGeom& g, int32_t T, int32_t T_out, const void* weight,
                            const void* bias, const void* x, void* y, hipStream_t stream);

hipError_t launch_pool_step(const PoolGeom& g, const PoolLayout& L, char* state,
                            const StepIO& io, const co_pool_plan& plan, bool update_state,
                            bool pad_frame, hipStream_t stream);

hipError_t launch_pool_init(const PoolGeom& g, const PoolLayout& L, char* state,
                            const StateHeader& hdr, hipStream_t stream);

// Persistent forward_steps of a pool (same conventions as the depthwise one):
// temporal stride 1 and dilation 1, kT <= 5, a spatial window of at most 64,
// clips below 2^31 bytes.
bool pool_steps_supported(const PoolGeom& g, int64_t x_frames, int64_t y_frames);
// Validity flags of the FIFO slots that pool steps n0 .. n0 + count - 1 wrote
// (the first T real frames, the rest end padding).
hipError_t launch_pool_valid(float* valid, int32_t R, int64_t n0, int32_t count, int32_t T,
                             hipStream_t stream);
hipError_t launch_pool_steps(const PoolGeom& g, const PoolLayout& L, char* state, const void* x,
                             int64_t x_bc, int32_t nreal, int32_t count, void* y, int64_t y_bc,
                             int64_t n0, bool update, hipStream_t stream);

hipError_t launch_pool_clip(const PoolGeom& g, int32_t T, int32_t T_out, const void* x, void* y,
                            hipStream_t stream);

// Per-algorithm step launchers (defined next to their kernels).
hipError_t launch_conv_step_direct(const ConvGeom& g, const ConvLayout& L, char* state,
                                   const StepIO& io, const co_step_plan& plan, bool zero_frame,
                                   hipStream_t stream);
// One step of a GEMM-family layer whose frame the kernel cannot address in
// place (an input plane stride or an output stride that takes the reach past
// 2^31 bytes, or a misaligned input): the frame is copied into a contiguous
// stream-ordered buffer, stepped, and an output staged the same way is
// copied back.  Fails when the frame is already contiguous and aligned.
// With io.ws set the copies live there (io.ws_bytes must cover
// conv_step_staging_bytes) and nothing is allocated.
hipError_t launch_conv_step_staged(const ConvGeom& g, const ConvLayout& L, char* state,
                                   const StepIO& io, const co_step_plan& plan, hipStream_t stream);
// Device bytes a step with this frame and output (io.x, io.x_bc, io.y,
// io.y_bc) needs for staging: 0 when the handle's kernel reads the frame in
// place.  Each staged buffer is rounded up to 256 bytes.
int64_t conv_step_staging_bytes(const ConvGeom& g, const StepIO& io);
// Whether the GEMM-family step kernels read this frame in place (false) or
// have it staged (true).
bool gemm_step_needs_staging(const ConvGeom& g, const StepIO& io);
bool reg_step_needs_staging(const ConvGeom& g, const StepIO& io);
// Persistent forward_steps of small direct layers (same conventions as the
// depthwise one): temporal stride 1 and dilation 1, kT <= 4 and
// C_in/G * kH * kW <= 16.
bool direct_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames);
hipError_t launch_conv_steps_direct(const ConvGeom& g, const ConvLayout& L, char* state,
                                    const void* x, int64_t x_bc, int32_t T, int32_t count,
                                    void* y, int64_t y_bc, int64_t n0, bool update,
                                    hipStream_t stream);
hipError_t launch_conv_step_depthwise(const ConvGeom& g, const ConvLayout& L, char* state,
                                      const StepIO& io, const co_step_plan& plan,
                                      hipStream_t stream);

// Persistent forward_steps of the depthwise step: `count` frames (the first T
// read from the clip x with plane stride x_bc, the rest end-padding zero
// frames) in one launch, starting at step counter n0; emitted frames go to
// y in order.  Temporal stride 1 and dilation 1, kT <= 5, 3x3 or 1x1 stencils.
bool dw_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames);
hipError_t launch_conv_steps_depthwise(const ConvGeom& g, const ConvLayout& L, char* state,
                                       const void* x, int64_t x_bc, int32_t T, int32_t count,
                                       void* y, int64_t y_bc, int64_t n0, bool update,
                                       hipStream_t stream);
hipError_t launch_conv_step_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                                 const StepIO& io, const co_step_plan& plan, hipStream_t stream);
hipError_t launch_conv_step_reg(const ConvGeom& g, const ConvLayout& L, char* state,
                                const StepIO& io, const co_step_plan& plan, hipStream_t stream);
// Persistent forward_steps of the register-GEMM step (same conventions as
// the depthwise one): temporal stride 1 and dilation 1, kT within what the
// step kernel's instantiation can hold in registers.
bool reg_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames);
hipError_t launch_conv_steps_reg(const ConvGeom& g, const ConvLayout& L, char* state,
                                 const void* x, int64_t x_bc, int32_t T, int32_t count, void* y,
                                 int64_t y_bc, int64_t n0, bool update, hipStream_t stream);
hipError_t launch_pack_reg(const ConvGeom& g, const ConvLayout& L, char* state,
                           const void* weight, const float* wscale, hipStream_t stream);
// Persistent forward_steps of the LDS-tiled GEMM (bf16; same conventions as
// the depthwise one): temporal stride 1 and dilation 1, kT <= 3, 3x3 or 1x1
// taps, tiles within the LDS and staging budgets.  x is the clip pointer
// (pixel pairs must be 4-byte aligned when rows are even).
bool gemm_steps_supported(const ConvGeom& g, int64_t x_frames, int64_t y_frames, const void* x);
hipError_t launch_conv_steps_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                                  const void* x, int64_t x_bc, int32_t T, int32_t count, void* y,
                                  int64_t y_bc, int64_t n0, bool update, hipStream_t stream);
hipError_t launch_pack_gemm_steps(const ConvGeom& g, const ConvLayout& L, char* state,
                                  const void* weight, const float* wscale, hipStream_t stream);
// Weight packing: wscale (float32, C_out) multiplies each output channel's
// weights before they are rounded to the packed dtype (batch normalisation
// folded at init); null leaves them as given.
hipError_t launch_pack_gemm(const ConvGeom& g, const ConvLayout& L, char* state,
                            const void* weight, const float* wscale, hipStream_t stream);
// The warp-specialized configuration of the GEMM step (conv_gemm_ws.hip):
// bf16, 3x3 taps; its weights packed in the order its consumer waves load.
hipError_t launch_conv_step_gemm_ws(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L,
                                    char* state, const StepIO& io, const co_step_plan& plan,
                                    hipStream_t stream);
hipError_t launch_pack_gemm_ws(const ConvGeom& g, const GemmConfig& c, const ConvLayout& L,
                               char* state, const void* weight, const float* wscale,
                               hipStream_t stream);

// Fused depthwise convolution step + global spatial pool step (convpool.hip):
// one launch per step; pplan is null when the convolution does not emit
// (the pool does not step); x_bc is the element stride between frame planes.
// The pair must satisfy convpool_supported, and the planes reachable from x
// must span fewer than 2^31 bytes.
bool convpool_supported(const ConvGeom& g, const PoolGeom& pg);
hipError_t launch_convpool_step(const ConvGeom& g, const ConvLayout& L, char* cstate,
                                const PoolGeom& pg, const PoolLayout& PL, char* pstate,
                                const void* x, int64_t x_bc, void* z, int64_t z_bc,
                                const co_step_plan& cplan, const co_pool_plan* pplan, bool update,
                                hipStream_t stream);
// The same pair over a clip x (B, C, T, H, W) in one launch, from the
// handles' step counters n0c (convolution) and n0p (pool): the pooled
// outputs go to z (B, C, z_cap, 1, 1) from frame 0; with update the ring, the
// FIFO and the FIFO's validity flags advance (the host advances the counters).
bool convpool_steps_supported(const ConvGeom& g, const PoolGeom& pg, int64_t T);
hipError_t launch_convpool_steps(const ConvGeom& g, const ConvLayout& L, char* cstate,
                                 const PoolGeom& pg, const PoolLayout& PL, char* pstate,
                                 const void* x, int32_t T, void* z, int64_t z_cap, int64_t n0c,
                                 int64_t n0p, bool update, hipStream_t stream);

// Fused X3D-style bottleneck step (convpool.hip): a pointwise (1x1x1,
// direct-packed, delay 0) convolution with activation act1, a depthwise
// convolution with activation act2 and the pool over its plane, in one
// launch; the three handles' plans as for the separate steps (the pointwise
// one always emits).  Input planes x_bc elements apart.
bool bneck_supported(const ConvGeom& pw, const ConvGeom& g, const PoolGeom& pg);
hipError_t launch_bneck_step(const ConvGeom& pw, const ConvLayout& PWL, char* pwstate,
                             int32_t act1, const ConvGeom& g, const ConvLayout& L, char* cstate,
                             int32_t act2, const PoolGeom& pg, const PoolLayout& PL, char* pstate,
                             const void* x, int64_t x_bc, void* z, int64_t z_bc,
                             const co_step_plan& cplan, const co_pool_plan* pplan, bool update,
                             hipStream_t stream);

// Delay line and residual merges (delay.hip).
hipError_t launch_delay_init(const DelayGeom& g, char* state, const StateHeader& hdr,
                             hipStream_t stream);
hipError_t launch_delay_step(const DelayGeom& g, char* state, const void* x, const void* a,
                             void* y, int64_t n, bool emit, bool update, hipStream_t stream);
hipError_t launch_delay_steps(const DelayGeom& g, char* state, const void* x, int32_t T,
                              const void* a, void* y, int32_t y_frames, int64_t n0,
                              int32_t t_first, int32_t nout, bool update, hipStream_t stream);
// Elementwise activation of n contiguous elements (y may alias x).
hipError_t launch_act(const void* x, void* y, int64_t n, int32_t dtype, int32_t act,
                      hipStream_t stream);
hipError_t launch_add_frames(const void* a, const void* x, void* y, int64_t rows, int32_t E,
                             int32_t a_frames, int32_t x_frames, int32_t x_offset, int32_t dtype,
                             hipStream_t stream);

}  // namespace coinf
