/*
 * coinf.h -- continual convolution and pooling steps on AMD MI355X (gfx950).
 *
 * C ABI of libcoinf.so.  The operations follow the statement of Continual
 * Inference Networks in Hedegaard & Iosifidis, "Continual Inference: A Library
 * for Efficient Online Inference with Deep Neural Networks in PyTorch"
 * (arXiv 2204.03418):
 *
 *   - Definition 1 (section 2): step inference equals batch inference for
 *     identical receptive fields, with one set of parameters;
 *   - Principle 1 (section 3.1): forward, weights and constructor arguments as
 *     PyTorch's nn.ConvNd / nn.AvgPoolNd / nn.MaxPoolNd;
 *   - Assumption 1 (section 3.1): clip tensors are (B, C, T, S1, S2), step
 *     tensors are (B, C, S1, S2);
 *   - Principle 2 (section 3.1): the call modes forward, forward_step and
 *     forward_steps;
 *   - Principle 3 (section 3.1): state rules (steps use and update state,
 *     update_state = 0 computes without updating, forward is stateless,
 *     clean_state wipes, outputs are empty until the delay has elapsed);
 *   - Principle 4 (section 3.1): delay d = f - p - 1, f the receptive field and
 *     p the temporal padding; padding reduces the delay and end padding is
 *     only applied on request (pad_end);
 *   - Principle 5 (section 3.1): a temporal stride s gives one non-empty output
 *     every s steps.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  Every tensor argument is a DEVICE pointer to contiguous memory in
 * the layout stated at the function.  The caller allocates and frees all
 * device memory (inputs, outputs, weights, bias and the state buffer, whose
 * size *_query reports).  The library allocates only the small host handle
 * (freed by *_destroy) and, in co_conv_forward_steps / co_pool_forward_steps
 * with update_state = 0, a stream-ordered temporary copy of the state that it
 * frees on the same stream.  It keeps the state pointer until destroy and no
 * other pointer past the call.
 *
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  All device
 * work is enqueued on it; no call synchronises the host except
 * *_attach_state, which reads the state header back.
 *
 * Status.  CO_OK: an output frame was written.  CO_EMPTY: the call was valid
 * and produced no output (before the delay, or between strided outputs);
 * the output buffer is untouched and the state advanced if update_state.
 * Negative values: nothing was enqueued and the handle is unchanged.  The
 * OK/EMPTY decision depends only on the step counter, so it is known on
 * return, before the device work runs.
 *
 * Dtypes.  CO_F32 and CO_BF16 name the dtype of x, y, weight and bias.
 * Accumulation and the state are float32 in both cases; bf16 results are
 * rounded to nearest-even once, when written.
 *
 * Threads.  A handle is not thread-safe; distinct handles are independent.
 * Concurrent calls on one state buffer race.
 *
 * Handles.  The library keeps a registry of the handles it has made and not
 * yet destroyed: a call with a destroyed handle, a second destroy, or a
 * handle of another kind returns CO_EINVAL.  A step counter stays below
 * 2^62: a call that would pass it returns CO_EINVAL.
 */
#ifndef COINF_H
#define COINF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t co_status;
#define CO_OK        0   /* output written */
#define CO_EMPTY     1   /* valid call, no output (Figure 1: empty outputs) */
#define CO_EINVAL   -1   /* invalid argument or descriptor */
#define CO_ENOTSUP  -2   /* valid but unsupported (e.g. a forced algorithm) */
#define CO_ESTATE   -3   /* state buffer too small or not made for this descriptor */
#define CO_EHIP     -4   /* the HIP runtime reported an error */
#define CO_ESCRATCH -5   /* the call needs more than the no-allocation scratch holds */

#define CO_F32   0
#define CO_BF16  1

/* Algorithm choice for a convolution (all compute the same result). */
#define CO_ALGO_AUTO       0   /* library heuristic: depthwise where it applies;
                                  else the register GEMM below 3e8
                                  multiply-accumulates per step, the
                                  warp-specialized GEMM, the LDS-tiled GEMM,
                                  the register GEMM, the direct kernel: the
                                  first that applies (tiny layers direct) */
#define CO_ALGO_DIRECT     1   /* generic direct kernel, any shape */
#define CO_ALGO_GEMM       2   /* implicit GEMM on MFMA, operand tiles staged
                                  through LDS (groups = 1) */
#define CO_ALGO_DEPTHWISE  3   /* depthwise stencil (groups = C_in = C_out) */
#define CO_ALGO_GEMM_REG   4   /* implicit GEMM on MFMA with register operands
                                  (groups = 1, small kH*kW*C_in) */
#define CO_ALGO_GEMM_WS    5   /* implicit GEMM on MFMA, warp-specialized: producer
                                  waves stage the input, consumer waves stream the
                                  weights from L2 (bf16, groups = 1, 3x3 spatial
                                  taps, stride and dilation 1, spatial padding <= 1,
                                  Ho*Wo a multiple of 4) */

#define CO_POOL_AVG  0
#define CO_POOL_MAX  1

/* Elementwise activations (section 3.2: activation functions compose with
 * continual modules as stateless per-frame maps). */
#define CO_ACT_NONE  0
#define CO_ACT_RELU  1         /* max(x, 0) */

#define CO_MAX_TAPS  64        /* largest temporal kernel size kT */

/* Per-tap actions of one convolution step (see co_conv_plan_step). */
#define CO_TAP_NONE        0   /* tap inactive this step */
#define CO_TAP_START       1   /* first contribution: ring slot := partial */
#define CO_TAP_ACC         2   /* ring slot += partial */
#define CO_TAP_EMIT        3   /* y := ring slot + partial + bias (output completes) */
#define CO_TAP_EMIT_FRESH  4   /* y := partial + bias (the output's only real tap) */

/*
 * Convolution descriptor (Principle 1: the nn.ConvNd constructor arguments).
 * spatial_dims 0, 1, 2 selects Conv1d, Conv2d, Conv3d; the first axis of
 * kernel/stride/padding/dilation is time, the rest are spatial.  Unused
 * spatial axes must have in_size 1, kernel 1, stride 1, padding 0, dilation 1.
 * Temporal padding must satisfy 0 <= padding[0] <= f - 1 (non-negative
 * delay, Principle 4); spatial padding is ordinary zero padding per frame.
 */
typedef struct co_conv_desc {
  int32_t spatial_dims;
  int32_t batch;                  /* B independent streams, one shared clock (Principle 7) */
  int32_t in_channels;
  int32_t out_channels;
  int32_t groups;
  int32_t in_size[2];             /* S1, S2 */
  int32_t kernel[3];
  int32_t stride[3];
  int32_t padding[3];
  int32_t dilation[3];
  int32_t has_bias;
  int32_t dtype;                  /* CO_F32 | CO_BF16 */
  int32_t algo;                   /* CO_ALGO_* */
} co_conv_desc;

typedef struct co_conv_info {
  int32_t receptive_field;        /* f = dilation[0] * (kernel[0] - 1) + 1 */
  int32_t delay;                  /* d = f - padding[0] - 1 (Principle 4) */
  int32_t out_size[2];            /* spatial output sizes, unused axes 1 */
  int32_t ring_slots;             /* partial-sum frames kept in the state */
  int32_t algo;                   /* algorithm resolved from desc->algo */
  int64_t state_bytes;            /* size of the caller-allocated state buffer */
} co_conv_info;

/* What one step does, as decided on the host from the step counter alone. */
typedef struct co_step_plan {
  int32_t emit;                   /* 1 when the step outputs a frame */
  int32_t n_taps;                 /* kernel[0] */
  int64_t out_index;              /* index of the emitted output frame, -1 if none */
  int8_t  action[CO_MAX_TAPS];    /* CO_TAP_* per temporal tap j */
  int32_t slot[CO_MAX_TAPS];      /* ring slot the tap touches, -1 if none */
  int64_t target[CO_MAX_TAPS];    /* output frame the tap contributes to, -1 if none */
} co_step_plan;

typedef struct co_conv_handle co_conv_handle;

/* Human-readable name of a status code (static string). */
const char* co_status_str(co_status s);

/*
 * Validate a descriptor and report receptive field, delay (Principle 4),
 * spatial output sizes and the state size.  Host only; touches no device.
 * Returns CO_EINVAL for an invalid descriptor, CO_ENOTSUP when a forced
 * algorithm cannot run it.
 */
co_status co_conv_query(const co_conv_desc* desc, co_conv_info* info);

/*
 * The schedule of step n (0-based count of frames consumed since a clean
 * state): which temporal taps of the newly arrived frame are active, the
 * output frame each feeds and its ring slot, and whether an output completes
 * (Principles 3-5).  update_state = 0 keeps only the completing tap, since
 * nothing else may change the state.  The plan of an end-padding frame
 * (pad_end) is the plan of its step.  Host only; touches no device.
 */
co_status co_conv_plan_step(const co_conv_desc* desc, int64_t n, int32_t update_state,
                            co_step_plan* plan);

/*
 * Create a handle over a caller-allocated state buffer of at least
 * info.state_bytes bytes.  Packs `weight` (C_out, C_in/groups, kT[, kH[, kW]],
 * desc->dtype) and `bias` (C_out, desc->dtype; may be NULL when !has_bias)
 * into the state -- one set of parameters for step and clip inference
 * (Definition 1) -- and starts from a clean state (step counter 0, the
 * padding "pre-saturating" the state as described after Example 2).  The
 * weight and bias buffers are read on `stream` and may be freed once that
 * work has completed.
 */
co_status co_conv_init_state(const co_conv_desc* desc, const void* weight, const void* bias,
                             void* state, int64_t state_bytes, void* stream,
                             co_conv_handle** out);

/*
 * co_conv_init_state with an evaluation-mode batch normalisation of the
 * convolution's output folded in (section 3.2: the library's continual
 * convolutions compose with nn.BatchNorm layers; the paper's Inception listing
 * wraps each one as conv -> BatchNorm3d -> ReLU).  Per output channel o,
 * scale = gamma[o] / sqrt(var[o] + eps) multiplies the weights of o before
 * they are rounded to the packed dtype (bf16 for the matrix-core kernels,
 * float32 for the direct and depthwise kernels) and the bias becomes
 * bias[o] * scale + beta[o] - mean[o] * scale (bias taken as 0 when
 * has_bias = 0); every step then emits BN(conv(x)).  gamma, beta, mean and
 * var are float32 device arrays of C_out; eps >= 0.  Otherwise as
 * co_conv_init_state.
 */
co_status co_conv_init_state_bn(const co_conv_desc* desc, const void* weight, const void* bias,
                                const float* gamma, const float* beta, const float* mean,
                                const float* var, float eps, void* state, int64_t state_bytes,
                                void* stream, co_conv_handle** out);

/*
 * The folded layer itself, for clip mode (co_conv_forward) over the same
 * layer: w_out (C_out, C_in/groups, kT, kH, kW) and b_out (C_out) in the io
 * dtype, caller-allocated device arrays.  Each weight is scaled and rounded
 * to the io dtype exactly as the matrix-core packing of
 * co_conv_init_state_bn rounds it; the bias is the float32 folded bias
 * rounded to the io dtype (so a bf16 clip carries a bf16 bias where the
 * steps add the float32 one).
 */
co_status co_conv_fold_bn(const co_conv_desc* desc, const void* weight, const void* bias,
                          const float* gamma, const float* beta, const float* mean,
                          const float* var, float eps, void* w_out, void* b_out, void* stream);

/*
 * forward_step (Principle 2): consume one frame x_t (B, C_in, S1, S2) and,
 * when the schedule emits, write the completed output y_t (B, C_out, So1, So2)
 * for the output frame delayed by `delay` steps.  Returns CO_OK or CO_EMPTY.
 * update_state = 0 computes the same output without changing the state
 * (Principle 3).
 */
co_status co_conv_forward_step(co_conv_handle* h, const void* x_t, void* y_t,
                               int32_t update_state, void* stream);

/*
 * forward_steps (Principle 2): consume T frames of x (B, C_in, T, S1, S2) as
 * T forward_step calls and write the non-empty outputs, in order, into
 * y (B, C_out, y_cap_frames, So1, So2) starting at frame 0.  pad_end = 1
 * appends padding[0] end-padding zero frames (Principle 4 text).  *n_out
 * receives the number of frames written.  CO_EINVAL (nothing enqueued) when
 * more than y_cap_frames outputs would be produced.  update_state = 0 leaves
 * the state as it was before the call.
 */
co_status co_conv_forward_steps(co_conv_handle* h, const void* x, int32_t T, void* y,
                                int32_t y_cap_frames, int32_t pad_end, int32_t update_state,
                                void* stream, int32_t* n_out);

/*
 * forward_steps without device allocation, for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Arguments, outputs, status and state semantics are those of
 * co_conv_forward_steps; the two give bitwise equal outputs and states.
 *
 * Where co_conv_forward_steps makes stream-ordered allocations -- the
 * backup of the ring for update_state = 0 when the call loops over step
 * launches, and contiguous copies of a frame (or output) that a matrix-core
 * step kernel cannot address in place (misaligned, or past 2^31 bytes of
 * reach) -- this entry point uses a scratch array the library holds in
 * device memory: 64 MiB per GPU (co_conv_scratch_bytes), allocated when the
 * library's code object is loaded on that GPU and held until the process
 * ends.  It calls no hipMalloc, hipFree or allocating library routine.
 *
 * Returns CO_ESCRATCH (nothing enqueued, handle unchanged) when the call
 * needs more scratch than that: the ring's bytes (R x B x C_out x Ho x Wo x 4,
 * rounded up to 256) with update_state = 0 on the looping path, plus the
 * staged frame copies.  A call that runs as one persistent launch
 * (co_conv_steps_fused) needs none.
 *
 * All calls on one GPU share that GPU's scratch, and each call leaves its
 * contents behind: calls whose device work overlaps on one GPU (different
 * streams, or threads) race.  Calls ordered on one stream do not.
 */
co_status co_conv_forward_steps_noalloc(co_conv_handle* h, const void* x, int32_t T, void* y,
                                        int32_t y_cap_frames, int32_t pad_end,
                                        int32_t update_state, void* stream, int32_t* n_out);

/* Bytes of device scratch co_conv_forward_steps_noalloc holds per GPU.  Host-only. */
co_status co_conv_scratch_bytes(int64_t* bytes);

/*
 * How co_conv_forward_steps runs a call over T frames into y_cap_frames
 * output frames: *fused = 1 when the whole call is one persistent kernel
 * launch that keeps the partial sums on chip across frames, 0 when it
 * enqueues one step per frame.  Both give the same outputs, bit for bit.
 * With temporal stride and dilation 1 the depthwise, direct, register-GEMM
 * and bf16 GEMM families run fused within their kernels' size limits; with
 * a temporal stride or dilation above 1 (Principle 5) the depthwise family
 * on planes of at most 64 pixels, the direct family and the register GEMM's
 * 1x1-spatial shapes do, following the step plans, when the ring has at most
 * 8 slots, kT <= 10, sT R <= 64 and (kT - 1) dT <= 32.  Host-only.
 */
co_status co_conv_steps_fused(const co_conv_handle* h, int32_t T, int32_t y_cap_frames,
                              int32_t* fused);

/*
 * forward (Principle 2, clip mode): the regular convolution of the clip
 * x (B, C_in, T, S1, S2) with symmetric temporal padding padding[0], written
 * to y (B, C_out, T_out, So1, So2), T_out = floor((T + 2p - f)/s) + 1 (0 when
 * negative: nothing is written).  Stateless (Principle 3): no handle.
 */
co_status co_conv_forward(const co_conv_desc* desc, const void* weight, const void* bias,
                          const void* x, int32_t T, void* y, void* stream);

/* Evaluation-mode batch normalisation of a convolution's output, as
 * co_conv_init_state_bn takes it: float32 device arrays of C_out. */
typedef struct {
  const float* gamma;
  const float* beta;
  const float* mean;
  const float* var;
  float eps;
} co_bn_params;

/*
 * forward (clip mode) on the step kernels: the same result as
 * co_conv_forward (Principle 2: a clip processed by the continual layer from
 * a clean state, with padding[0] end-padding frames, emits exactly the
 * regular convolution's T_out frames; Example 1, Principle 4) up to
 * summation order, computed by building a clean state in the caller's
 * workspace (workspace_bytes >= state_bytes of co_conv_query; CO_ESTATE
 * otherwise) and running co_conv_forward_steps with end padding over x read
 * in place -- on the matrix-core kernels AUTO (or desc->algo) picks, one
 * persistent launch where co_conv_steps_fused says so.  bn, when not NULL,
 * folds a batch normalisation in as co_conv_init_state_bn does, so a folded
 * layer's clip equals its steps bit for bit.  The workspace is scratch: its
 * contents are undefined afterwards.  Nothing is allocated, except the
 * stream-ordered staging copy co_conv_forward_steps makes for a clip whose
 * reach passes 2^31 bytes on a kernel that loops over steps.
 */
co_status co_conv_forward_ws(const co_conv_desc* desc, const void* weight, const void* bias,
                             const co_bn_params* bn, const void* x, int32_t T, void* y,
                             void* workspace, int64_t workspace_bytes, void* stream);

/* Number of T_out frames co_conv_forward produces for a clip of T frames. */
co_status co_conv_clip_frames(const co_conv_desc* desc, int32_t T, int32_t* t_out);

/* clean_state (Principle 3): wipe the state; the next step is step 0. */
co_status co_conv_clean_state(co_conv_handle* h, void* stream);

/* Step counter n of the handle (frames consumed since the last clean state). */
co_status co_conv_get_steps(const co_conv_handle* h, int64_t* n);

/*
 * Output frames a forward_steps call over T frames (plus padding[0] end
 * frames when pad_end) emits when it starts at step counter n0: the steps
 * m in [n0, n0 + count) with m >= delay and (m - delay) mod stride[0] == 0
 * (Principles 4-5: the first output after `delay` steps, then one every
 * temporal stride).  With n0 = co_conv_get_steps of a handle, the capacity
 * co_conv_forward_steps needs.  Host-only.
 */
co_status co_conv_out_frames(const co_conv_desc* desc, int64_t n0, int32_t T, int32_t pad_end,
                             int32_t* n_out);

/*
 * Resume from a state buffer that co_conv_init_state prepared for the same
 * descriptor, after its step-counter value `n` (e.g. a copy saved mid-stream).
 * Nothing is zeroed or re-packed.  Reads the state header back synchronously;
 * CO_ESTATE when it does not match the descriptor.
 */
co_status co_conv_attach_state(const co_conv_desc* desc, void* state, int64_t state_bytes,
                               int64_t n, void* stream, co_conv_handle** out);

/* Free the host handle (the state buffer stays the caller's). */
co_status co_conv_destroy(co_conv_handle* h);

/* Name of the kernel family a handle runs ("direct", "gemm_bf16", ...). */
const char* co_conv_algo_name(const co_conv_handle* h);

/*
 * Continual pooling (section 3.2, pooling; Principles 1-5).  The receptive
 * field f = dilation[0] (kernel[0] - 1) + 1 and the delay f - padding[0] - 1
 * follow Principle 4 as for convolutions.  Each arriving frame is reduced
 * spatially once; the state keeps the last f reduced frames (a FIFO of
 * fifo_slots float32 frames with a validity flag each), and an emitting step
 * reduces the window's frames over time.  Layouts, ownership, streams,
 * status and update_state are those of the convolution calls above.
 *
 * Pool descriptor (Principle 1: nn.AvgPoolNd / nn.MaxPoolNd arguments;
 * stride must be given explicitly, ceil_mode is not supported).  An input
 * frame (B x C x S1 x S2 elements) must stay below 2^31 bytes (CO_EINVAL).  Padding on
 * each axis is at most kernel/2 as in PyTorch; dilation is only allowed for
 * CO_POOL_MAX.  Average pooling counts pads in the divisor when
 * count_include_pad is set (PyTorch's default); maximum pooling ignores pads.
 */
typedef struct co_pool_desc {
  int32_t kind;                   /* CO_POOL_AVG | CO_POOL_MAX */
  int32_t spatial_dims;
  int32_t batch;
  int32_t channels;
  int32_t in_size[2];
  int32_t kernel[3];
  int32_t stride[3];
  int32_t padding[3];
  int32_t dilation[3];
  int32_t count_include_pad;
  int32_t dtype;
} co_pool_desc;

typedef struct co_pool_info {
  int32_t receptive_field;
  int32_t delay;
  int32_t out_size[2];
  int32_t fifo_slots;             /* spatially pooled frames kept in the state */
  int32_t reserved;
  int64_t state_bytes;
} co_pool_info;

/* One pool step: the FIFO slot written and, when emitting, the window read. */
typedef struct co_pool_plan {
  int32_t emit;
  int32_t n_taps;
  int64_t out_index;
  int32_t write_slot;             /* slot of the newly arrived frame */
  int32_t reserved;
  int32_t src[CO_MAX_TAPS];       /* per tap: slot, -1 = start padding, -2 = this frame */
} co_pool_plan;

typedef struct co_pool_handle co_pool_handle;

/* Receptive field, delay (Principle 4), output frame size and state bytes of
 * a descriptor; CO_EINVAL / CO_ENOTSUP as co_conv_query.  Host-only. */
co_status co_pool_query(const co_pool_desc* desc, co_pool_info* info);

/* The schedule of step n (Principles 3-5): whether it emits, which output,
 * the FIFO slot the arriving frame takes and the slots the window reads.
 * Host-only. */
co_status co_pool_plan_step(const co_pool_desc* desc, int64_t n, co_pool_plan* plan);

/* Clean state (Principle 3) over a caller-allocated buffer of
 * info.state_bytes bytes: the header is written, the FIFO marked empty.
 * CO_ESTATE when the buffer is too small. */
co_status co_pool_init_state(const co_pool_desc* desc, void* state, int64_t state_bytes,
                             void* stream, co_pool_handle** out);

/* forward_step of a continual pool (Principle 2): x_t (B, C, S1, S2) ->
 * y_t (B, C, So1, So2), written when the step emits (CO_OK), else CO_EMPTY
 * with y_t untouched.  Average pools divide by the window volume (pads
 * counted, count_include_pad) or by the valid positions; maximum pools skip
 * pads.  update_state = 0 neither stores x_t nor advances the counter. */
co_status co_pool_forward_step(co_pool_handle* h, const void* x_t, void* y_t,
                               int32_t update_state, void* stream);

/* forward_steps of a continual pool (Principle 2; pad_end appends padding[0]
 * pad frames as at the end of Example 1's clip); same conventions as
 * co_conv_forward_steps. */
co_status co_pool_forward_steps(co_pool_handle* h, const void* x, int32_t T, void* y,
                                int32_t y_cap_frames, int32_t pad_end, int32_t update_state,
                                void* stream, int32_t* n_out);

/* As co_conv_steps_fused, for co_pool_forward_steps: fused for kT <= 5
 * and windows of at most 64 positions; with a temporal stride or dilation
 * above 1, global spatial pools over frames of 17 to 64 positions with
 * (kT - 1) dT < 32, and the other windows with a temporal stride alone. */
co_status co_pool_steps_fused(const co_pool_handle* h, int32_t T, int32_t y_cap_frames,
                              int32_t* fused);

/* forward (Principle 2, clip mode; Principle 1: the nn pool's result):
 * pooling of x (B, C, T, S1, S2) with symmetric temporal padding into
 * y (B, C, T_out, So1, So2); stateless. */
co_status co_pool_forward(const co_pool_desc* desc, const void* x, int32_t T, void* y,
                          void* stream);
/* Number of T_out frames co_pool_forward produces for a clip of T frames. */
co_status co_pool_clip_frames(const co_pool_desc* desc, int32_t T, int32_t* t_out);

/* clean_state (Principle 3): the next step is step 0; no device work. */
co_status co_pool_clean_state(co_pool_handle* h, void* stream);
/* Step counter n of the handle. */
co_status co_pool_get_steps(const co_pool_handle* h, int64_t* n);
/* As co_conv_out_frames (Principles 4-5), for co_pool_forward_steps. */
co_status co_pool_out_frames(const co_pool_desc* desc, int64_t n0, int32_t T, int32_t pad_end,
                             int32_t* n_out);
/* Resume from a copied state after step n; as co_conv_attach_state. */
co_status co_pool_attach_state(const co_pool_desc* desc, void* state, int64_t state_bytes,
                               int64_t n, void* stream, co_pool_handle** out);
/* Free the host handle (the state buffer stays the caller's). */
co_status co_pool_destroy(co_pool_handle* h);

/*
 * Fused step of a depthwise convolution and the pool that consumes its output
 * (sections 3.2-3.3; the X3D bottleneck closes with such a pair), when the
 * pool's spatial window is the whole output plane (kernel = stride = the
 * plane, no spatial padding: a 1x1 pooled frame), the plane has at most 64
 * pixels, the kernels are 3x3 or 1x1 with at most 8 temporal taps.  The
 * fused handle borrows the two
 * handles (it neither owns nor frees them) and advances their states and
 * step counters exactly as co_conv_forward_step followed, when the
 * convolution emits, by co_pool_forward_step would: the results are
 * identical, and fused and separate calls can be mixed.  The intermediate
 * frame is not written anywhere.  CO_ENOTSUP when the pair does not fit.
 */
typedef struct co_convpool_handle co_convpool_handle;

co_status co_convpool_bind(co_conv_handle* conv, co_pool_handle* pool, co_convpool_handle** out);

/* One step: x_t (B, C, S1, S2) in; the pool's output z_t (B, C, 1, 1) when
 * both emit (CO_OK), else CO_EMPTY with z_t untouched. */
co_status co_convpool_forward_step(co_convpool_handle* h, const void* x_t, void* z_t,
                                   int32_t update_state, void* stream);

/* T steps over x (B, C, T, S1, S2); the non-empty outputs, in order, into
 * z (B, C, z_cap_frames, 1, 1); *n_out = their count.  With temporal stride
 * and dilation 1 in both modules, both kT <= 5 and a padded input plane of
 * at most 128 elements the clip runs as one launch that keeps both states in
 * registers; otherwise as one fused launch per frame.  Same results either
 * way, and the same results as stepping. */
co_status co_convpool_forward_steps(co_convpool_handle* h, const void* x, int32_t T, void* z,
                                    int32_t z_cap_frames, int32_t update_state, void* stream,
                                    int32_t* n_out);

co_status co_convpool_destroy(co_convpool_handle* h);

/*
 * Fused step of an X3D-style bottleneck (sections 3.2-3.3; Table 2's CoX3D
 * networks are built from such blocks): a pointwise convolution (1x1x1,
 * stride 1, no padding, groups 1: delay 0) on the register-GEMM kernel
 * (CO_ALGO_GEMM_REG, which AUTO picks for such layers) and its activation
 * act1, a depthwise continual convolution and its activation act2, and the
 * pool over the depthwise output's whole plane (the pair co_convpool_bind
 * accepts), with batch normalisations folded into the convolutions by
 * co_conv_init_state_bn.  One launch per step: each workgroup computes a
 * 16-channel slice of the pointwise output on the matrix cores into LDS and
 * runs the depthwise and pool steps from there, so neither intermediate
 * frame is written anywhere.  The handle borrows the three handles and
 * advances their step counters and states exactly as the separate steps
 * (co_conv_forward_step, co_act_forward, co_conv_forward_step,
 * co_act_forward, co_pool_forward_step) would: the results are identical
 * bit for bit, and fused and separate calls can be mixed.  The chain's delay
 * is the depthwise convolution's plus the pool's (Principle 6; the pointwise
 * convolution adds none).  Planes of at most 64 pixels (128 with the
 * depthwise padding).  CO_ENOTSUP when the layers do not fit, CO_EINVAL for
 * an unknown activation.
 */
typedef struct co_bneck_handle co_bneck_handle;

co_status co_bneck_bind(co_conv_handle* pw, int32_t act1, co_conv_handle* dw, int32_t act2,
                        co_pool_handle* pool, co_bneck_handle** out);

/* One step: x_t (B, C_in, S1, S2) in; the pool's output z_t (B, C, 1, 1) when
 * the depthwise convolution and the pool both emit (CO_OK), else CO_EMPTY
 * with z_t untouched. */
co_status co_bneck_forward_step(co_bneck_handle* h, const void* x_t, void* z_t,
                                int32_t update_state, void* stream);

/* T steps over x (B, C_in, T, S1, S2), one fused launch per frame; the
 * non-empty outputs, in order, into z (B, C, z_cap_frames, 1, 1); *n_out =
 * their count.  With update_state = 0 the states are restored afterwards
 * (a stream-ordered copy, as co_conv_forward_steps). */
co_status co_bneck_forward_steps(co_bneck_handle* h, const void* x, int32_t T, void* z,
                                 int32_t z_cap_frames, int32_t update_state, void* stream,
                                 int32_t* n_out);

co_status co_bneck_destroy(co_bneck_handle* h);

/*
 * Delay (section 3.2, co.Delay): shifts a stream by `delay` steps, so that
 * parallel branches with different delays meet on the same frame
 * (Principle 7; residual connections, section 3.1.1).  Step n outputs input
 * frame n - delay; the first `delay` steps are empty.  The state is a ring of
 * `delay` input frames in the io dtype.  A frame is (batch, channels,
 * frame_elems) contiguous elements; frame_elems is the product of the
 * spatial sizes (1 for a 1-D stream).
 */
typedef struct co_delay_desc {
  int32_t batch;
  int32_t channels;
  int32_t frame_elems;
  int32_t delay;                  /* >= 0 */
  int32_t dtype;                  /* CO_F32 | CO_BF16 */
} co_delay_desc;

typedef struct co_delay_handle co_delay_handle;

/* State size of a descriptor (CO_EINVAL for an invalid one).  Host only. */
co_status co_delay_query(const co_delay_desc* desc, int64_t* state_bytes);

/* Clean state over a caller-allocated buffer of at least state_bytes bytes. */
co_status co_delay_init_state(const co_delay_desc* desc, void* state, int64_t state_bytes,
                              void* stream, co_delay_handle** out);

/*
 * forward_step: y_t := x_{n - delay} (CO_OK) or nothing (CO_EMPTY, n < delay).
 * y_t may be NULL to only advance the stream.  update_state = 0 reads
 * without storing x_t or advancing.
 */
co_status co_delay_forward_step(co_delay_handle* h, const void* x_t, void* y_t,
                                int32_t update_state, void* stream);

/*
 * Residual merge step (Principle 7, reduce "sum"): y_t := a_t + x_{n - delay}
 * in one pass, a_t being the wrapped module's output of this step (a_t and
 * y_t may alias).  CO_EMPTY with y_t untouched while n < delay; the stream
 * still advances.  Accumulates in float32 and rounds once to the io dtype.
 */
co_status co_delay_add_step(co_delay_handle* h, const void* x_t, const void* a_t, void* y_t,
                            int32_t update_state, void* stream);

/*
 * forward_steps over x (batch, channels, T, frame_elems): the non-empty
 * outputs, in order, into y (batch, channels, y_cap_frames, frame_elems);
 * *n_out = their count.  CO_EINVAL when they would exceed y_cap_frames.
 */
co_status co_delay_forward_steps(co_delay_handle* h, const void* x, int32_t T, void* y,
                                 int32_t y_cap_frames, int32_t update_state, void* stream,
                                 int32_t* n_out);

/*
 * Residual merge over clips: y[b, c, i] := a[b, c, i] + x[b, c, i + lag] for
 * i < a_frames, where the wrapped module's outputs a (batch, channels,
 * a_frames, frame_elems) are aligned with the last a_frames steps of this
 * call and lag = T - a_frames - delay + (steps before the call) is the
 * residual's offset into x.  Advances the stream by T steps like
 * co_delay_forward_steps (x_{n - delay} earlier than x comes from the ring).
 * CO_EINVAL when some residual frame precedes the stream.
 */
co_status co_delay_add_steps(co_delay_handle* h, const void* x, int32_t T, const void* a,
                             int32_t a_frames, void* y, int32_t update_state, void* stream);

/*
 * Clip-mode merge (no state): y[bc, i, e] := a[bc, i, e] + x[bc, i + x_offset, e]
 * for bc < rows, i < a_frames, e < frame_elems; a and y hold a_frames frames
 * per row, x holds x_frames.  Used by residual connections in clip mode,
 * where a centred residual is shrunk by x_offset frames (section 3.1.1).
 */
co_status co_add_frames(const void* a, const void* x, void* y, int32_t rows, int32_t frame_elems,
                        int32_t a_frames, int32_t x_frames, int32_t x_offset, int32_t dtype,
                        void* stream);

/*
 * Elementwise activation of n contiguous elements of dtype (a frame or a
 * clip): y = act(x); y may equal x.  Stateless, delay 0.  ReLU maps NaN to 0.
 * CO_EINVAL for an unknown act or dtype.
 */
co_status co_act_forward(const void* x, void* y, int64_t n, int32_t dtype, int32_t act,
                         void* stream);

co_status co_delay_clean_state(co_delay_handle* h, void* stream);
co_status co_delay_get_steps(const co_delay_handle* h, int64_t* n);
co_status co_delay_destroy(co_delay_handle* h);

/*
 * Alignment of a residual connection (section 3.1.1, Principle 7) around a
 * module of temporal receptive field f, stride s and padding p whose own
 * delay is module_delay: the input joins the module's output on the centre
 * of its receptive field, so the residual branch is delayed by
 * *res_delay = floor((f - 1) / 2) steps; in clip mode the input's first and
 * last *shrink = *res_delay - p frames have no module output to join;
 * the whole's delay is *delay = max(module_delay, *res_delay) (a step is
 * empty while either branch is).  CO_EINVAL unless s == 1 and
 * 0 <= 2p <= f - 1 (a longer output than input cannot be joined).
 * Host-only.
 */
co_status co_residual_align(int64_t f, int64_t s, int64_t p, int64_t module_delay,
                            int64_t* res_delay, int64_t* shrink, int64_t* delay);

/*
 * Accumulated receptive field and delay of a chain of n layers (Principle 6),
 * each layer given by its temporal receptive field f, stride s and padding p,
 * in the form the principle's worked example evaluates (f = {3, 3},
 * s = {2, 1}, p = {2, 0} gives f_acc = 7, p_acc = 2, d = 4):
 *   f_acc(0) = f(0), p_acc(0) = p(0), s_acc(0) = s(0);
 *   f_acc(i) = f_acc(i-1) + (f(i) - 1) * s_acc(i-1);
 *   p_acc(i) = p_acc(i-1) + p(i) * s_acc(i-1);
 *   s_acc(i) = s_acc(i-1) * s(i);
 *   d(i) = f_acc(i) - p_acc(i) - 1.
 * Writes the values of the last layer.  Host only.
 */
co_status co_chain_delay(int32_t n, const int32_t* f, const int32_t* s, const int32_t* p,
                         int64_t* f_acc, int64_t* p_acc, int64_t* s_acc, int64_t* delay);

#ifdef __cplusplus
}
#endif

#endif /* COINF_H */
