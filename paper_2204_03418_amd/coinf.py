"""ctypes binding of libcoinf.so (include/coinf.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI.  Tensors are PyTorch device tensors (the caller's
memory); the stream is PyTorch's current stream.  Importing this module loads
the library and raises ImportError when it has not been built; there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcoinf.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libcoinf.so is not built ({LIB_PATH}); run __graft_entry__.build()")
lib = ctypes.CDLL(LIB_PATH)

# ---------------------------------------------------------------- constants
CO_OK, CO_EMPTY, CO_EINVAL, CO_ENOTSUP, CO_ESTATE, CO_EHIP = 0, 1, -1, -2, -3, -4
CO_ESCRATCH = -5
CO_F32, CO_BF16 = 0, 1
CO_ALGO_AUTO, CO_ALGO_DIRECT, CO_ALGO_GEMM, CO_ALGO_DEPTHWISE, CO_ALGO_GEMM_REG = 0, 1, 2, 3, 4
CO_ALGO_GEMM_WS = 5
CO_ACT_NONE, CO_ACT_RELU = 0, 1
CO_POOL_AVG, CO_POOL_MAX = 0, 1
CO_MAX_TAPS = 64
CO_TAP_NONE, CO_TAP_START, CO_TAP_ACC, CO_TAP_EMIT, CO_TAP_EMIT_FRESH = 0, 1, 2, 3, 4

ALGOS = {"auto": CO_ALGO_AUTO, "direct": CO_ALGO_DIRECT, "gemm": CO_ALGO_GEMM,
         "depthwise": CO_ALGO_DEPTHWISE, "gemm_reg": CO_ALGO_GEMM_REG,
         "gemm_ws": CO_ALGO_GEMM_WS}
DTYPES = {torch.float32: CO_F32, torch.bfloat16: CO_BF16}

i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
I32x2, I32x3 = i32 * 2, i32 * 3


class ConvDesc(ctypes.Structure):
    _fields_ = [("spatial_dims", i32), ("batch", i32), ("in_channels", i32),
                ("out_channels", i32), ("groups", i32), ("in_size", I32x2),
                ("kernel", I32x3), ("stride", I32x3), ("padding", I32x3),
                ("dilation", I32x3), ("has_bias", i32), ("dtype", i32), ("algo", i32)]


class ConvInfo(ctypes.Structure):
    _fields_ = [("receptive_field", i32), ("delay", i32), ("out_size", I32x2),
                ("ring_slots", i32), ("algo", i32), ("state_bytes", i64)]


class StepPlan(ctypes.Structure):
    _fields_ = [("emit", i32), ("n_taps", i32), ("out_index", i64),
                ("action", ctypes.c_int8 * CO_MAX_TAPS), ("slot", i32 * CO_MAX_TAPS),
                ("target", i64 * CO_MAX_TAPS)]


class PoolDesc(ctypes.Structure):
    _fields_ = [("kind", i32), ("spatial_dims", i32), ("batch", i32), ("channels", i32),
                ("in_size", I32x2), ("kernel", I32x3), ("stride", I32x3), ("padding", I32x3),
                ("dilation", I32x3), ("count_include_pad", i32), ("dtype", i32)]


class PoolInfo(ctypes.Structure):
    _fields_ = [("receptive_field", i32), ("delay", i32), ("out_size", I32x2),
                ("fifo_slots", i32), ("reserved", i32), ("state_bytes", i64)]


class DelayDesc(ctypes.Structure):
    _fields_ = [("batch", i32), ("channels", i32), ("frame_elems", i32), ("delay", i32),
                ("dtype", i32)]


class PoolPlan(ctypes.Structure):
    _fields_ = [("emit", i32), ("n_taps", i32), ("out_index", i64), ("write_slot", i32),
                ("reserved", i32), ("src", i32 * CO_MAX_TAPS)]


def _sig(name, res, args):
    f = getattr(lib, name)
    f.restype = res
    f.argtypes = args
    return f


CD, CI, PD, PI = (ctypes.POINTER(ConvDesc), ctypes.POINTER(ConvInfo),
                  ctypes.POINTER(PoolDesc), ctypes.POINTER(PoolInfo))
pi32, pi64, pvp = ctypes.POINTER(i32), ctypes.POINTER(i64), ctypes.POINTER(vp)

co_status_str = _sig("co_status_str", ctypes.c_char_p, [i32])
co_conv_query = _sig("co_conv_query", i32, [CD, CI])
co_conv_plan_step = _sig("co_conv_plan_step", i32, [CD, i64, i32, ctypes.POINTER(StepPlan)])
co_conv_init_state = _sig("co_conv_init_state", i32, [CD, vp, vp, vp, i64, vp, pvp])
co_conv_forward_step = _sig("co_conv_forward_step", i32, [vp, vp, vp, i32, vp])
co_conv_forward_steps = _sig("co_conv_forward_steps", i32,
                             [vp, vp, i32, vp, i32, i32, i32, vp, pi32])
co_conv_forward = _sig("co_conv_forward", i32, [CD, vp, vp, vp, i32, vp, vp])
co_conv_clip_frames = _sig("co_conv_clip_frames", i32, [CD, i32, pi32])
co_conv_clean_state = _sig("co_conv_clean_state", i32, [vp, vp])
co_conv_get_steps = _sig("co_conv_get_steps", i32, [vp, pi64])
co_conv_attach_state = _sig("co_conv_attach_state", i32, [CD, vp, i64, i64, vp, pvp])
co_conv_destroy = _sig("co_conv_destroy", i32, [vp])
co_conv_algo_name = _sig("co_conv_algo_name", ctypes.c_char_p, [vp])
co_conv_steps_fused = _sig("co_conv_steps_fused", i32, [vp, i32, i32, pi32])
co_conv_forward_steps_noalloc = _sig("co_conv_forward_steps_noalloc", i32,
                                     [vp, vp, i32, vp, i32, i32, i32, vp, pi32])
co_conv_scratch_bytes = _sig("co_conv_scratch_bytes", i32, [pi64])
co_conv_out_frames = _sig("co_conv_out_frames", i32, [CD, i64, i32, i32, pi32])
co_pool_query = _sig("co_pool_query", i32, [PD, PI])
co_pool_plan_step = _sig("co_pool_plan_step", i32, [PD, i64, ctypes.POINTER(PoolPlan)])
co_pool_init_state = _sig("co_pool_init_state", i32, [PD, vp, i64, vp, pvp])
co_pool_forward_step = _sig("co_pool_forward_step", i32, [vp, vp, vp, i32, vp])
co_pool_forward_steps = _sig("co_pool_forward_steps", i32,
                             [vp, vp, i32, vp, i32, i32, i32, vp, pi32])
co_pool_forward = _sig("co_pool_forward", i32, [PD, vp, i32, vp, vp])
co_pool_steps_fused = _sig("co_pool_steps_fused", i32, [vp, i32, i32, pi32])
co_pool_out_frames = _sig("co_pool_out_frames", i32, [PD, i64, i32, i32, pi32])
co_pool_clip_frames = _sig("co_pool_clip_frames", i32, [PD, i32, pi32])
co_pool_clean_state = _sig("co_pool_clean_state", i32, [vp, vp])
co_pool_get_steps = _sig("co_pool_get_steps", i32, [vp, pi64])
co_pool_attach_state = _sig("co_pool_attach_state", i32, [PD, vp, i64, i64, vp, pvp])
co_pool_destroy = _sig("co_pool_destroy", i32, [vp])
DD = ctypes.POINTER(DelayDesc)
co_delay_query = _sig("co_delay_query", i32, [DD, pi64])
co_delay_init_state = _sig("co_delay_init_state", i32, [DD, vp, i64, vp, pvp])
co_delay_forward_step = _sig("co_delay_forward_step", i32, [vp, vp, vp, i32, vp])
co_delay_add_step = _sig("co_delay_add_step", i32, [vp, vp, vp, vp, i32, vp])
co_delay_forward_steps = _sig("co_delay_forward_steps", i32,
                              [vp, vp, i32, vp, i32, i32, vp, pi32])
co_delay_add_steps = _sig("co_delay_add_steps", i32, [vp, vp, i32, vp, i32, vp, i32, vp])
co_add_frames = _sig("co_add_frames", i32, [vp, vp, vp, i32, i32, i32, i32, i32, i32, vp])
co_delay_clean_state = _sig("co_delay_clean_state", i32, [vp, vp])
co_delay_get_steps = _sig("co_delay_get_steps", i32, [vp, pi64])
co_delay_destroy = _sig("co_delay_destroy", i32, [vp])
co_chain_delay = _sig("co_chain_delay", i32, [i32, pi32, pi32, pi32, pi64, pi64, pi64, pi64])
co_convpool_bind = _sig("co_convpool_bind", i32, [vp, vp, pvp])
co_convpool_forward_step = _sig("co_convpool_forward_step", i32, [vp, vp, vp, i32, vp])
co_convpool_forward_steps = _sig("co_convpool_forward_steps", i32,
                                 [vp, vp, i32, vp, i32, i32, vp, pi32])
co_convpool_destroy = _sig("co_convpool_destroy", i32, [vp])
pf32, f32 = ctypes.POINTER(ctypes.c_float), ctypes.c_float
co_conv_init_state_bn = _sig("co_conv_init_state_bn", i32,
                             [CD, vp, vp, vp, vp, vp, vp, f32, vp, i64, vp, pvp])
co_conv_fold_bn = _sig("co_conv_fold_bn", i32, [CD, vp, vp, vp, vp, vp, vp, f32, vp, vp, vp])
co_act_forward = _sig("co_act_forward", i32, [vp, vp, i64, i32, i32, vp])


class BnParams(ctypes.Structure):
    _fields_ = [("gamma", vp), ("beta", vp), ("mean", vp), ("var", vp), ("eps", ctypes.c_float)]


co_conv_forward_ws = _sig("co_conv_forward_ws", i32,
                          [CD, vp, vp, ctypes.POINTER(BnParams), vp, i32, vp, vp, i64, vp])
co_bneck_bind = _sig("co_bneck_bind", i32, [vp, i32, vp, i32, vp, pvp])
co_bneck_forward_step = _sig("co_bneck_forward_step", i32, [vp, vp, vp, i32, vp])
co_bneck_forward_steps = _sig("co_bneck_forward_steps", i32,
                              [vp, vp, i32, vp, i32, i32, vp, pi32])
co_bneck_destroy = _sig("co_bneck_destroy", i32, [vp])
co_residual_align = _sig("co_residual_align", i32, [i64, i64, i64, i64, pi64, pi64, pi64])


class CoinfError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {co_status_str(status).decode()} ({status})")


def check(status, what):
    if status < 0:
        raise CoinfError(status, what)
    return status


def _axes(v, nd, fill):
    """Per-axis 3-tuple (time first) from an int or sequence of nd values."""
    v = (int(v),) * nd if isinstance(v, int) else tuple(int(e) for e in v)
    assert len(v) == nd, v
    return v + (fill,) * (3 - nd)


def conv_desc(batch, in_channels, out_channels, kernel, in_size=(), stride=1, padding=0,
              dilation=1, groups=1, has_bias=True, dtype=CO_F32, algo="auto"):
    """Build a ConvDesc; kernel/stride/padding/dilation are time first."""
    sd = len(in_size)
    nd = sd + 1
    d = ConvDesc()
    d.spatial_dims = sd
    d.batch, d.in_channels, d.out_channels, d.groups = batch, in_channels, out_channels, groups
    d.in_size = I32x2(*(tuple(in_size) + (1,) * (2 - sd)))
    d.kernel = I32x3(*_axes(kernel, nd, 1))
    d.stride = I32x3(*_axes(stride, nd, 1))
    d.padding = I32x3(*_axes(padding, nd, 0))
    d.dilation = I32x3(*_axes(dilation, nd, 1))
    d.has_bias = 1 if has_bias else 0
    d.dtype = dtype
    d.algo = ALGOS[algo] if isinstance(algo, str) else int(algo)
    return d


def pool_desc(kind, batch, channels, kernel, in_size=(), stride=None, padding=0, dilation=1,
              count_include_pad=True, dtype=CO_F32):
    sd = len(in_size)
    nd = sd + 1
    d = PoolDesc()
    d.kind = CO_POOL_MAX if kind == "max" else CO_POOL_AVG
    d.spatial_dims = sd
    d.batch, d.channels = batch, channels
    d.in_size = I32x2(*(tuple(in_size) + (1,) * (2 - sd)))
    d.kernel = I32x3(*_axes(kernel, nd, 1))
    d.stride = I32x3(*_axes(kernel if stride is None else stride, nd, 1))
    d.padding = I32x3(*_axes(padding, nd, 0))
    d.dilation = I32x3(*_axes(dilation, nd, 1))
    d.count_include_pad = 1 if count_include_pad else 0
    d.dtype = dtype
    return d


def conv_query(desc):
    info = ConvInfo()
    check(co_conv_query(ctypes.byref(desc), ctypes.byref(info)), "co_conv_query")
    return info


def conv_plan(desc, n, update_state=True):
    p = StepPlan()
    check(co_conv_plan_step(ctypes.byref(desc), n, 1 if update_state else 0, ctypes.byref(p)),
          "co_conv_plan_step")
    return p


def pool_query(desc):
    info = PoolInfo()
    check(co_pool_query(ctypes.byref(desc), ctypes.byref(info)), "co_pool_query")
    return info


def pool_plan(desc, n):
    p = PoolPlan()
    check(co_pool_plan_step(ctypes.byref(desc), n, ctypes.byref(p)), "co_pool_plan_step")
    return p


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _need(t, dtype, shape, what):
    if t.device.type != "cuda":
        raise ValueError(f"{what} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{what} has dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")


class CoConv:
    """A continual ConvNd layer over a device state buffer (co_conv_* ABI).

    weight (C_out, C_in/groups, kT, *kS) and bias (C_out,) are device tensors
    of one dtype (float32 or bfloat16); batch and in_size fix the frame shape
    (B, C_in, *in_size).  kernel geometry comes from weight.shape.  bn =
    (gamma, beta, running_mean, running_var, eps), float32 device tensors of
    C_out and a float, folds an evaluation-mode batch normalisation of the
    output into the layer (co_conv_init_state_bn): every step emits
    BN(conv(x)).
    """

    def __init__(self, weight, bias=None, *, batch, in_size=(), stride=1, padding=0,
                 dilation=1, groups=1, algo="auto", state=None, attach_steps=None, bn=None):
        dt = DTYPES[weight.dtype]
        self.torch_dtype = weight.dtype
        self.desc = conv_desc(batch, weight.shape[1] * groups, weight.shape[0],
                              tuple(weight.shape[2:]), tuple(in_size), stride, padding, dilation,
                              groups, bias is not None, dt, algo)
        self.info = conv_query(self.desc)
        self.batch, self.in_size = batch, tuple(in_size)
        self.in_channels, self.out_channels = weight.shape[1] * groups, weight.shape[0]
        self.out_size = tuple(self.info.out_size[:len(in_size)])
        self.weight, self.bias, self.bn = weight, bias, bn
        dev = weight.device
        if state is None:
            state = torch.empty(self.info.state_bytes, dtype=torch.uint8, device=dev)
        self.state = state
        h = ctypes.c_void_p()
        if attach_steps is None:
            _need(weight, weight.dtype, weight.shape, "weight")
            if bias is not None:
                _need(bias, weight.dtype, (weight.shape[0],), "bias")
            if bn is None:
                check(co_conv_init_state(ctypes.byref(self.desc), _ptr(weight), _ptr(bias),
                                         _ptr(state), state.numel(), _stream(),
                                         ctypes.byref(h)), "co_conv_init_state")
            else:
                check(co_conv_init_state_bn(ctypes.byref(self.desc), _ptr(weight), _ptr(bias),
                                            *self._bn_args(), _ptr(state), state.numel(),
                                            _stream(), ctypes.byref(h)),
                      "co_conv_init_state_bn")
        else:
            check(co_conv_attach_state(ctypes.byref(self.desc), _ptr(state), state.numel(),
                                       int(attach_steps), _stream(), ctypes.byref(h)),
                  "co_conv_attach_state")
        self.handle = h

    def _bn_args(self):
        gamma, beta, mean, var, eps = self.bn
        for t, what in ((gamma, "gamma"), (beta, "beta"), (mean, "running_mean"),
                        (var, "running_var")):
            _need(t, torch.float32, (self.out_channels,), what)
        return _ptr(gamma), _ptr(beta), _ptr(mean), _ptr(var), float(eps)

    # the destroy function is bound as a default so that objects collected
    # during interpreter shutdown, after the module globals are cleared, still
    # release their handles
    def __del__(self, _destroy=co_conv_destroy):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            _destroy(h)
            self.handle = None

    @property
    def delay(self):
        return self.info.delay

    @property
    def receptive_field(self):
        return self.info.receptive_field

    @property
    def t_stride(self):
        return self.desc.stride[0]

    @property
    def t_padding(self):
        return self.desc.padding[0]

    @property
    def algo(self):
        return co_conv_algo_name(self.handle).decode()

    @property
    def steps(self):
        n = i64()
        check(co_conv_get_steps(self.handle, ctypes.byref(n)), "co_conv_get_steps")
        return n.value

    def frame_shape(self):
        return (self.batch, self.in_channels) + self.in_size

    def out_frame_shape(self):
        return (self.batch, self.out_channels) + self.out_size

    def new_output(self):
        return torch.empty(self.out_frame_shape(), dtype=self.torch_dtype, device=self.state.device)

    def forward_step(self, x_t, update_state=True, out=None):
        """Principle 2 forward_step; returns the output frame or None (empty)."""
        _need(x_t, self.torch_dtype, self.frame_shape(), "x_t")
        y = self.new_output() if out is None else out
        _need(y, self.torch_dtype, self.out_frame_shape(), "out")
        st = check(co_conv_forward_step(self.handle, _ptr(x_t), _ptr(y),
                                        1 if update_state else 0, _stream()),
                   "co_conv_forward_step")
        return y if st == CO_OK else None

    def forward_step_raw(self, x_ptr, y_ptr, update_state=True, stream=None):
        """forward_step on raw device pointers (no checks); returns the status."""
        return co_conv_forward_step(self.handle, x_ptr, y_ptr, 1 if update_state else 0,
                                    _stream(stream))

    def forward_steps(self, x, pad_end=False, update_state=True):
        """Principle 2 forward_steps over x (B, C_in, T, *S); None when empty.
        The result is contiguous, sized to the frames the call emits."""
        T = x.shape[2]
        _need(x, self.torch_dtype, (self.batch, self.in_channels, T) + self.in_size, "x")
        cap = self.out_frames(T, pad_end)
        y = torch.empty((self.batch, self.out_channels, cap) + self.out_size,
                        dtype=self.torch_dtype, device=x.device)
        n = i32()
        check(co_conv_forward_steps(self.handle, _ptr(x), T, _ptr(y), cap,
                                    1 if pad_end else 0, 1 if update_state else 0, _stream(),
                                    ctypes.byref(n)), "co_conv_forward_steps")
        if n.value == 0:
            return None
        return y[:, :, :n.value]

    def out_frames(self, T, pad_end=False):
        """Frames forward_steps over T frames emits from the current step."""
        return conv_out_frames(self.desc, self.steps, T, pad_end)

    def steps_fused(self, T, pad_end=False):
        """True when forward_steps over T frames runs as one persistent launch."""
        f = i32()
        check(co_conv_steps_fused(self.handle, T, self.out_frames(T, pad_end), ctypes.byref(f)),
              "co_conv_steps_fused")
        return bool(f.value)

    def folded(self):
        """(weight, bias) with the batch normalisation folded in, in the io
        dtype (co_conv_fold_bn); the layer's own when it has none."""
        if self.bn is None:
            return self.weight, self.bias
        w = torch.empty_like(self.weight)
        b = torch.empty(self.out_channels, dtype=self.torch_dtype, device=self.weight.device)
        check(co_conv_fold_bn(ctypes.byref(self.desc), _ptr(self.weight), _ptr(self.bias),
                              *self._bn_args(), _ptr(w), _ptr(b), _stream()), "co_conv_fold_bn")
        return w, b

    def forward(self, x):
        """Principle 2 forward (clip mode), stateless: on the step kernels
        from a clean state in a scratch workspace (co_conv_forward_ws), with
        the batch normalisation folded in as the steps have it."""
        bn = None
        if self.bn is not None:
            gamma, beta, mean, var, eps = self._bn_args()
            bn = BnParams(gamma, beta, mean, var, eps)
        return conv_forward(self.desc, self.weight, self.bias, x, bn=bn)

    def clean_state(self):
        check(co_conv_clean_state(self.handle, _stream()), "co_conv_clean_state")


def conv_out_frames(desc, n0, T, pad_end=False):
    """Frames forward_steps over T frames emits from step counter n0
    (co_conv_out_frames)."""
    n = i32()
    check(co_conv_out_frames(ctypes.byref(desc), int(n0), int(T), 1 if pad_end else 0,
                             ctypes.byref(n)), "co_conv_out_frames")
    return n.value


def pool_out_frames(desc, n0, T, pad_end=False):
    """Frames a pool's forward_steps over T frames emits from step counter n0
    (co_pool_out_frames)."""
    n = i32()
    check(co_pool_out_frames(ctypes.byref(desc), int(n0), int(T), 1 if pad_end else 0,
                             ctypes.byref(n)), "co_pool_out_frames")
    return n.value


def residual_align(f, s, p, module_delay):
    """(residual delay, clip shrink, delay of the whole) of a centred residual
    (co_residual_align); None when the clip shapes cannot be joined."""
    d_res, shrink, delay = i64(), i64(), i64()
    st = co_residual_align(int(f), int(s), int(p), int(module_delay), ctypes.byref(d_res),
                           ctypes.byref(shrink), ctypes.byref(delay))
    if st != CO_OK:
        return None
    return d_res.value, shrink.value, delay.value


def conv_forward(desc, weight, bias, x, bn=None, direct=False):
    """Clip-mode forward: on the step kernels AUTO picks, from a clean state
    in a scratch workspace (co_conv_forward_ws), or with direct=True on the
    direct clip kernel (co_conv_forward)."""
    T = x.shape[2]
    t_out = i32()
    check(co_conv_clip_frames(ctypes.byref(desc), T, ctypes.byref(t_out)), "co_conv_clip_frames")
    sd = desc.spatial_dims
    info = conv_query(desc)
    y = torch.empty((desc.batch, desc.out_channels, t_out.value) + tuple(info.out_size[:sd]),
                    dtype=x.dtype, device=x.device)
    if direct:
        if bn is not None:
            raise ValueError("the direct clip kernel takes no batch normalisation")
        check(co_conv_forward(ctypes.byref(desc), _ptr(weight), _ptr(bias), _ptr(x), T, _ptr(y),
                              _stream()), "co_conv_forward")
        return y
    ws = torch.empty(info.state_bytes, dtype=torch.uint8, device=x.device)
    check(co_conv_forward_ws(ctypes.byref(desc), _ptr(weight), _ptr(bias),
                             ctypes.byref(bn) if bn is not None else None, _ptr(x), T, _ptr(y),
                             _ptr(ws), ws.numel(), _stream()), "co_conv_forward_ws")
    return y


class CoPool:
    """A continual AvgPoolNd / MaxPoolNd layer over a device state buffer."""

    def __init__(self, kind, *, batch, channels, kernel, in_size=(), stride=None, padding=0,
                 dilation=1, count_include_pad=True, dtype=torch.float32, device="cuda",
                 state=None, attach_steps=None):
        self.torch_dtype = dtype
        self.desc = pool_desc(kind, batch, channels, kernel, tuple(in_size), stride, padding,
                              dilation, count_include_pad, DTYPES[dtype])
        self.info = pool_query(self.desc)
        self.batch, self.channels, self.in_size = batch, channels, tuple(in_size)
        self.out_size = tuple(self.info.out_size[:len(in_size)])
        if state is None:
            state = torch.empty(self.info.state_bytes, dtype=torch.uint8, device=device)
        self.state = state
        h = ctypes.c_void_p()
        if attach_steps is None:
            check(co_pool_init_state(ctypes.byref(self.desc), _ptr(state), state.numel(),
                                     _stream(), ctypes.byref(h)), "co_pool_init_state")
        else:
            check(co_pool_attach_state(ctypes.byref(self.desc), _ptr(state), state.numel(),
                                       int(attach_steps), _stream(), ctypes.byref(h)),
                  "co_pool_attach_state")
        self.handle = h

    # the destroy function is bound as a default so that objects collected
    # during interpreter shutdown, after the module globals are cleared, still
    # release their handles
    def __del__(self, _destroy=co_pool_destroy):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            _destroy(h)
            self.handle = None

    @property
    def delay(self):
        return self.info.delay

    @property
    def receptive_field(self):
        return self.info.receptive_field

    @property
    def t_stride(self):
        return self.desc.stride[0]

    @property
    def t_padding(self):
        return self.desc.padding[0]

    @property
    def steps(self):
        n = i64()
        check(co_pool_get_steps(self.handle, ctypes.byref(n)), "co_pool_get_steps")
        return n.value

    def frame_shape(self):
        return (self.batch, self.channels) + self.in_size

    def out_frame_shape(self):
        return (self.batch, self.channels) + self.out_size

    def forward_step(self, x_t, update_state=True, out=None):
        _need(x_t, self.torch_dtype, self.frame_shape(), "x_t")
        y = torch.empty(self.out_frame_shape(), dtype=self.torch_dtype,
                        device=x_t.device) if out is None else out
        _need(y, self.torch_dtype, self.out_frame_shape(), "out")
        st = check(co_pool_forward_step(self.handle, _ptr(x_t), _ptr(y),
                                        1 if update_state else 0, _stream()),
                   "co_pool_forward_step")
        return y if st == CO_OK else None

    def forward_step_raw(self, x_ptr, y_ptr, update_state=True, stream=None):
        return co_pool_forward_step(self.handle, x_ptr, y_ptr, 1 if update_state else 0,
                                    _stream(stream))

    def forward_steps(self, x, pad_end=False, update_state=True):
        T = x.shape[2]
        _need(x, self.torch_dtype, (self.batch, self.channels, T) + self.in_size, "x")
        cap = self.out_frames(T, pad_end)
        y = torch.empty((self.batch, self.channels, cap) + self.out_size,
                        dtype=self.torch_dtype, device=x.device)
        n = i32()
        check(co_pool_forward_steps(self.handle, _ptr(x), T, _ptr(y), cap,
                                    1 if pad_end else 0, 1 if update_state else 0, _stream(),
                                    ctypes.byref(n)), "co_pool_forward_steps")
        if n.value == 0:
            return None
        return y[:, :, :n.value]

    def out_frames(self, T, pad_end=False):
        """Frames forward_steps over T frames emits from the current step."""
        return pool_out_frames(self.desc, self.steps, T, pad_end)

    def steps_fused(self, T, pad_end=False):
        """True when forward_steps over T frames runs as one persistent launch."""
        f = i32()
        check(co_pool_steps_fused(self.handle, T, self.out_frames(T, pad_end), ctypes.byref(f)),
              "co_pool_steps_fused")
        return bool(f.value)

    def forward(self, x):
        T = x.shape[2]
        t_out = i32()
        check(co_pool_clip_frames(ctypes.byref(self.desc), T, ctypes.byref(t_out)),
              "co_pool_clip_frames")
        y = torch.empty((self.batch, self.channels, t_out.value) + self.out_size,
                        dtype=x.dtype, device=x.device)
        check(co_pool_forward(ctypes.byref(self.desc), _ptr(x), T, _ptr(y), _stream()),
              "co_pool_forward")
        return y

    def clean_state(self):
        check(co_pool_clean_state(self.handle, _stream()), "co_pool_clean_state")


def chain_delay(layers):
    """Principle 6 over a chain of layers (anything with receptive_field,
    t_stride and t_padding): (f_acc, p_acc, s_acc, delay) of the last one."""
    n = len(layers)
    arr = i32 * n
    f = arr(*[m.receptive_field for m in layers])
    st = arr(*[m.t_stride for m in layers])
    p = arr(*[m.t_padding for m in layers])
    out = [i64() for _ in range(4)]
    check(co_chain_delay(n, f, st, p, *[ctypes.byref(o) for o in out]), "co_chain_delay")
    return tuple(o.value for o in out)


class CoDelay:
    """co.Delay: step n outputs frame n - delay (empty before); clip mode is
    the identity.  Frames are (batch, channels, *in_size)."""

    def __init__(self, delay, *, batch, channels, in_size=(), dtype=torch.float32,
                 device="cuda"):
        self.torch_dtype = dtype
        self.batch, self.channels, self.in_size = batch, channels, tuple(in_size)
        self.out_channels, self.out_size = channels, tuple(in_size)
        E = 1
        for v in in_size:
            E *= int(v)
        self.E = E
        self.desc = DelayDesc(batch, channels, E, int(delay), DTYPES[dtype])
        nb = i64()
        check(co_delay_query(ctypes.byref(self.desc), ctypes.byref(nb)), "co_delay_query")
        self.state = torch.empty(max(nb.value, 1), dtype=torch.uint8, device=device)
        h = ctypes.c_void_p()
        check(co_delay_init_state(ctypes.byref(self.desc), _ptr(self.state), self.state.numel(),
                                  _stream(), ctypes.byref(h)), "co_delay_init_state")
        self.handle = h

    # the destroy function is bound as a default so that objects collected
    # during interpreter shutdown, after the module globals are cleared, still
    # release their handles
    def __del__(self, _destroy=co_delay_destroy):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            _destroy(h)
            self.handle = None

    delay = property(lambda self: self.desc.delay)
    receptive_field = property(lambda self: self.desc.delay + 1)
    t_stride = property(lambda self: 1)
    t_padding = property(lambda self: 0)

    @property
    def steps(self):
        n = i64()
        check(co_delay_get_steps(self.handle, ctypes.byref(n)), "co_delay_get_steps")
        return n.value

    def frame_shape(self):
        return (self.batch, self.channels) + self.in_size

    def forward_step(self, x_t, update_state=True, out=None, emit=True):
        """x_{n - delay}, or None while empty; emit=False only advances."""
        _need(x_t, self.torch_dtype, self.frame_shape(), "x_t")
        y = None
        if emit:
            y = torch.empty_like(x_t) if out is None else out
        st = check(co_delay_forward_step(self.handle, _ptr(x_t), _ptr(y),
                                         1 if update_state else 0, _stream()),
                   "co_delay_forward_step")
        return y if (st == CO_OK and emit) else None

    def add_step(self, x_t, a_t, update_state=True, out=None):
        """a_t + x_{n - delay} (the residual merge), or None while empty."""
        _need(x_t, self.torch_dtype, self.frame_shape(), "x_t")
        _need(a_t, self.torch_dtype, self.frame_shape(), "a_t")
        y = torch.empty_like(a_t) if out is None else out
        st = check(co_delay_add_step(self.handle, _ptr(x_t), _ptr(a_t), _ptr(y),
                                     1 if update_state else 0, _stream()), "co_delay_add_step")
        return y if st == CO_OK else None

    def forward_steps(self, x, update_state=True):
        T = x.shape[2]
        _need(x, self.torch_dtype, (self.batch, self.channels, T) + self.in_size, "x")
        y = torch.empty_like(x)
        n = i32()
        check(co_delay_forward_steps(self.handle, _ptr(x), T, _ptr(y), T,
                                     1 if update_state else 0, _stream(), ctypes.byref(n)),
              "co_delay_forward_steps")
        return y[:, :, :n.value] if n.value else None

    def add_steps(self, x, a, update_state=True):
        """a (the last a.shape[2] steps' module outputs) + the delayed x."""
        T = x.shape[2]
        _need(x, self.torch_dtype, (self.batch, self.channels, T) + self.in_size, "x")
        na = 0 if a is None else a.shape[2]
        y = None
        if na:
            _need(a, self.torch_dtype, (self.batch, self.channels, na) + self.in_size, "a")
            y = torch.empty_like(a)
        check(co_delay_add_steps(self.handle, _ptr(x), T, _ptr(a) if na else None, na,
                                 _ptr(y) if na else None, 1 if update_state else 0, _stream()),
              "co_delay_add_steps")
        return y

    def forward(self, x):
        return x

    def clean_state(self):
        check(co_delay_clean_state(self.handle, _stream()), "co_delay_clean_state")


def add_frames(a, x, x_offset=0):
    """y[:, :, i] = a[:, :, i] + x[:, :, i + x_offset] (clip-mode merge)."""
    rows = a.shape[0] * a.shape[1]
    E = 1
    for v in a.shape[3:]:
        E *= int(v)
    y = torch.empty_like(a)
    check(co_add_frames(_ptr(a), _ptr(x), _ptr(y), rows, E, a.shape[2], x.shape[2],
                        int(x_offset), DTYPES[a.dtype], _stream()), "co_add_frames")
    return y


ACTS = {"none": CO_ACT_NONE, "relu": CO_ACT_RELU}


def act_forward(x, act="relu", out=None):
    """Elementwise activation of any contiguous tensor (co_act_forward)."""
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    y = torch.empty_like(x) if out is None else out
    _need(y, x.dtype, x.shape, "out")
    check(co_act_forward(_ptr(x), _ptr(y), x.numel(), DTYPES[x.dtype], ACTS[act], _stream()),
          "co_act_forward")
    return y


class CoReLU:
    """ReLU as a continual module: stateless and elementwise, so it has delay
    0 and receptive field 1 (section 3.2's composition of per-frame
    layers); every step emits."""

    delay, receptive_field, t_stride, t_padding = 0, 1, 1, 0
    act = "relu"

    def forward_step(self, x_t, update_state=True):
        return act_forward(x_t)

    def forward_steps(self, x, update_state=True):
        return act_forward(x.contiguous())

    def forward(self, x):
        return act_forward(x.contiguous())

    def clean_state(self):
        pass


class Bottleneck:
    """The X3D bottleneck front (pointwise CoConv -> optional ReLU ->
    depthwise CoConv -> optional ReLU -> CoPool over its whole output plane,
    batch normalisations folded into the convolutions) stepped as one launch
    per frame (co_bneck_*).  The three modules keep their states and step
    counters, and the outputs equal stepping them separately bit for bit.
    The pointwise layer must be a 1x1x1 CoConv on the register-GEMM kernel
    (algo "gemm_reg", AUTO's choice for such layers)."""

    def __init__(self, pw, relu1, dw, relu2, pool):
        h = ctypes.c_void_p()
        check(co_bneck_bind(pw.handle, CO_ACT_RELU if relu1 else CO_ACT_NONE, dw.handle,
                            CO_ACT_RELU if relu2 else CO_ACT_NONE, pool.handle,
                            ctypes.byref(h)), "co_bneck_bind")
        self.pw, self.relu1, self.dw, self.relu2, self.pool = pw, relu1, dw, relu2, pool
        self.handle = h

    @staticmethod
    def fits(pw, dw, pool):
        h = ctypes.c_void_p()
        if co_bneck_bind(pw.handle, CO_ACT_NONE, dw.handle, CO_ACT_NONE, pool.handle,
                         ctypes.byref(h)) != CO_OK:
            return False
        co_bneck_destroy(h)
        return True

    # the destroy function is bound as a default so that objects collected
    # during interpreter shutdown, after the module globals are cleared, still
    # release their handles
    def __del__(self, _destroy=co_bneck_destroy):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            _destroy(h)
            self.handle = None

    def _chain(self):
        return [self.pw, self.dw, self.pool]

    delay = property(lambda self: chain_delay(self._chain())[3])
    receptive_field = property(lambda self: chain_delay(self._chain())[0])
    t_stride = property(lambda self: chain_delay(self._chain())[2])
    t_padding = property(lambda self: chain_delay(self._chain())[1])

    def forward_step(self, x_t, update_state=True):
        _need(x_t, self.pw.torch_dtype, self.pw.frame_shape(), "x_t")
        z = torch.empty(self.pool.out_frame_shape(), dtype=self.pool.torch_dtype,
                        device=x_t.device)
        st = check(co_bneck_forward_step(self.handle, _ptr(x_t), _ptr(z),
                                         1 if update_state else 0, _stream()),
                   "co_bneck_forward_step")
        return z if st == CO_OK else None

    def forward_steps(self, x, update_state=True):
        T = x.shape[2]
        w, c, p = self.pw, self.dw, self.pool
        _need(x, w.torch_dtype, (w.batch, w.in_channels, T) + w.in_size, "x")
        # the pointwise layer emits every frame; the pool once per depthwise frame
        cap = pool_out_frames(p.desc, p.steps, conv_out_frames(c.desc, c.steps, T))
        z = torch.empty((p.batch, p.channels, cap) + p.out_size, dtype=p.torch_dtype,
                        device=x.device)
        n = i32()
        check(co_bneck_forward_steps(self.handle, _ptr(x), T, _ptr(z), cap,
                                     1 if update_state else 0, _stream(), ctypes.byref(n)),
              "co_bneck_forward_steps")
        return z if n.value else None

    def forward(self, x):
        y = self.pw.forward(x)
        if self.relu1:
            y = act_forward(y)
        y = self.dw.forward(y)
        if self.relu2:
            y = act_forward(y)
        return self.pool.forward(y)

    def clean_state(self):
        for m in self._chain():
            m.clean_state()


class ConvPool:
    """A depthwise CoConv followed by a CoPool over its whole output plane,
    stepped as one launch (co_convpool_*).  Both modules keep their states and
    step counters, and the outputs equal stepping them separately."""

    def __init__(self, conv, pool):
        h = ctypes.c_void_p()
        check(co_convpool_bind(conv.handle, pool.handle, ctypes.byref(h)), "co_convpool_bind")
        self.conv, self.pool, self.handle = conv, pool, h

    @staticmethod
    def fits(conv, pool):
        h = ctypes.c_void_p()
        if co_convpool_bind(conv.handle, pool.handle, ctypes.byref(h)) != CO_OK:
            return False
        co_convpool_destroy(h)
        return True

    # the destroy function is bound as a default so that objects collected
    # during interpreter shutdown, after the module globals are cleared, still
    # release their handles
    def __del__(self, _destroy=co_convpool_destroy):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            _destroy(h)
            self.handle = None

    delay = property(lambda self: chain_delay([self.conv, self.pool])[3])
    receptive_field = property(lambda self: chain_delay([self.conv, self.pool])[0])
    t_stride = property(lambda self: chain_delay([self.conv, self.pool])[2])
    t_padding = property(lambda self: chain_delay([self.conv, self.pool])[1])

    def _out(self, frames, device):
        return torch.empty((self.pool.batch, self.pool.channels, frames) + self.pool.out_size,
                           dtype=self.pool.torch_dtype, device=device)

    def forward_step(self, x_t, update_state=True):
        _need(x_t, self.conv.torch_dtype, self.conv.frame_shape(), "x_t")
        z = torch.empty(self.pool.out_frame_shape(), dtype=self.pool.torch_dtype,
                        device=x_t.device)
        st = check(co_convpool_forward_step(self.handle, _ptr(x_t), _ptr(z),
                                            1 if update_state else 0, _stream()),
                   "co_convpool_forward_step")
        return z if st == CO_OK else None

    def forward_steps(self, x, update_state=True):
        T = x.shape[2]
        c, p = self.conv, self.pool
        _need(x, c.torch_dtype, (c.batch, c.in_channels, T) + c.in_size, "x")
        # the pool steps once per emitted convolution frame
        cap = pool_out_frames(p.desc, p.steps, conv_out_frames(c.desc, c.steps, T))
        z = self._out(cap, x.device)
        n = i32()
        check(co_convpool_forward_steps(self.handle, _ptr(x), T, _ptr(z), cap,
                                        1 if update_state else 0, _stream(), ctypes.byref(n)),
              "co_convpool_forward_steps")
        return z if n.value else None

    def forward(self, x):
        return self.pool.forward(self.conv.forward(x))

    def clean_state(self):
        self.conv.clean_state()
        self.pool.clean_state()


class Sequential:
    """Section 3.3's Sequential: modules in a chain; an empty step output
    ends the step (downstream modules do not advance), and the chain's delay
    follows Principle 6.  With fuse (the default) a pointwise CoConv, an
    optional CoReLU, a depthwise CoConv, an optional CoReLU and a CoPool
    over its whole output plane run as one Bottleneck launch per step, and
    a depthwise CoConv directly followed by such a CoPool as one ConvPool
    launch, with identical results."""

    def __init__(self, *modules, fuse=True):
        mods = list(modules)
        if fuse:
            mods = self._fuse(mods)
        self.modules = mods

    @staticmethod
    def _bottleneck_at(mods, i):
        """(Bottleneck, modules consumed) starting at mods[i], or None."""
        j = i
        parts = []
        for kind in ("conv", "relu", "conv", "relu", "pool"):
            m = mods[j] if j < len(mods) else None
            if kind == "relu":
                parts.append(isinstance(m, CoReLU))
                j += 1 if isinstance(m, CoReLU) else 0
                continue
            want = CoConv if kind == "conv" else CoPool
            if not isinstance(m, want):
                return None
            parts.append(m)
            j += 1
        pw, r1, dw, r2, pool = parts
        if not Bottleneck.fits(pw, dw, pool):
            return None
        return Bottleneck(pw, r1, dw, r2, pool), j - i

    def _fuse(self, mods):
        out, i = [], 0
        while i < len(mods):
            a = mods[i]
            b = mods[i + 1] if i + 1 < len(mods) else None
            bn = self._bottleneck_at(mods, i)
            if bn is not None:
                out.append(bn[0])
                i += bn[1]
            elif isinstance(a, CoConv) and isinstance(b, CoPool) and ConvPool.fits(a, b):
                out.append(ConvPool(a, b))
                i += 2
            else:
                out.append(a)
                i += 1
        return out

    @property
    def delay(self):
        return chain_delay(self.modules)[3]

    @property
    def receptive_field(self):
        return chain_delay(self.modules)[0]

    @property
    def t_stride(self):
        return chain_delay(self.modules)[2]

    @property
    def t_padding(self):
        return chain_delay(self.modules)[1]

    def forward_step(self, x_t, update_state=True):
        for m in self.modules:
            x_t = m.forward_step(x_t, update_state=update_state)
            if x_t is None:
                return None
        return x_t

    def forward_steps(self, x, update_state=True):
        for m in self.modules:
            x = m.forward_steps(x, update_state=update_state)
            if x is None:
                return None
        return x

    def forward(self, x):
        for m in self.modules:
            x = m.forward(x)
        return x

    def clean_state(self):
        for m in self.modules:
            m.clean_state()


class Residual:
    """Section 3.1.1's residual connection around a module with equal input
    and output frames (stride 1): the input joins the module's output aligned
    on the centre of its receptive field, so the residual branch is delayed by
    (f - 1) // 2 steps (Principle 7: the whole has the module's delay, and a
    step is empty while either branch is).  With equal temporal padding
    ((f - 1) / 2) clip mode adds the input as is; a module with less padding
    needs residual_shrink=True, which drops the border frames of the input in
    clip mode (the centred residual)."""

    def __init__(self, module, residual_shrink=False):
        if module.t_stride != 1:
            raise ValueError("residual connections need temporal stride 1")
        al = residual_align(module.receptive_field, module.t_stride, module.t_padding,
                            module.delay)
        if al is None:
            raise ValueError("clip shapes differ: the module's temporal padding exceeds "
                             "(f - 1) / 2")
        self.module = module
        self.d_res, self.shrink, self._delay = al
        if self.shrink > 0 and not residual_shrink:
            raise ValueError("clip shapes differ: give the module padding (f - 1) / 2 or "
                             "residual_shrink=True")
        self.line = CoDelay(self.d_res, batch=module.batch, channels=module.out_channels,
                            in_size=module.out_size, dtype=module.torch_dtype,
                            device=module.state.device)

    delay = property(lambda self: self._delay)
    receptive_field = property(lambda self: self.module.receptive_field)
    t_stride = property(lambda self: 1)
    t_padding = property(lambda self: self.module.t_padding)
    batch = property(lambda self: self.module.batch)
    out_channels = property(lambda self: self.module.out_channels)
    out_size = property(lambda self: self.module.out_size)
    torch_dtype = property(lambda self: self.module.torch_dtype)

    def forward_step(self, x_t, update_state=True):
        a = self.module.forward_step(x_t, update_state=update_state)
        if a is None:
            self.line.forward_step(x_t, update_state=update_state, emit=False)
            return None
        return self.line.add_step(x_t, a, update_state=update_state, out=a)

    def forward_steps(self, x, update_state=True):
        a = self.module.forward_steps(x, update_state=update_state)
        return self.line.add_steps(x, a, update_state=update_state)

    def forward(self, x):
        a = self.module.forward(x)
        return add_frames(a, x, self.shrink)

    def clean_state(self):
        self.module.clean_state()
        self.line.clean_state()
