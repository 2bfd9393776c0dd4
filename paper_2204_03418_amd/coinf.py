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
CO_F32, CO_BF16 = 0, 1
CO_ALGO_AUTO, CO_ALGO_DIRECT, CO_ALGO_GEMM, CO_ALGO_DEPTHWISE, CO_ALGO_GEMM_REG = 0, 1, 2, 3, 4
CO_ALGO_GEMM_IMG = 5
CO_POOL_AVG, CO_POOL_MAX = 0, 1
CO_MAX_TAPS = 64
CO_TAP_NONE, CO_TAP_START, CO_TAP_ACC, CO_TAP_EMIT, CO_TAP_EMIT_FRESH = 0, 1, 2, 3, 4

ALGOS = {"auto": CO_ALGO_AUTO, "direct": CO_ALGO_DIRECT, "gemm": CO_ALGO_GEMM,
         "depthwise": CO_ALGO_DEPTHWISE, "gemm_reg": CO_ALGO_GEMM_REG,
         "gemm_img": CO_ALGO_GEMM_IMG}
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
co_pool_query = _sig("co_pool_query", i32, [PD, PI])
co_pool_plan_step = _sig("co_pool_plan_step", i32, [PD, i64, ctypes.POINTER(PoolPlan)])
co_pool_init_state = _sig("co_pool_init_state", i32, [PD, vp, i64, vp, pvp])
co_pool_forward_step = _sig("co_pool_forward_step", i32, [vp, vp, vp, i32, vp])
co_pool_forward_steps = _sig("co_pool_forward_steps", i32,
                             [vp, vp, i32, vp, i32, i32, i32, vp, pi32])
co_pool_forward = _sig("co_pool_forward", i32, [PD, vp, i32, vp, vp])
co_pool_steps_fused = _sig("co_pool_steps_fused", i32, [vp, i32, i32, pi32])
co_pool_clip_frames = _sig("co_pool_clip_frames", i32, [PD, i32, pi32])
co_pool_clean_state = _sig("co_pool_clean_state", i32, [vp, vp])
co_pool_get_steps = _sig("co_pool_get_steps", i32, [vp, pi64])
co_pool_attach_state = _sig("co_pool_attach_state", i32, [PD, vp, i64, i64, vp, pvp])
co_pool_destroy = _sig("co_pool_destroy", i32, [vp])


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
    (B, C_in, *in_size).  kernel geometry comes from weight.shape.
    """

    def __init__(self, weight, bias=None, *, batch, in_size=(), stride=1, padding=0,
                 dilation=1, groups=1, algo="auto", state=None, attach_steps=None):
        dt = DTYPES[weight.dtype]
        self.torch_dtype = weight.dtype
        self.desc = conv_desc(batch, weight.shape[1] * groups, weight.shape[0],
                              tuple(weight.shape[2:]), tuple(in_size), stride, padding, dilation,
                              groups, bias is not None, dt, algo)
        self.info = conv_query(self.desc)
        self.batch, self.in_size = batch, tuple(in_size)
        self.in_channels, self.out_channels = weight.shape[1] * groups, weight.shape[0]
        self.out_size = tuple(self.info.out_size[:len(in_size)])
        self.weight, self.bias = weight, bias
        dev = weight.device
        if state is None:
            state = torch.empty(self.info.state_bytes, dtype=torch.uint8, device=dev)
        self.state = state
        h = ctypes.c_void_p()
        if attach_steps is None:
            _need(weight, weight.dtype, weight.shape, "weight")
            if bias is not None:
                _need(bias, weight.dtype, (weight.shape[0],), "bias")
            check(co_conv_init_state(ctypes.byref(self.desc), _ptr(weight), _ptr(bias),
                                     _ptr(state), state.numel(), _stream(), ctypes.byref(h)),
                  "co_conv_init_state")
        else:
            check(co_conv_attach_state(ctypes.byref(self.desc), _ptr(state), state.numel(),
                                       int(attach_steps), _stream(), ctypes.byref(h)),
                  "co_conv_attach_state")
        self.handle = h

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            co_conv_destroy(h)
            self.handle = None

    @property
    def delay(self):
        return self.info.delay

    @property
    def receptive_field(self):
        return self.info.receptive_field

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
        """Principle 2 forward_steps over x (B, C_in, T, *S); None when empty."""
        T = x.shape[2]
        _need(x, self.torch_dtype, (self.batch, self.in_channels, T) + self.in_size, "x")
        cap = T + (self.desc.padding[0] if pad_end else 0)
        y = torch.empty((self.batch, self.out_channels, cap) + self.out_size,
                        dtype=self.torch_dtype, device=x.device)
        n = i32()
        check(co_conv_forward_steps(self.handle, _ptr(x), T, _ptr(y), cap,
                                    1 if pad_end else 0, 1 if update_state else 0, _stream(),
                                    ctypes.byref(n)), "co_conv_forward_steps")
        if n.value == 0:
            return None
        return y[:, :, :n.value]

    def steps_fused(self, T, pad_end=False):
        """True when forward_steps over T frames runs as one persistent launch."""
        cap = T + (self.desc.padding[0] if pad_end else 0)
        f = i32()
        check(co_conv_steps_fused(self.handle, T, cap, ctypes.byref(f)), "co_conv_steps_fused")
        return bool(f.value)

    def forward(self, x):
        """Principle 2 forward (clip mode), stateless."""
        return conv_forward(self.desc, self.weight, self.bias, x)

    def clean_state(self):
        check(co_conv_clean_state(self.handle, _stream()), "co_conv_clean_state")


def conv_forward(desc, weight, bias, x):
    T = x.shape[2]
    t_out = i32()
    check(co_conv_clip_frames(ctypes.byref(desc), T, ctypes.byref(t_out)), "co_conv_clip_frames")
    sd = desc.spatial_dims
    info = conv_query(desc)
    y = torch.empty((desc.batch, desc.out_channels, t_out.value) + tuple(info.out_size[:sd]),
                    dtype=x.dtype, device=x.device)
    check(co_conv_forward(ctypes.byref(desc), _ptr(weight), _ptr(bias), _ptr(x), T, _ptr(y),
                          _stream()), "co_conv_forward")
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

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            co_pool_destroy(h)
            self.handle = None

    @property
    def delay(self):
        return self.info.delay

    @property
    def receptive_field(self):
        return self.info.receptive_field

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
        cap = T + (self.desc.padding[0] if pad_end else 0)
        y = torch.empty((self.batch, self.channels, cap) + self.out_size,
                        dtype=self.torch_dtype, device=x.device)
        n = i32()
        check(co_pool_forward_steps(self.handle, _ptr(x), T, _ptr(y), cap,
                                    1 if pad_end else 0, 1 if update_state else 0, _stream(),
                                    ctypes.byref(n)), "co_pool_forward_steps")
        if n.value == 0:
            return None
        return y[:, :, :n.value]

    def steps_fused(self, T, pad_end=False):
        """True when forward_steps over T frames runs as one persistent launch."""
        cap = T + (self.desc.padding[0] if pad_end else 0)
        f = i32()
        check(co_pool_steps_fused(self.handle, T, cap, ctypes.byref(f)), "co_pool_steps_fused")
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
