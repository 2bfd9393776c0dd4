"""Oracle for continual convolution and pooling steps.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no code
with the HIP library (``paper_2204_03418_amd``) and never imports it; the HIP
library never imports this package.

What it computes
----------------
The paper's Definition 1 (section 2) requires a continual network to produce
the same outputs in step inference as in batch inference for the same
receptive field, and Example 1 (section 3.1) asserts it for ``co.Conv3d``.  The
continual step therefore reaches exactly (up to rounding order) a result with a
plain definition, and this oracle is that definition written out:

* ``conv`` / ``pool`` -- ordinary N-d convolution and pooling (Principle 1:
  identical ``forward``), in ``oracle.c``, accumulated in float64;
* ``ContinualConv`` / ``ContinualPool`` -- a sliding-window driver that keeps
  the last ``f - 1`` real input frames (an input FIFO, deliberately *not* the
  partial-sum ring the GPU library keeps) and, on each step the schedule says
  is non-empty, runs the ordinary operation over the ``f`` virtual frames of
  that output's window (Principles 2-5).

Readings where the paper is silent or garbled are listed at the top of each
function that relies on them.

Pins (things other than this code that fix its values) live in
``tests/test_oracle_*.py``: PyTorch's CPU float64 convolution and pooling,
closed forms (impulse responses, constant inputs, box sums), linearity and
time-shift equivariance, brute-force window enumeration on tiny inputs, the
paper's Example 1 and the Principle 6 worked example.  Parity of exact float32
or bfloat16 bits with any GPU path is unpinned (summation order differs).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from collections import OrderedDict

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc into ``liboracle.so`` (plain C, -O2, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
             "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    i64 = ctypes.c_int64
    dp = ctypes.POINTER(ctypes.c_double)
    u8p = ctypes.POINTER(ctypes.c_uint8)
    lib.ora_conv.restype = None
    lib.ora_conv.argtypes = [dp, u8p] + [i64] * 5 + [dp] + [i64] * 5 + [dp] + [i64] * 8 + [dp]
    lib.ora_pool.restype = None
    lib.ora_pool.argtypes = ([ctypes.c_int32, dp, u8p] + [i64] * 5 + [i64] * 3 + [i64] * 3
                             + [i64] * 2 + [i64] * 3 + [ctypes.c_int32, dp])
    lib.ora_out_len.restype = i64
    lib.ora_out_len.argtypes = [i64] * 5
    lib.ora_set_threads.restype = None
    lib.ora_set_threads.argtypes = [ctypes.c_int32]
    lib.ora_max_threads.restype = ctypes.c_int32
    lib.ora_max_threads.argtypes = []
    _lib = lib
    return lib


def _dptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _u8ptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))


def set_threads(n: int) -> None:
    """Thread count of the oracle's OpenMP loops (process-wide)."""
    _load().ora_set_threads(int(n))


def max_threads() -> int:
    """Threads the oracle's OpenMP loops use now."""
    return int(_load().ora_max_threads())


def out_len(L: int, k: int, s: int, p: int, d: int) -> int:
    """Output length of one axis: floor((L + 2p - d(k-1) - 1)/s) + 1, or 0."""
    return int(_load().ora_out_len(L, k, s, p, d))


def _as5d(x, spatial_dims):
    """View a (B, C, T, *S) array as 5-D (B, C, T, H, W) with unit spatial axes."""
    x = np.asarray(x, dtype=np.float64)
    while x.ndim < 5:
        x = x[..., None]
    return np.ascontiguousarray(x)


def _expand(v, nd):
    """Per-axis tuple of length nd (time first) from an int or a sequence."""
    if isinstance(v, (int, np.integer)):
        return (int(v),) * nd
    v = tuple(int(e) for e in v)
    assert len(v) == nd, v
    return v


def conv_window(xw, tvalid, weight, bias, groups, stride_t, stride_s, pad_s, dil):
    """Ordinary convolution of an already temporally-padded window.

    xw      float64 (B, C_in, T, H, W); frames with tvalid == 0 are zero frames
    weight  float64 (C_out, C_in/groups, kT, kH, kW)
    stride_t temporal stride; stride_s (sH, sW); pad_s (pH, pW); dil (dT, dH, dW)
    Returns float64 (B, C_out, To, Ho, Wo).
    """
    lib = _load()
    xw = np.ascontiguousarray(xw, dtype=np.float64)
    tv = np.ascontiguousarray(tvalid, dtype=np.uint8)
    w = np.ascontiguousarray(weight, dtype=np.float64)
    B, Cin, T, H, W = xw.shape
    Cout, Cg, kT, kH, kW = w.shape
    assert Cin == Cg * groups and Cout % groups == 0
    assert tv.shape == (T,)
    dT, dH, dW = dil
    sH, sW = stride_s
    pH, pW = pad_s
    To = out_len(T, kT, stride_t, 0, dT)
    Ho = out_len(H, kH, sH, pH, dH)
    Wo = out_len(W, kW, sW, pW, dW)
    y = np.zeros((B, Cout, To, Ho, Wo), dtype=np.float64)
    if y.size == 0:
        return y
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float64)
    lib.ora_conv(_dptr(xw), _u8ptr(tv), B, Cin, T, H, W, _dptr(w), Cout, groups, kT, kH, kW,
                 _dptr(b) if b is not None else None,
                 stride_t, sH, sW, pH, pW, dT, dH, dW, _dptr(y))
    return y


def pool_window(kind, xw, tvalid, kernel, stride, pad_s, dil, count_include_pad):
    """Ordinary pooling of an already temporally-padded window.

    kind 'avg' | 'max'; xw float64 (B, C, T, H, W); kernel/stride/dil (T, H, W);
    pad_s (pH, pW).  Returns float64 (B, C, To, Ho, Wo).
    """
    lib = _load()
    xw = np.ascontiguousarray(xw, dtype=np.float64)
    tv = np.ascontiguousarray(tvalid, dtype=np.uint8)
    B, C, T, H, W = xw.shape
    kT, kH, kW = kernel
    sT, sH, sW = stride
    dT, dH, dW = dil
    pH, pW = pad_s
    To = out_len(T, kT, sT, 0, dT)
    Ho = out_len(H, kH, sH, pH, dH)
    Wo = out_len(W, kW, sW, pW, dW)
    y = np.zeros((B, C, To, Ho, Wo), dtype=np.float64)
    if y.size == 0:
        return y
    lib.ora_pool(1 if kind == "max" else 0, _dptr(xw), _u8ptr(tv), B, C, T, H, W,
                 kT, kH, kW, sT, sH, sW, pH, pW, dT, dH, dW,
                 1 if count_include_pad else 0, _dptr(y))
    return y


def _squeeze_spatial(y5, spatial_dims):
    """Drop the unit spatial axes added by _as5d: keep (B, C, T) + spatial_dims axes."""
    return y5.reshape(y5.shape[:3 + spatial_dims])


def _pad_time(x5, pT):
    B, C, T, H, W = x5.shape
    xp = np.zeros((B, C, T + 2 * pT, H, W), dtype=np.float64)
    xp[:, :, pT:pT + T] = x5
    tv = np.zeros(T + 2 * pT, dtype=np.uint8)
    tv[pT:pT + T] = 1
    return xp, tv


def conv_forward(x, weight, bias=None, stride=1, padding=0, dilation=1, groups=1):
    """Clip-mode forward (Principle 2, ``forward``): the regular N-d convolution.

    x (B, C_in, T, *S) with 0-2 spatial axes; weight (C_out, C_in/groups, kT, *kS).
    stride/padding/dilation: int or per-axis tuple, time first.  Symmetric
    temporal padding pT on both ends, exactly as nn.ConvNd.
    """
    x = np.asarray(x, dtype=np.float64)
    nd = x.ndim - 2
    sdims = nd - 1
    w = np.asarray(weight, dtype=np.float64)
    st, pd, dl = _expand(stride, nd), _expand(padding, nd), _expand(dilation, nd)
    st = st + (1,) * (3 - nd)
    pd = pd + (0,) * (3 - nd)
    dl = dl + (1,) * (3 - nd)
    x5 = _as5d(x, sdims)
    w5 = _as5d(w, sdims)
    xp, tv = _pad_time(x5, pd[0])
    y5 = conv_window(xp, tv, w5, bias, groups, st[0], st[1:], pd[1:], dl)
    return _squeeze_spatial(y5, sdims)


def pool_forward(kind, x, kernel, stride=None, padding=0, dilation=1, count_include_pad=True):
    """Clip-mode pooling (nn.AvgPoolNd / nn.MaxPoolNd forward; stride None = kernel)."""
    x = np.asarray(x, dtype=np.float64)
    nd = x.ndim - 2
    sdims = nd - 1
    k = _expand(kernel, nd)
    st = k if stride is None else _expand(stride, nd)
    pd, dl = _expand(padding, nd), _expand(dilation, nd)
    k = k + (1,) * (3 - nd)
    st = st + (1,) * (3 - nd)
    pd = pd + (0,) * (3 - nd)
    dl = dl + (1,) * (3 - nd)
    x5 = _as5d(x, sdims)
    xp, tv = _pad_time(x5, pd[0])
    y5 = pool_window(kind, xp, tv, k, st, pd[1:], dl, count_include_pad)
    return _squeeze_spatial(y5, sdims)


PAD = None  # marker for a padded (zero / ignored) frame in the FIFO


class _ContinualBase:
    """Sliding-window continual driver shared by the conv and pool oracles.

    State (Principle 3): the most recent ``f - 1`` frames (an input FIFO keyed by
    the 0-based frame index) and the step counter ``n``.  Emission schedule
    (Principles 4 and 5): step ``n`` is non-empty iff ``n >= d`` and
    ``(n - d) mod sT == 0``; its output index is ``tau = (n - d) / sT`` and it
    covers virtual (padded) frames ``v = tau*sT .. tau*sT + f - 1``, where
    virtual frame ``v`` is real frame ``v - pT`` when that is >= 0, otherwise a
    start-padding zero frame (padding is pre-saturated state: section 3.1, text
    after Example 2).

    Readings: the delay is the same ``d = f - pT - 1`` for every stride, with the
    first output at step ``d`` and then one every ``sT`` steps; ``pT > f - 1``
    (negative delay) is rejected; ``pad_end`` appends exactly ``pT`` pad frames
    processed as ordinary steps.
    """

    def __init__(self, kT, sT, pT, dT, spatial_dims):
        self.kT, self.sT, self.pT, self.dT = kT, sT, pT, dT
        self.f = dT * (kT - 1) + 1          # receptive field
        self.d = self.f - pT - 1            # Principle 4: d = f - p - 1
        if self.d < 0:
            raise ValueError("temporal padding larger than receptive field - 1 (negative delay)")
        self.spatial_dims = spatial_dims
        self.clean_state()

    @property
    def delay(self):
        return self.d

    @property
    def receptive_field(self):
        return self.f

    def clean_state(self):
        """Principle 3: wipe the module state."""
        self.frames = OrderedDict()
        self.n = 0

    def _window(self, n):
        """Frames (or PAD) of the f virtual positions of the output emitted at step n."""
        v = n + self.pT
        out = []
        for vv in range(v - self.f + 1, v + 1):
            r = vv - self.pT
            out.append(PAD if r < 0 else self.frames[r])
        return out

    def forward_step(self, x_t, update_state=True):
        """One step (Principle 2); returns the output frame or None (empty)."""
        n = self.n
        saved = (OrderedDict(self.frames), self.n)
        self.frames[n] = None if x_t is PAD else np.asarray(x_t, dtype=np.float64)
        y = None
        if n >= self.d and (n - self.d) % self.sT == 0:
            y = self._reduce(self._window(n))
        # keep only what future windows can reach: the last f - 1 frames
        for k in list(self.frames.keys()):
            if k <= n - (self.f - 1):
                del self.frames[k]
        self.n = n + 1
        if not update_state:
            self.frames, self.n = saved
        return y

    def forward_steps(self, x, pad_end=False, update_state=True):
        """Principle 2 ``forward_steps``: repeated forward_step over the T axis,
        non-empty outputs concatenated along T (empty outputs dropped, as in
        Example 1 where 4 frames give 2 outputs).  ``pad_end`` appends pT
        padded frames.  With update_state False the state is left unchanged."""
        saved = (OrderedDict(self.frames), self.n)
        x = np.asarray(x, dtype=np.float64)
        outs = []
        for t in range(x.shape[2]):
            y = self.forward_step(x[:, :, t])
            if y is not None:
                outs.append(y)
        if pad_end:
            for _ in range(self.pT):
                y = self.forward_step(PAD)
                if y is not None:
                    outs.append(y)
        if not update_state:
            self.frames, self.n = saved
        if not outs:
            return None
        return np.stack(outs, axis=2)

    def _stack_window(self, win, like_shape):
        xs, tv = [], []
        for fr in win:
            if fr is None:
                xs.append(np.zeros(like_shape))
                tv.append(0)
            else:
                xs.append(fr)
                tv.append(1)
        x = np.stack(xs, axis=2)              # (B, C, f, *S)
        return x, np.array(tv, dtype=np.uint8)

    def _frame_shape(self, win):
        for fr in win:
            if fr is not None:
                return fr.shape
        raise AssertionError("an emitted window always holds the newest real frame")


class ContinualConv(_ContinualBase):
    """Continual ConvNd oracle (co.Conv1d/2d/3d semantics, section 3.2).

    weight (C_out, C_in/groups, kT, *kS) float64; bias (C_out,) or None;
    stride/padding/dilation ints or per-axis tuples (time first).  Spatial
    padding is ordinary per-frame zero padding; only temporal padding turns
    into a delay reduction.
    """

    def __init__(self, weight, bias=None, stride=1, padding=0, dilation=1, groups=1):
        w = np.asarray(weight, dtype=np.float64)
        nd = w.ndim - 2
        st, pd, dl = _expand(stride, nd), _expand(padding, nd), _expand(dilation, nd)
        self.weight = w
        self.bias = None if bias is None else np.asarray(bias, dtype=np.float64)
        self.groups = groups
        self.stride, self.padding, self.dilation = st, pd, dl
        super().__init__(w.shape[2], st[0], pd[0], dl[0], nd - 1)

    def _reduce(self, win):
        shape = self._frame_shape(win)
        xw, tv = self._stack_window(win, shape)
        sd = self.spatial_dims
        x5 = _as5d(xw, sd)
        w5 = _as5d(self.weight, sd)
        st = self.stride + (1,) * (2 - sd)
        pd = self.padding + (0,) * (2 - sd)
        dl = self.dilation + (1,) * (2 - sd)
        # the window is exactly f frames: temporal stride is irrelevant (one output)
        y5 = conv_window(x5, tv, w5, self.bias, self.groups, 1, st[1:], pd[1:], dl)
        assert y5.shape[2] == 1
        return y5[:, :, 0].reshape(y5.shape[:2] + y5.shape[3:3 + sd])

    def forward(self, x):
        """Principle 3: forward neither uses nor updates the state."""
        return conv_forward(x, self.weight, self.bias, self.stride, self.padding,
                            self.dilation, self.groups)


class ContinualPool(_ContinualBase):
    """Continual AvgPoolNd / MaxPoolNd oracle (co.AvgPool*, co.MaxPool*).

    kind 'avg' | 'max'; kernel/stride/padding/dilation time first; stride None
    means stride = kernel (nn default).  Readings: average counts pads as zeros
    and in the divisor when count_include_pad (nn default); maximum ignores
    pads (nn pads with -inf).
    """

    def __init__(self, kind, kernel, stride=None, padding=0, dilation=1,
                 count_include_pad=True, spatial_dims=2):
        nd = spatial_dims + 1
        k = _expand(kernel, nd)
        st = k if stride is None else _expand(stride, nd)
        self.kind = kind
        self.kernel, self.stride = k, st
        self.padding, self.dilation = _expand(padding, nd), _expand(dilation, nd)
        self.count_include_pad = count_include_pad
        super().__init__(k[0], st[0], self.padding[0], self.dilation[0], spatial_dims)

    def _reduce(self, win):
        shape = self._frame_shape(win)
        xw, tv = self._stack_window(win, shape)
        sd = self.spatial_dims
        x5 = _as5d(xw, sd)
        k = self.kernel + (1,) * (2 - sd)
        st = (1,) + self.stride[1:] + (1,) * (2 - sd)
        pd = self.padding + (0,) * (2 - sd)
        dl = self.dilation + (1,) * (2 - sd)
        y5 = pool_window(self.kind, x5, tv, k, st, pd[1:], dl, self.count_include_pad)
        assert y5.shape[2] == 1
        return y5[:, :, 0].reshape(y5.shape[:2] + y5.shape[3:3 + sd])

    def forward(self, x):
        return pool_forward(self.kind, x, self.kernel, self.stride, self.padding,
                            self.dilation, self.count_include_pad)


# ---------------------------------------------------------------- composition
#
# Section 3.1.1 (residual connections), section 3.2 (co.Delay), section 3.3
# (containers) and Principles 6-7.  Written from the text: a delay is a FIFO
# of input frames; parallel branches follow one clock and a merge of an empty
# value is empty (Principle 7); a chain passes each non-empty output on.


class ContinualDelay:
    """co.Delay(d): step n returns input frame n - d, empty (None) for n < d;
    forward (clip mode) is the identity."""

    def __init__(self, d):
        if d < 0:
            raise ValueError("negative delay")
        self.d = d
        self.clean_state()

    delay = property(lambda self: self.d)
    receptive_field = property(lambda self: self.d + 1)

    def clean_state(self):
        self.fifo = []
        self.n = 0

    def forward_step(self, x_t, update_state=True):
        fifo = self.fifo + [np.asarray(x_t, dtype=np.float64)]
        y = fifo.pop(0) if len(fifo) > self.d else None
        if update_state:
            self.fifo, self.n = fifo, self.n + 1
        return y

    def forward(self, x):
        return np.asarray(x, dtype=np.float64)


class BatchNormEval:
    """Batch normalisation in evaluation mode over channel axis 1 (the
    nn.BatchNorm1d/2d/3d modules a continual network composes with, section
    3.2): a per-channel affine map with the running statistics,

        y[:, c, ...] = (x[:, c, ...] - mean[c]) / sqrt(var[c] + eps) * gamma[c] + beta[c].

    It holds no state across time, so forward_step and forward apply the same
    map to a frame or a clip, and the delay is 0."""

    def __init__(self, gamma, beta, mean, var, eps=1e-5):
        self.gamma = np.asarray(gamma, dtype=np.float64)
        self.beta = np.asarray(beta, dtype=np.float64)
        self.mean = np.asarray(mean, dtype=np.float64)
        self.var = np.asarray(var, dtype=np.float64)
        self.eps = float(eps)

    delay = property(lambda self: 0)
    receptive_field = property(lambda self: 1)

    def clean_state(self):
        pass

    def forward(self, x):
        x = np.asarray(x, dtype=np.float64)
        shape = (1, -1) + (1,) * (x.ndim - 2)
        inv = 1.0 / np.sqrt(self.var + self.eps)
        return ((x - self.mean.reshape(shape)) * inv.reshape(shape) * self.gamma.reshape(shape)
                + self.beta.reshape(shape))

    def forward_step(self, x_t, update_state=True):
        return self.forward(x_t)


class ReLU:
    """The rectifier max(x, 0), elementwise (nn.ReLU in a continual network,
    section 3.2): stateless, delay 0."""

    delay = property(lambda self: 0)
    receptive_field = property(lambda self: 1)

    def clean_state(self):
        pass

    def forward(self, x):
        return np.maximum(np.asarray(x, dtype=np.float64), 0.0)

    def forward_step(self, x_t, update_state=True):
        return self.forward(x_t)


def _steps(mod, x):
    """forward_step over the T axis; non-empty outputs stacked (None if none)."""
    outs = [mod.forward_step(x[:, :, t]) for t in range(x.shape[2])]
    outs = [o for o in outs if o is not None]
    return np.stack(outs, axis=2) if outs else None


class ContinualParallelSum:
    """Two branches on one input stream and one clock, merged by a sum
    (Principle 7: the merge is empty whenever a branch's value is)."""

    def __init__(self, a, b):
        self.a, self.b = a, b

    delay = property(lambda self: max(self.a.delay, self.b.delay))

    def clean_state(self):
        self.a.clean_state()
        self.b.clean_state()

    def forward_step(self, x_t, update_state=True):
        ya = self.a.forward_step(x_t, update_state)
        yb = self.b.forward_step(x_t, update_state)
        if ya is None or yb is None:
            return None
        return ya + yb

    def forward_steps(self, x):
        return _steps(self, np.asarray(x, dtype=np.float64))


class ContinualResidual(ContinualParallelSum):
    """Residual connection (section 3.1.1) around a stride-1 module with
    receptive field f and temporal padding p: the input branch is delayed by
    (f - 1) // 2 steps, which aligns it with the centre of the module's
    window; clip mode adds the input shrunk by (f - 1) // 2 - p frames at each
    end (the centred residual; nothing is dropped with equal padding)."""

    def __init__(self, module):
        self.module = module
        self.shrink = (module.f - 1) // 2 - module.pT
        if self.shrink < 0:
            raise ValueError("more temporal padding than the centre alignment allows")
        super().__init__(module, ContinualDelay((module.f - 1) // 2))

    def forward(self, x):
        y = self.module.forward(x)
        x = np.asarray(x, dtype=np.float64)
        return y + x[:, :, self.shrink:self.shrink + y.shape[2]]


class ContinualChain:
    """Modules in sequence: each non-empty step output feeds the next module;
    an empty one ends the step (section 3.3, Sequential)."""

    def __init__(self, *mods):
        self.mods = list(mods)

    def clean_state(self):
        for m in self.mods:
            m.clean_state()

    def forward_step(self, x_t, update_state=True):
        for m in self.mods:
            x_t = m.forward_step(x_t, update_state)
            if x_t is None:
                return None
        return x_t

    def forward_steps(self, x):
        return _steps(self, np.asarray(x, dtype=np.float64))

    def forward(self, x):
        for m in self.mods:
            x = m.forward(x)
        return x


def chain_delay(f, s, p):
    """Principle 6 for layers with temporal receptive fields f, strides s and
    paddings p, in the form its worked example evaluates (the printed
    recurrences give f_acc = 5 and p_acc = 0 on that example, which states 7
    and 2): each layer's receptive field and padding count in units of the
    accumulated stride of the layers before it.  Returns the last layer's
    (f_acc, p_acc, s_acc, delay)."""
    f_acc, p_acc, s_acc = f[0], p[0], s[0]
    for fi, si, pi in zip(f[1:], s[1:], p[1:]):
        f_acc = f_acc + (fi - 1) * s_acc
        p_acc = p_acc + pi * s_acc
        s_acc = s_acc * si
    return f_acc, p_acc, s_acc, f_acc - p_acc - 1
