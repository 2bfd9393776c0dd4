"""Pins for the oracle's ordinary convolution (definition of Principle 1).

Each pin is something other than the oracle's own code: PyTorch's CPU float64
convolution (an independent library routine), closed forms (impulse response,
constant input, box sums computed with cumulative sums), and the algebraic
invariants of a convolution (linearity, time-shift equivariance).  The
``planted`` tests show that a plausible mistake (a tap-order flip, a dropped
bias, transposed spatial axes, a wrong group mapping) makes a pin fail.
"""
import itertools

import zlib

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

TORCH_CONV = {0: F.conv1d, 1: F.conv2d, 2: F.conv3d}


def _case_grid():
    rng = np.random.default_rng(1234)
    cases = []
    for sd in (0, 1, 2):
        for _ in range(14):
            nd = sd + 1
            k = tuple(int(v) for v in rng.integers(1, 4, nd))
            s = tuple(int(v) for v in rng.integers(1, 3, nd))
            d = tuple(int(v) for v in rng.integers(1, 3, nd))
            p = tuple(int(rng.integers(0, d[i] * (k[i] - 1) + 1)) for i in range(nd))
            G = int(rng.choice([1, 2]))
            cin = G * int(rng.integers(1, 3))
            cout = G * int(rng.integers(1, 3))
            # every axis long enough for at least one window (torch raises otherwise)
            size = tuple(max(int(v), d[i] * (k[i] - 1) + 1 - 2 * p[i])
                         for i, v in enumerate(rng.integers(3, 7, nd)))
            cases.append((sd, k, s, p, d, G, cin, cout, size, bool(rng.integers(0, 2))))
    return cases


@pytest.mark.parametrize("case", _case_grid())
def test_conv_matches_torch_float64(case):
    sd, k, s, p, d, G, cin, cout, size, has_bias = case
    rng = np.random.default_rng(zlib.crc32(repr(case).encode()))
    x = rng.standard_normal((2, cin) + size)
    w = rng.standard_normal((cout, cin // G) + k)
    b = rng.standard_normal(cout) if has_bias else None
    y = oracle.conv_forward(x, w, b, stride=s, padding=p, dilation=d, groups=G)
    ref = TORCH_CONV[sd](torch.tensor(x), torch.tensor(w), None if b is None else torch.tensor(b),
                         stride=s, padding=p, dilation=d, groups=G).numpy()
    assert y.shape == ref.shape
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def impulse_expected(w, b, shape_in, pos, stride, padding, dilation, groups, shape_out):
    """Closed form of the response to a unit impulse at pos = (c, t0, h0, w0).

    Output (o, tau, i, j) equals bias[o] + W[o, c - g*Cg, a, u, v] when
    tau*sT + a*dT - pT = t0, i*sH + u*dH - pH = h0, j*sW + v*dW - pW = w0 and o
    is in the group of c; otherwise bias[o].  The tap indices are solved from
    these equations, not summed.
    """
    Cout, Cg, kT, kH, kW = w.shape
    c, t0, h0, w0 = pos
    g = c // Cg
    Og = Cout // groups
    y = np.zeros(shape_out)
    if b is not None:
        y += b[:, None, None, None]
    _, To, Ho, Wo = shape_out

    def tap(out_idx, src, s, p, dd, k):
        num = src + p - out_idx * s
        if num < 0 or num % dd:
            return None
        a = num // dd
        return a if a < k else None

    for o in range(g * Og, (g + 1) * Og):
        for tau, i, j in itertools.product(range(To), range(Ho), range(Wo)):
            a = tap(tau, t0, stride[0], padding[0], dilation[0], kT)
            u = tap(i, h0, stride[1], padding[1], dilation[1], kH)
            v = tap(j, w0, stride[2], padding[2], dilation[2], kW)
            if a is not None and u is not None and v is not None:
                y[o, tau, i, j] += w[o, c - g * Cg, a, u, v]
    return y


def _impulse_case(conv=oracle.conv_forward, mutate_w=None):
    rng = np.random.default_rng(7)
    groups, cin, cout = 2, 4, 6
    k, s, p, d = (3, 3, 2), (2, 1, 1), (2, 1, 0), (1, 2, 1)
    size = (9, 7, 5)
    w = rng.standard_normal((cout, cin // groups) + k)
    b = rng.standard_normal(cout)
    ok = True
    for pos in [(0, 0, 3, 2), (3, 4, 0, 4), (1, 8, 6, 0), (2, 5, 2, 1)]:
        x = np.zeros((1, cin) + size)
        x[(0,) + pos] = 1.0
        wc = w if mutate_w is None else mutate_w(w)
        y = conv(x, wc, b, stride=s, padding=p, dilation=d, groups=groups)[0]
        e = impulse_expected(w, b, size, pos, s, p, d, groups, y.shape)
        ok &= y.shape == e.shape and np.allclose(y, e, rtol=0, atol=1e-12)
    return ok


def test_impulse_response_closed_form():
    assert _impulse_case()


def test_planted_tap_flip_fails_impulse_pin():
    # a temporal tap-order flip (convolution instead of cross-correlation)
    assert not _impulse_case(mutate_w=lambda w: w[:, :, ::-1].copy())


def test_planted_spatial_transpose_fails_impulse_pin():
    assert not _impulse_case(mutate_w=lambda w: np.ascontiguousarray(w[:, :, :, ::-1, :]))


def test_planted_group_mixup_fails_impulse_pin():
    # channels taken from the wrong group: swap the two groups' weights
    def swap(w):
        h = w.shape[0] // 2
        return np.concatenate([w[h:], w[:h]], axis=0)
    assert not _impulse_case(mutate_w=swap)


def _constant_check(y, w, b, kval, interior):
    """Interior outputs of a constant input k equal bias + k * sum(W[o])."""
    expect = (0 if b is None else b) + kval * w.reshape(w.shape[0], -1).sum(1)
    return np.allclose(y[interior], np.broadcast_to(expect[:, None, None, None],
                                                    y.shape)[interior], rtol=1e-12, atol=1e-12)


def test_constant_input_closed_form():
    rng = np.random.default_rng(3)
    w = rng.standard_normal((5, 3, 3, 3, 3))
    b = rng.standard_normal(5)
    x = np.full((1, 3, 7, 8, 8), 2.5)
    y = oracle.conv_forward(x, w, b, padding=(0, 1, 1))[0]
    interior = (slice(None), slice(None), slice(1, -1), slice(1, -1))
    assert _constant_check(y, w, b, 2.5, interior)
    # planted: a dropped bias fails the pin
    y_nobias = oracle.conv_forward(x, w, None, padding=(0, 1, 1))[0]
    assert not _constant_check(y_nobias, w, b, 2.5, interior)


def test_all_ones_kernel_gives_box_sums():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((1, 1, 11, 6, 9))
    k = (4, 2, 3)
    w = np.ones((1, 1) + k)
    y = oracle.conv_forward(x, w)[0, 0]
    # box sums through a 3-D summed-area table
    S = np.zeros(tuple(n + 1 for n in x.shape[2:]))
    S[1:, 1:, 1:] = x[0, 0].cumsum(0).cumsum(1).cumsum(2)
    T, H, W = (n - kk + 1 for n, kk in zip(x.shape[2:], k))
    t, h, ww = np.meshgrid(np.arange(T), np.arange(H), np.arange(W), indexing="ij")
    a, bb, c = k
    box = (S[t + a, h + bb, ww + c] - S[t, h + bb, ww + c] - S[t + a, h, ww + c]
           - S[t + a, h + bb, ww] + S[t, h, ww + c] + S[t, h + bb, ww] + S[t + a, h, ww]
           - S[t, h, ww])
    np.testing.assert_allclose(y, box, rtol=1e-10, atol=1e-10)


def test_linearity():
    rng = np.random.default_rng(11)
    w = rng.standard_normal((4, 2, 3, 2))
    x1 = rng.standard_normal((2, 2, 8, 5))
    x2 = rng.standard_normal((2, 2, 8, 5))
    kw = dict(stride=(2, 1), padding=(1, 1), dilation=(1, 2))
    lhs = oracle.conv_forward(1.5 * x1 - 0.25 * x2, w, None, **kw)
    rhs = 1.5 * oracle.conv_forward(x1, w, None, **kw) - 0.25 * oracle.conv_forward(x2, w, None, **kw)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12, atol=1e-12)


def test_time_shift_equivariance():
    """Delaying the input by sT frames delays the (unpadded) output by one frame."""
    rng = np.random.default_rng(13)
    sT = 2
    w = rng.standard_normal((3, 2, 3, 3))
    b = rng.standard_normal(3)
    x = rng.standard_normal((1, 2, 12, 6))
    y = oracle.conv_forward(x, w, b, stride=(sT, 1), dilation=(2, 1))
    xs = np.concatenate([rng.standard_normal((1, 2, sT, 6)), x], axis=2)
    ys = oracle.conv_forward(xs, w, b, stride=(sT, 1), dilation=(2, 1))
    np.testing.assert_allclose(ys[:, :, 1:], y, rtol=1e-12, atol=1e-12)


def test_empty_output_when_window_does_not_fit():
    w = np.ones((2, 1, 5))
    y = oracle.conv_forward(np.ones((1, 1, 3)), w)
    assert y.shape == (1, 2, 0)
