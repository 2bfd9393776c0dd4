"""Pins for the oracle's ordinary pooling (nn.AvgPoolNd / nn.MaxPoolNd forward).

Pins: PyTorch's CPU float64 pooling, constant inputs, increasing ramps (the
maximum is the newest frame of the window) and the identity "average pool =
depthwise convolution with uniform weights", checked against the
independently pinned convolution oracle.
"""
import zlib

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

AVG = {0: F.avg_pool1d, 1: F.avg_pool2d, 2: F.avg_pool3d}
MAX = {0: F.max_pool1d, 1: F.max_pool2d, 2: F.max_pool3d}


def _grid():
    rng = np.random.default_rng(99)
    out = []
    for sd in (0, 1, 2):
        for kind in ("avg", "max"):
            for _ in range(8):
                nd = sd + 1
                k = tuple(int(v) for v in rng.integers(1, 4, nd))
                s = tuple(int(v) for v in rng.integers(1, 3, nd))
                d = tuple(int(v) for v in rng.integers(1, 3, nd)) if kind == "max" else (1,) * nd
                p = tuple(int(rng.integers(0, k[i] // 2 + 1)) for i in range(nd))
                cip = bool(rng.integers(0, 2))
                size = tuple(int(v) for v in rng.integers(4, 8, nd))
                out.append((sd, kind, k, s, p, d, cip, size))
    return out


@pytest.mark.parametrize("case", _grid())
def test_pool_matches_torch_float64(case):
    sd, kind, k, s, p, d, cip, size = case
    rng = np.random.default_rng(zlib.crc32(repr(case).encode()))
    x = rng.standard_normal((2, 3) + size)
    y = oracle.pool_forward(kind, x, k, s, p, d, cip)
    xt = torch.tensor(x)
    if kind == "avg":
        ref = AVG[sd](xt, k, s, p, count_include_pad=cip).numpy()
    else:
        ref = MAX[sd](xt, k, s, p, d).numpy()
    assert y.shape == ref.shape
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_constant_input_pools_to_constant():
    x = np.full((1, 2, 6, 5, 5), -1.75)
    for kind in ("avg", "max"):
        y = oracle.pool_forward(kind, x, (3, 2, 2), (1, 1, 1), 0)
        np.testing.assert_allclose(y, -1.75, rtol=0, atol=1e-14)


def test_max_of_increasing_ramp_is_newest_frame():
    T = 9
    x = np.arange(T, dtype=np.float64)[None, None, :, None, None] * np.ones((1, 1, T, 3, 3))
    y = oracle.pool_forward("max", x, (4, 3, 3), (1, 1, 1), 0)
    np.testing.assert_array_equal(y[0, 0, :, 0, 0], np.arange(3, T))


def test_avg_pool_equals_uniform_depthwise_conv():
    rng = np.random.default_rng(21)
    C, k = 3, (2, 3, 3)
    x = rng.standard_normal((2, C, 7, 6, 6))
    y = oracle.pool_forward("avg", x, k, (1, 2, 2), (0, 1, 1), 1, True)
    w = np.full((C, 1) + k, 1.0 / np.prod(k))
    yc = oracle.conv_forward(x, w, None, stride=(1, 2, 2), padding=(0, 1, 1), groups=C)
    np.testing.assert_allclose(y, yc, rtol=1e-12, atol=1e-12)
