"""Helpers shared by the GPU parity tests: conversions, the error measure and
oracle runs on the same seeded inputs the GPU consumes."""
import sys

import numpy as np
import torch

import oracle

# fp32: normwise max relative error 1e-5; bf16 in, fp32 accumulate: 2e-2
TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}


def np64(t):
    return t.detach().float().cpu().double().numpy()


def relerr(got, ref):
    """Normwise error: largest absolute error over the largest |oracle| value."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    scale = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (scale if scale > 0 else 1.0))


def assert_close(got, ref, dtype, what=""):
    e = relerr(got, ref)
    assert e <= TOL[dtype], f"{what}: normwise rel err {e:.3e} > {TOL[dtype]:.0e}"
    return e


def say(*a):
    """Name the case before each GPU step (flushed, so a fault still shows it)."""
    print(*a, flush=True)
    sys.stdout.flush()


def oracle_conv(w, b, stride, padding, dilation, groups):
    return oracle.ContinualConv(np64(w), None if b is None else np64(b), stride=stride,
                                padding=padding, dilation=dilation, groups=groups)
