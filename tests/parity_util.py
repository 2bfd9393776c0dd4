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


# Elementwise bound |g - o| <= atol + rtol |o| next to the normwise one.
#  rtol: the unit roundoff of the output dtype (the result is rounded once
#        to it: 2^-8 for bfloat16, 2^-24 for float32);
#  atol: the float32 accumulation of `terms` values per output -- products
#        of the io-dtype inputs (exact for bfloat16, rounded once for
#        float32), partial sums and the bias -- bounded by
#        terms^1.5 * 2^-24 * rms(o): a recursive sum of K terms errs by at
#        most about K u sum|a_i|, and sum|a_i| ~ sqrt(K) rms(o) for terms of
#        random sign; plus `extra_atol` where an intermediate was rounded to
#        the io dtype (a chain of layers).
U32 = 2.0 ** -24
UNIT_ROUNDOFF = {torch.float32: 2.0 ** -24, torch.bfloat16: 2.0 ** -8}


def conv_terms(w, bias=True):
    """Values a convolution output accumulates: C_in/groups * kT * kH * kW
    products, plus the bias."""
    n = 1
    for s in tuple(w.shape)[1:]:
        n *= int(s)
    return n + (1 if bias else 0)


def window_terms(kernel):
    """Values a pooled output reduces: the window volume."""
    n = 1
    for k in kernel:
        n *= int(k)
    return n


def elementwise_excess(got, ref, dtype, terms, extra_atol=0.0):
    """(largest |g - o| / bound, its flat index, |g - o|, bound) over the
    elements, with the bound above."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    # the accumulation error is rounded along with the result: (1 + rtol) atol
    rtol = UNIT_ROUNDOFF[dtype]
    atol = (extra_atol + float(terms) ** 1.5 * U32 * rms) * (1.0 + rtol)
    bound = atol + rtol * np.abs(ref)
    err = np.abs(got - ref)
    ratio = np.where(bound > 0, err / np.where(bound > 0, bound, 1.0),
                     np.where(err > 0, np.inf, 0.0))
    i = int(np.argmax(ratio)) if ratio.size else 0
    if not ratio.size:
        return 0.0, 0, 0.0, 0.0
    return float(ratio.flat[i]), i, float(err.flat[i]), float(bound.flat[i])


def assert_close(got, ref, dtype, what="", *, terms, extra_atol=0.0):
    """Normwise error within TOL[dtype], and every element within the
    elementwise bound; logs the worst element."""
    e = relerr(got, ref)
    assert e <= TOL[dtype], f"{what}: normwise rel err {e:.3e} > {TOL[dtype]:.0e}"
    r, i, err, bound = elementwise_excess(got, ref, dtype, terms, extra_atol)
    say(f"{what}: normwise {e:.2e}; worst element #{i}: |g-o| {err:.3e} of bound {bound:.3e} "
        f"({r:.3f} of it; {terms} terms)")
    assert r <= 1.0, (f"{what}: element {i} off by {err:.3e}, above the elementwise bound "
                      f"{bound:.3e}")
    return e


def chain_atol(intermediate, terms, dtype=torch.bfloat16, gain=1.0):
    """Extra absolute error of a layer fed by an intermediate that was
    accumulated from `terms` values and rounded to `dtype`: each of its values
    is off by at most the unit roundoff of itself plus its own accumulation
    error, and a layer whose weights sum to at most `gain` in magnitude
    (1 for an average or a maximum) passes on at most `gain` times the
    largest of those errors."""
    a = np.abs(np.asarray(intermediate, dtype=np.float64))
    if not a.size:
        return 0.0
    rms = float(np.sqrt(np.mean(a * a)))
    return gain * (UNIT_ROUNDOFF[dtype] * float(a.max()) + float(terms) ** 1.5 * U32 * rms)


def say(*a):
    """Name the case before each GPU step (flushed, so a fault still shows it)."""
    print(*a, flush=True)
    sys.stdout.flush()


def oracle_conv(w, b, stride, padding, dilation, groups):
    return oracle.ContinualConv(np64(w), None if b is None else np64(b), stride=stride,
                                padding=padding, dilation=dilation, groups=groups)
