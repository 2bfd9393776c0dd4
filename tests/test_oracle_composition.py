"""Pins for the oracle's composition pieces: co.Delay (section 3.2), residual
connections (section 3.1.1, Example 3), chains (section 3.3) and the delay
bookkeeping of Principles 6 and 7.

Pins: the Principle 6 worked example's printed values (tests/golden/), the
first non-empty step of stepped chains (counted, not computed from the
formula), shifted inputs (delay closed form) and PyTorch's CPU float64 clip
convolution / pooling for residual and chain outputs.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_chain_delay_worked_example():
    g = golden("principle6_worked_example.json")
    f = [l["receptive_field"] for l in g["layers"]]
    s = [l["stride"] for l in g["layers"]]
    p = [l["padding"] for l in g["layers"]]
    for i in range(len(f)):
        fa, pa, sa, d = oracle.chain_delay(f[:i + 1], s[:i + 1], p[:i + 1])
        assert (fa, pa, sa, d) == (g["f_acc"][i], g["p_acc"][i], g["s_acc"][i], g["d_acc"][i])
    assert oracle.chain_delay(f, s, p)[3] == g["d_NN"]
    assert oracle.chain_delay(f, s, p)[2] == g["s_NN"]


def _first_step(layers, T, cin, rng):
    x = rng.standard_normal((1, cin, T))
    steps = []
    for t in range(T):
        y = x[:, :, t]
        for m in layers:
            y = m.forward_step(y)
            if y is None:
                break
        if y is not None:
            steps.append(t)
    return steps


@pytest.mark.parametrize("seed", range(12))
def test_chain_delay_matches_stepped_chains(seed):
    """The formula against the counted first output and output period of
    random 2-3 layer chains with strides, paddings and dilations."""
    rng = np.random.default_rng(900 + seed)
    n = int(rng.integers(2, 4))
    layers, f, s, p = [], [], [], []
    for _ in range(n):
        k = int(rng.integers(1, 4))
        dil = int(rng.integers(1, 3))
        fr = dil * (k - 1) + 1
        st = int(rng.integers(1, 3))
        pd = int(rng.integers(0, fr))
        w = rng.standard_normal((2, 2, k))
        layers.append(oracle.ContinualConv(w, None, stride=st, padding=pd, dilation=dil))
        f.append(fr)
        s.append(st)
        p.append(pd)
    fa, pa, sa, d = oracle.chain_delay(f, s, p)
    steps = _first_step(layers, d + 4 * sa + 8, 2, rng)
    assert steps[0] == d
    assert all(b - a == sa for a, b in zip(steps, steps[1:]))


def test_delay_fifo_closed_form():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 3, 9, 4))
    for d in (0, 1, 3):
        dl = oracle.ContinualDelay(d)
        outs = [dl.forward_step(x[:, :, t]) for t in range(9)]
        assert all(o is None for o in outs[:d])
        for t in range(d, 9):
            np.testing.assert_array_equal(outs[t], x[:, :, t - d])
        np.testing.assert_array_equal(dl.forward(x), x)
        # update_state=False: the same output, no advance
        n0 = dl.n
        peek = dl.forward_step(x[:, :, 0], update_state=False)
        assert dl.n == n0
        if d == 0:
            np.testing.assert_array_equal(peek, x[:, :, 0])


def _conv3d_np(x, w, b, padding):
    return F.conv3d(torch.tensor(x), torch.tensor(w), torch.tensor(b), padding=padding).numpy()


def test_residual_equal_padding_and_example3_forms():
    """Example 3: a residual block over a k=3 Conv3d with padding 1, written as
    explicit parallel branches (conv, Delay(1)) merged by a sum and as a
    Residual, gives the same steps; both equal conv(x) + x in clip mode
    (delay 1: the first step is empty)."""
    rng = np.random.default_rng(5)
    C = 3
    w = rng.standard_normal((C, C, 3, 3, 3)) * 0.3
    b = rng.standard_normal(C) * 0.1
    x = rng.standard_normal((2, C, 10, 4, 5))

    def conv():
        return oracle.ContinualConv(w, b, padding=(1, 1, 1))

    res1 = oracle.ContinualParallelSum(conv(), oracle.ContinualDelay(1))
    res3 = oracle.ContinualResidual(conv())
    assert res1.delay == res3.delay == 1
    y1, y3 = res1.forward_steps(x), res3.forward_steps(x)
    np.testing.assert_array_equal(y1, y3)
    clip = _conv3d_np(x, w, b, (1, 1, 1)) + x
    np.testing.assert_allclose(y3, clip[:, :, :y3.shape[2]], rtol=1e-12, atol=1e-12)
    assert y3.shape[2] == x.shape[2] - 1
    np.testing.assert_allclose(res3.forward(x), clip, rtol=1e-12, atol=1e-12)


def test_centred_residual_without_padding():
    """Section 3.1.1's centred residual: a k=3 conv without temporal padding
    has delay 2, the input joins delayed by 1 (the window's centre), and the
    clip-mode residual is the input shrunk by one frame at each end."""
    rng = np.random.default_rng(7)
    C = 2
    w = rng.standard_normal((C, C, 3, 1, 1))
    b = rng.standard_normal(C) * 0.1
    x = rng.standard_normal((1, C, 9, 3, 3))
    res = oracle.ContinualResidual(oracle.ContinualConv(w, b, padding=(0, 0, 0)))
    assert res.delay == 2 and res.shrink == 1
    clip = _conv3d_np(x, w, b, (0, 0, 0)) + x[:, :, 1:-1]
    np.testing.assert_allclose(res.forward(x), clip, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(res.forward_steps(x), clip, rtol=1e-12, atol=1e-12)
    # a module with more temporal padding than the centre alignment has no
    # centred residual
    with pytest.raises(ValueError):
        oracle.ContinualResidual(oracle.ContinualConv(rng.standard_normal((C, C, 3)), None,
                                                      padding=2))


def test_x3d_bottleneck_chain():
    """Pointwise conv -> depthwise CoConv3d (3x3x3, temporal padding 1) ->
    average pool over 4 frames (7x7 plane): stepping equals the clip chain of
    PyTorch operations, and the first output comes at the Principle 6 delay
    (f_acc = 1 + 2 + 3 = 6, p_acc = 1, d = 4)."""
    rng = np.random.default_rng(11)
    Ci, C = 3, 4
    w1 = rng.standard_normal((C, Ci, 1, 1, 1))
    w2 = rng.standard_normal((C, 1, 3, 3, 3))
    b2 = rng.standard_normal(C) * 0.1
    x = rng.standard_normal((2, Ci, 12, 7, 7))
    chain = oracle.ContinualChain(
        oracle.ContinualConv(w1, None),
        oracle.ContinualConv(w2, b2, padding=(1, 1, 1), groups=C),
        oracle.ContinualPool("avg", (4, 7, 7), stride=(1, 7, 7)))
    assert oracle.chain_delay([1, 3, 4], [1, 1, 1], [0, 1, 0]) == (6, 1, 1, 4)
    outs = [chain.forward_step(x[:, :, t]) for t in range(12)]
    first = next(i for i, o in enumerate(outs) if o is not None)
    assert first == 4
    z = F.conv3d(torch.tensor(x), torch.tensor(w1))
    z = F.conv3d(z, torch.tensor(w2), torch.tensor(b2), padding=(1, 1, 1), groups=C)
    z = F.avg_pool3d(z, (4, 7, 7), (1, 7, 7)).numpy()
    got = np.stack([o for o in outs if o is not None], axis=2)
    np.testing.assert_allclose(got, z[:, :, :got.shape[2]], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(chain.forward(x), z, rtol=1e-12, atol=1e-12)
