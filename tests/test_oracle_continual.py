"""Pins for the oracle's continual (step-wise) driver.

The paper fixes what step inference must return: Definition 1 (identical
outputs for identical receptive fields), Principle 2 (forward_step /
forward_steps), Principle 3 (state rules), Principle 4 (delay d = f - p - 1),
Principle 5 (stride and prediction rate), Example 1, the captions of Figures 1
and 2 and the Principle 6 worked example (tests/golden/).  The step outputs
are compared with PyTorch's CPU float64 clip convolution / pooling, never with
the oracle's own clip path.
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


def torch_conv1d(x, w, b, s, p, d):
    if x.shape[2] + 2 * p < d * (w.shape[2] - 1) + 1:   # torch raises when nothing fits
        return np.zeros((x.shape[0], w.shape[0], 0))
    return F.conv1d(torch.tensor(x), torch.tensor(w), None if b is None else torch.tensor(b),
                    stride=s, padding=p, dilation=d).numpy()


def n_outputs_without_end_pad(T, f, p, s):
    return (T + p - f) // s + 1 if T + p >= f else 0


GRID = [(k, s, p, d, T)
        for k in (1, 2, 3) for s in (1, 2, 3) for d in (1, 2)
        for p in range(0, d * (k - 1) + 1) for T in (1, 4, 5, 9)]


@pytest.mark.parametrize("k,s,p,d,T", GRID)
def test_steps_equal_clip_forward_I1_I2_I7(k, s, p, d, T):
    rng = np.random.default_rng(k * 1000 + s * 100 + p * 10 + d + T * 7)
    w = rng.standard_normal((3, 2, k))
    b = rng.standard_normal(3)
    x = rng.standard_normal((2, 2, T))
    ref = torch_conv1d(x, w, b, s, p, d)          # symmetric temporal padding p
    f = d * (k - 1) + 1
    co = oracle.ContinualConv(w, b, stride=s, padding=p, dilation=d)
    assert co.receptive_field == f and co.delay == f - p - 1
    # I7: leading empties = delay, then one output every s steps
    flags = []
    for t in range(T):
        flags.append(co.forward_step(x[:, :, t], update_state=False) is not None)
        co.forward_step(x[:, :, t])
    expect_flags = [n >= co.delay and (n - co.delay) % s == 0 for n in range(T)]
    assert flags == expect_flags
    # I1: steps from clean state == the first N1 outputs of forward
    co.clean_state()
    ys = co.forward_steps(x)
    n1 = n_outputs_without_end_pad(T, f, p, s)
    if n1 == 0:
        assert ys is None
    else:
        np.testing.assert_allclose(ys, ref[:, :, :n1], rtol=1e-12, atol=1e-12)
    # I2: with pad_end the step outputs equal forward exactly in count
    co.clean_state()
    ys = co.forward_steps(x, pad_end=True)
    if ref.shape[2] == 0:
        assert ys is None
    else:
        assert ys.shape == ref.shape
        np.testing.assert_allclose(ys, ref, rtol=1e-12, atol=1e-12)


def test_step_equals_window_convolution_I3():
    """Each emitted step equals torch's convolution of that window alone."""
    rng = np.random.default_rng(17)
    w = rng.standard_normal((4, 3, 3, 3, 3))
    b = rng.standard_normal(4)
    x = rng.standard_normal((2, 3, 8, 5, 6))
    co = oracle.ContinualConv(w, b, padding=(1, 1, 0), dilation=(2, 1, 1))
    pT, f = 1, 5
    xp = np.concatenate([np.zeros((2, 3, pT, 5, 6)), x], axis=2)
    for n in range(8):
        y = co.forward_step(x[:, :, n])
        if n < co.delay:
            assert y is None
            continue
        win = xp[:, :, n + pT - f + 1:n + pT + 1]
        ref = F.conv3d(torch.tensor(win), torch.tensor(w), torch.tensor(b),
                       padding=(0, 1, 0), dilation=(2, 1, 1)).numpy()[:, :, 0]
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_forward_steps_is_concatenated_forward_step_I4():
    rng = np.random.default_rng(19)
    w = rng.standard_normal((2, 2, 3, 2))
    x = rng.standard_normal((1, 2, 11, 4))
    a = oracle.ContinualConv(w, None, stride=(2, 1), padding=(1, 0))
    bb = oracle.ContinualConv(w, None, stride=(2, 1), padding=(1, 0))
    ys = a.forward_steps(x)
    outs = [bb.forward_step(x[:, :, t]) for t in range(11)]
    np.testing.assert_array_equal(ys, np.stack([o for o in outs if o is not None], axis=2))


def test_update_state_false_leaves_state_I5():
    rng = np.random.default_rng(23)
    w = rng.standard_normal((2, 1, 3))
    co = oracle.ContinualConv(w, None)
    x = rng.standard_normal((1, 1, 6))
    for t in range(4):
        co.forward_step(x[:, :, t])
    frames_before = {k: v.copy() for k, v in co.frames.items()}
    n_before = co.n
    y_peek = co.forward_step(x[:, :, 4], update_state=False)
    assert co.n == n_before and set(co.frames) == set(frames_before)
    for k in frames_before:
        np.testing.assert_array_equal(co.frames[k], frames_before[k])
    y_real = co.forward_step(x[:, :, 4])
    np.testing.assert_array_equal(y_peek, y_real)
    # forward_steps with update_state=False as well
    co2 = oracle.ContinualConv(w, None)
    co2.forward_steps(x[:, :, :3])
    n2 = co2.n
    co2.forward_steps(x[:, :, 3:], update_state=False)
    assert co2.n == n2


def test_clean_state_replay_identical_I6():
    rng = np.random.default_rng(29)
    w = rng.standard_normal((3, 2, 2, 3))
    x = rng.standard_normal((2, 2, 7, 5))
    co = oracle.ContinualConv(w, None, padding=(1, 1))
    y1 = co.forward_steps(x)
    co.clean_state()
    y2 = co.forward_steps(x)
    np.testing.assert_array_equal(y1, y2)


def test_example1_conv3d_forward_modes():
    """Example 1: co.Conv3d(4, 8, 3) -- delay 2, receptive field 3, forward equals
    the regular convolution, steps over the first 4 frames give the first
    ``delay`` outputs and one more step gives output ``delay``."""
    g = golden("example1.json")
    rng = np.random.default_rng(31)
    cin, cout, k = g["in_channels"], g["out_channels"], g["kernel_size"]
    w = rng.standard_normal((cout, cin, k, k, k))
    b = rng.standard_normal(cout)
    x = rng.standard_normal(tuple(g["x_shape"]))
    co = oracle.ContinualConv(w, b)
    assert co.delay == g["delay"] and co.receptive_field == g["receptive_field"]
    y = co.forward(x)
    z = F.conv3d(torch.tensor(x), torch.tensor(w), torch.tensor(b)).numpy()
    assert list(z.shape) == [2, 8, 3, 4, 5]
    np.testing.assert_allclose(y, z, rtol=1e-12, atol=1e-12)
    firsts = co.forward_steps(x[:, :, :g["steps_first_call"]])
    assert firsts.shape[2] == g["outputs_first_call"]
    np.testing.assert_allclose(firsts, z[:, :, :co.delay], rtol=1e-12, atol=1e-12)
    last = co.forward_step(x[:, :, g["forward_step_frame"]])
    np.testing.assert_allclose(last, z[:, :, g["forward_step_output_index"]], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", golden("figures.json")["cases"])
def test_figure_delays(case):
    f, p = case["receptive_field"], case["padding"]
    w = np.ones((1, 1, f))
    co = oracle.ContinualConv(w, None, padding=p)
    assert co.delay == case["delay"]
    outs = [co.forward_step(np.ones((1, 1))) for _ in range(6)]
    lead = next(i for i, o in enumerate(outs) if o is not None)
    assert lead == case["leading_empty_outputs"]


def _chain_step(layers, x_t):
    """Principle 7: an empty value entering a layer gives an empty output."""
    for layer in layers:
        if x_t is None:
            return None
        x_t = layer.forward_step(x_t)
    return x_t


def test_principle6_worked_example_two_layer_chain():
    g = golden("principle6_worked_example.json")
    rng = np.random.default_rng(37)
    l1, l2 = g["layers"]
    w1 = rng.standard_normal((2, 2, l1["receptive_field"]))
    w2 = rng.standard_normal((2, 2, l2["receptive_field"]))
    c1 = oracle.ContinualConv(w1, None, stride=l1["stride"], padding=l1["padding"])
    c2 = oracle.ContinualConv(w2, None, stride=l2["stride"], padding=l2["padding"])
    assert [c1.delay, c2.delay] == [g["d_acc"][0], 2]
    T = 15
    x = rng.standard_normal((1, 2, T))
    outs = [_chain_step([c1, c2], x[:, :, t]) for t in range(T)]
    steps = [t for t, o in enumerate(outs) if o is not None]
    # network delay d_NN: first non-empty output at step d_NN
    assert steps[0] == g["d_NN"]
    # prediction rate r_NN = 1 / s_NN: one output every s_NN steps
    assert all(b - a == g["s_NN"] for a, b in zip(steps, steps[1:]))
    assert len(steps) / (T - steps[0]) == pytest.approx(g["r_NN"], abs=0.1)
    # values: equal to the clip-mode chain without end padding
    z = torch_conv1d(torch_conv1d(x, w1, None, l1["stride"], l1["padding"], 1), w2, None,
                     l2["stride"], l2["padding"], 1)
    got = np.stack([outs[t] for t in steps], axis=2)
    np.testing.assert_allclose(got, z[:, :, :got.shape[2]], rtol=1e-12, atol=1e-12)
    # accumulated receptive field: the number of (virtual) input positions the
    # first network output depends on, padded ones included, is f_acc = 7
    dep = []
    for t in range(T):
        xp = x.copy()
        xp[:, :, t] += 1.0
        c1.clean_state()
        c2.clean_state()
        o = [_chain_step([c1, c2], xp[:, :, u]) for u in range(T)][steps[0]]
        if not np.allclose(o, outs[steps[0]]):
            dep.append(t)
    p_acc = g["p_acc"][1]
    assert dep[-1] - (-p_acc) + 1 == g["f_acc"][1]
    assert dep[-1] == g["d_NN"]


def test_depthwise_conv_then_pool_chain_delay():
    """Depthwise conv (k=3, p=0) followed by an average pool over 4 frames
    (stride 1): f_acc = 4 + (3 - 1) * 1 = 6, so the chain's delay is 5."""
    rng = np.random.default_rng(41)
    C = 3
    w = rng.standard_normal((C, 1, 3, 3, 3))
    conv = oracle.ContinualConv(w, None, padding=(0, 1, 1), groups=C)
    pool = oracle.ContinualPool("avg", (4, 3, 3), stride=(1, 3, 3))
    x = rng.standard_normal((2, C, 12, 3, 3))
    outs = [_chain_step([conv, pool], x[:, :, t]) for t in range(12)]
    first = next(i for i, o in enumerate(outs) if o is not None)
    assert first == 5
    zc = F.conv3d(torch.tensor(x), torch.tensor(w), padding=(0, 1, 1), groups=C)
    zp = F.avg_pool3d(zc, (4, 3, 3), (1, 3, 3)).numpy()
    got = np.stack([o for o in outs if o is not None], axis=2)
    np.testing.assert_allclose(got, zp, rtol=1e-12, atol=1e-12)


POOL_GRID = [(kind, k, s, p, d, cip, T)
             for kind in ("avg", "max") for k in (1, 2, 3, 4) for s in (1, 2)
             for d in ((1,) if kind == "avg" else (1, 2)) for p in range(0, k // 2 + 1)
             for cip in ((True, False) if kind == "avg" else (True,)) for T in (7, 10)]


@pytest.mark.parametrize("kind,k,s,p,d,cip,T", POOL_GRID)
def test_continual_pool_equals_clip_pool(kind, k, s, p, d, cip, T):
    rng = np.random.default_rng(k * 100 + s * 10 + p + T + d * 1000 + int(cip) * 5)
    x = rng.standard_normal((2, 3, T, 5, 4))
    co = oracle.ContinualPool(kind, (k, 3, 2), stride=(s, 2, 1), padding=(p, 1, 0),
                              dilation=(d, 1, 1), count_include_pad=cip)
    xt = torch.tensor(x)
    if kind == "avg":
        ref = F.avg_pool3d(xt, (k, 3, 2), (s, 2, 1), (p, 1, 0), count_include_pad=cip).numpy()
    else:
        ref = F.max_pool3d(xt, (k, 3, 2), (s, 2, 1), (p, 1, 0), (d, 1, 1)).numpy()
    ys = co.forward_steps(x, pad_end=True)
    if ref.shape[2] == 0:
        assert ys is None
    else:
        assert ys.shape == ref.shape
        np.testing.assert_allclose(ys, ref, rtol=1e-12, atol=1e-12)
    co.clean_state()
    ys = co.forward_steps(x)
    n1 = n_outputs_without_end_pad(T, d * (k - 1) + 1, p, s)
    if n1:
        np.testing.assert_allclose(ys, ref[:, :, :n1], rtol=1e-12, atol=1e-12)
    else:
        assert ys is None


def test_negative_delay_rejected():
    with pytest.raises(ValueError):
        oracle.ContinualConv(np.ones((1, 1, 3)), None, padding=3)
