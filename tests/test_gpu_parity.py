"""GPU parity: the HIP path (through the C ABI) against the oracle.

Every case draws seeded inputs once on the host, feeds the identical values
to the oracle (float64) and to the GPU, and compares element by element with
the normwise bound of parity_util.TOL.  Sizes span several thread blocks and
leave ragged tails; edge cases cover kT = 1, delay 0, all-empty streams,
strides, dilations, groups, end padding and both dtypes.
"""
import itertools
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_2204_03418_amd import synth
from parity_util import (TOL, assert_close, chain_atol, conv_terms, np64, oracle_conv, relerr,
                         say, window_terms)

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2204_03418_amd import coinf
DEV = "cuda"


def _fuzz_cases():
    rng = np.random.default_rng(2204)
    out = []
    for idx in range(36):
        sd = idx % 3
        nd = sd + 1
        k = tuple(int(v) for v in rng.integers(1, 4, nd))
        s = (int(rng.integers(1, 3)),) + tuple(int(v) for v in rng.integers(1, 3, sd))
        dil = tuple(int(v) for v in rng.integers(1, 3, nd))
        p = tuple(int(rng.integers(0, dil[i] * (k[i] - 1) + 1)) for i in range(nd))
        G = int(rng.choice([1, 1, 2, 3]))
        cin = G * int(rng.integers(1, 4))
        cout = G * int(rng.integers(1, 6))
        size = tuple(max(int(v), dil[i + 1] * (k[i + 1] - 1) + 1)
                     for i, v in enumerate(rng.integers(3, 12, sd)))
        B = int(rng.integers(1, 4))
        T = int(rng.integers(1, 13))
        dt = "bf16" if idx % 4 == 3 else "f32"
        out.append((idx, B, cin, cout, G, k, s, p, dil, size, T, dt))
    return out


@pytest.mark.parametrize("case", _fuzz_cases(), ids=lambda c: f"fuzz{c[0]}")
def test_fuzz_conv_steps_and_clip(case):
    idx, B, cin, cout, G, k, s, p, dil, size, T, dt = case
    say("fuzz", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=k, in_size=size,
                          stride=s, padding=p, dilation=dil, groups=G, dtype=dt)
    x, w, b = synth.conv_inputs(spec, T, 50000 + 10 * idx, "normal")
    tdt = synth.torch_dtype(dt)
    for algo in ("direct", "auto"):
        co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=s, padding=p,
                          dilation=dil, groups=G, algo=algo)
        ref = oracle_conv(w, b, s, p, dil, G)
        ys = co.forward_steps(x.to(DEV), pad_end=True)
        r = ref.forward_steps(np64(x), pad_end=True)
        if r is None:
            assert ys is None
        else:
            assert_close(np64(ys), r, tdt, f"steps {algo}", terms=conv_terms(w))
        clip = co.forward(x.to(DEV))
        rc = oracle.conv_forward(np64(x), np64(w), np64(b), s, p, dil, G)
        assert tuple(clip.shape) == rc.shape
        if rc.size:
            assert_close(np64(clip), rc, tdt, f"clip {algo}", terms=conv_terms(w))


def _run_steps(co, x):
    """forward_step per frame (the benchmark's launch configuration)."""
    outs = []
    for t in range(x.shape[2]):
        y = co.forward_step(x[:, :, t].contiguous())
        if y is not None:
            outs.append(y.clone())
    return outs


@pytest.mark.parametrize("name", ["conv1d_b1_c4to8_k3_f32", "conv3d_b1_c24_k3_56x56_f32"])
def test_workload_full_clip(name):
    """Whole clip, every output element, forward_step per frame."""
    wl = synth.WORKLOADS[name]
    c = wl.conv
    say("workload", name)
    x, w, b = synth.workload_inputs(name)
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=c.batch, in_size=c.in_size, stride=c.stride,
                      padding=c.padding, dilation=c.dilation, groups=c.groups)
    outs = _run_steps(co, x.to(DEV))
    torch.cuda.synchronize()
    ref = oracle_conv(w, b, c.stride, c.padding, c.dilation, c.groups).forward_steps(np64(x))
    got = np.stack([np64(o) for o in outs], axis=2)
    assert_close(got, ref, synth.torch_dtype(c.dtype), name, terms=conv_terms(w))


@pytest.mark.parametrize("name,streams,frames", [
    ("conv3d_b64_c192_k3_14x14_bf16", (0, 37, 63), 8),
    ("conv2d_b32_c64to256_k9x1_v25_f32", (0, 31), 300),
    ("conv2d_b32_c64to256_k9x1_v25_bf16", (5, 17), 300),
])
def test_workload_sampled_streams(name, streams, frames):
    """Full-size run on the GPU; the oracle recomputes sampled streams (the B
    streams are independent, one shared clock) over the first `frames` frames."""
    wl = synth.WORKLOADS[name]
    c = wl.conv
    say("workload", name, "streams", streams, "frames", frames)
    x, w, b = synth.workload_inputs(name)
    x = x[:, :, :frames].contiguous()
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=c.batch, in_size=c.in_size, stride=c.stride,
                      padding=c.padding, dilation=c.dilation, groups=c.groups)
    outs = _run_steps(co, x.to(DEV))
    torch.cuda.synchronize()
    sel = list(streams)
    got = np.stack([np64(o[sel]) for o in outs], axis=2)
    ref = oracle_conv(w, b, c.stride, c.padding, c.dilation, c.groups).forward_steps(np64(x[sel]))
    assert_close(got, ref, synth.torch_dtype(c.dtype), name, terms=conv_terms(w))


def test_workload_depthwise_then_pool():
    name = "dwconv3d_b16_c432_k3_7x7_avgpool_bf16"
    wl = synth.WORKLOADS[name]
    c, pl = wl.conv, wl.pool
    say("workload", name)
    x, w, b = synth.workload_inputs(name)
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=c.batch, in_size=c.in_size, padding=c.padding,
                      groups=c.groups)
    assert co.algo == "depthwise"
    po = coinf.CoPool("avg", batch=pl.batch, channels=pl.channels, kernel=pl.kernel,
                      in_size=pl.in_size, stride=pl.stride, dtype=torch.bfloat16)
    assert co.delay + po.delay == 5
    xd = x.to(DEV)
    conv_outs, pool_outs = [], []
    for t in range(x.shape[2]):
        y = co.forward_step(xd[:, :, t].contiguous())
        if y is None:
            continue
        conv_outs.append(y.clone())
        z = po.forward_step(y)
        if z is not None:
            pool_outs.append(z.clone())
    torch.cuda.synchronize()
    ref_c = oracle_conv(w, b, c.stride, c.padding, c.dilation, c.groups).forward_steps(np64(x))
    got_c = np.stack([np64(o) for o in conv_outs], axis=2)
    assert_close(got_c, ref_c, torch.bfloat16, "depthwise conv", terms=conv_terms(w))
    # the pool oracle chains on the oracle's own (float64) conv outputs; the
    # GPU pool sees the bf16-rounded conv outputs, within the bf16 bound
    rp = oracle.ContinualPool("avg", pl.kernel, pl.stride).forward_steps(ref_c)
    got_p = np.stack([np64(o) for o in pool_outs], axis=2)
    assert got_p.shape == rp.shape
    assert_close(got_p, rp, torch.bfloat16, "avg pool", terms=window_terms(pl.kernel),
                 extra_atol=chain_atol(ref_c, conv_terms(w), torch.bfloat16))
    # the chain's output count: T - 5 frames after a delay of 5
    assert got_p.shape[2] == x.shape[2] - 5


def _pool_cases():
    out = []
    for i, (kind, k, s, p, d, cip, sd) in enumerate(itertools.product(
            ("avg", "max"), (1, 3, 4), (1, 2), (0, 1), (1, 2), (True, False), (0, 1, 2))):
        if kind == "avg" and d == 2:
            continue
        if kind == "max" and not cip:
            continue
        if p > k // 2:
            continue
        out.append((i, kind, k, s, p, d, cip, sd))
    return out


@pytest.mark.parametrize("case", _pool_cases(), ids=lambda c: f"pool{c[0]}")
def test_pool_fuzz(case):
    i, kind, k, s, p, d, cip, sd = case
    say("pool", case)
    size = {0: (), 1: (9,), 2: (7, 6)}[sd]
    ks = (k,) + ((3, 2) if sd == 2 else (3,) if sd == 1 else ())
    ss = (s,) + ((2, 1) if sd == 2 else (2,) if sd == 1 else ())
    ps = (p,) + ((1, 0) if sd == 2 else (1,) if sd == 1 else ())
    ds = (d,) + ((1, 2) if (sd == 2 and kind == "max") else (1,) * sd)
    dt = torch.bfloat16 if i % 3 == 0 else torch.float32
    x = synth.normal((3, 5, 11) + size, 7000 + i, dtype="bf16" if dt == torch.bfloat16 else "f32")
    po = coinf.CoPool(kind, batch=3, channels=5, kernel=ks, in_size=size, stride=ss, padding=ps,
                      dilation=ds, count_include_pad=cip, dtype=dt)
    ys = po.forward_steps(x.to(DEV), pad_end=True)
    r = oracle.ContinualPool(kind, ks, ss, ps, ds, cip, spatial_dims=sd).forward_steps(
        np64(x), pad_end=True)
    assert_close(np64(ys), r, dt, "pool steps", terms=window_terms(ks))
    clip = po.forward(x.to(DEV))
    rc = oracle.pool_forward(kind, np64(x), ks, ss, ps, ds, cip)
    assert_close(np64(clip), rc, dt, "pool clip", terms=window_terms(ks))


def _small_conv(algo="auto", dtype="f32", **kw):
    spec = synth.ConvSpec(batch=2, in_channels=6, out_channels=10, kernel=(3, 3, 3),
                          in_size=(9, 11), padding=kw.get("padding", (1, 1, 1)), dtype=dtype)
    x, w, b = synth.conv_inputs(spec, 12, 90000, "normal")
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=2, in_size=(9, 11), padding=spec.padding,
                      algo=algo)
    return co, x.to(DEV), w, b, spec


def test_update_state_false_leaves_state_bitwise():
    say("update_state=False")
    co, x, *_ = _small_conv()
    for t in range(5):
        co.forward_step(x[:, :, t].contiguous())
    torch.cuda.synchronize()
    before = co.state.clone()
    n = co.steps
    peek = co.forward_step(x[:, :, 5].contiguous(), update_state=False)
    torch.cuda.synchronize()
    assert co.steps == n
    assert torch.equal(co.state, before)
    real = co.forward_step(x[:, :, 5].contiguous())
    assert torch.equal(peek, real)
    # forward_steps with update_state=False: same outputs, state restored
    torch.cuda.synchronize()
    before = co.state.clone()
    n = co.steps
    a = co.forward_steps(x[:, :, 6:].contiguous(), update_state=False)
    torch.cuda.synchronize()
    assert co.steps == n and torch.equal(co.state, before)
    bb = co.forward_steps(x[:, :, 6:].contiguous())
    assert torch.equal(a, bb)


def test_clean_state_replay_and_determinism():
    say("clean_state replay")
    co, x, *_ = _small_conv()
    y1 = co.forward_steps(x).clone()
    co.clean_state()
    assert co.steps == 0
    y2 = co.forward_steps(x).clone()
    assert torch.equal(y1, y2)


def test_snapshot_attach_resume_bitwise():
    say("snapshot/attach")
    co, x, w, b, spec = _small_conv()
    T = x.shape[2]
    co.forward_steps(x[:, :, :5].contiguous())
    snap = co.state.clone()
    n = co.steps
    rest = co.forward_steps(x[:, :, 5:].contiguous()).clone()
    del co
    co2 = coinf.CoConv(w.to(DEV), b.to(DEV), batch=2, in_size=(9, 11), padding=spec.padding,
                       state=snap, attach_steps=n)
    assert co2.steps == n
    rest2 = co2.forward_steps(x[:, :, 5:T].contiguous())
    assert torch.equal(rest, rest2)


def test_attach_rejects_foreign_state():
    say("attach mismatch")
    co, x, w, b, spec = _small_conv()
    torch.cuda.synchronize()
    with pytest.raises(coinf.CoinfError) as e:
        coinf.CoConv(w.to(DEV), b.to(DEV), batch=2, in_size=(9, 11), padding=(0, 1, 1),
                     state=co.state, attach_steps=0)
    assert e.value.status == coinf.CO_ESTATE


@pytest.mark.parametrize("k,p,s,dil", [(1, 0, 1, 1), (3, 2, 1, 1), (4, 0, 3, 2), (2, 1, 2, 3),
                                       (5, 3, 1, 2)])
def test_temporal_edge_cases(k, p, s, dil):
    """kT = 1 (no ring), delay 0, stride > kT with dilation, end padding."""
    say("edge", k, p, s, dil)
    spec = synth.ConvSpec(batch=3, in_channels=5, out_channels=7, kernel=(k, 3), in_size=(13,),
                          stride=(s, 1), padding=(p, 1), dilation=(dil, 1))
    x, w, b = synth.conv_inputs(spec, 17, 31000 + k * 100 + p * 10 + s, "normal")
    ref = oracle_conv(w, b, spec.stride, spec.padding, spec.dilation, 1)
    for algo in ("direct", "auto"):
        co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=3, in_size=(13,), stride=spec.stride,
                          padding=spec.padding, dilation=spec.dilation, algo=algo)
        ref.clean_state()
        r = ref.forward_steps(np64(x), pad_end=True)
        ys = co.forward_steps(x.to(DEV), pad_end=True)
        assert_close(np64(ys), r, torch.float32, f"edge {algo}", terms=conv_terms(w))


def test_all_empty_and_zero_length():
    say("all empty")
    spec = synth.ConvSpec(batch=1, in_channels=2, out_channels=3, kernel=(5,), dtype="f32")
    x, w, b = synth.conv_inputs(spec, 3, 123, "normal")
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=1)
    assert co.forward_steps(x.to(DEV)) is None          # 3 frames < delay 4
    assert co.steps == 3
    assert co.forward_steps(x[:, :, :0].contiguous().to(DEV)) is None
    assert co.steps == 3
    y = co.forward_step(x[:, :, 0].contiguous().to(DEV))
    assert y is None                                     # step 3 < delay 4
    y = co.forward_step(x[:, :, 1].contiguous().to(DEV))  # step 4 emits
    assert y is not None


GEMM_CASES = [
    # B, Cin, Cout, kT, (kH, kW), in_size, (pH, pW), sT, pT, dT, dtype
    (3, 40, 24, 3, (3, 3), (9, 11), (1, 1), 1, 0, 1, "bf16"),    # 2 channel chunks, ragged
    (2, 20, 36, 2, (3, 3), (7, 6), (0, 1), 1, 1, 1, "f32"),      # valid rows, ragged N
    (5, 64, 48, 4, (1,), (25,), (0,), 1, 0, 1, "f32"),           # (kT, 1) over joints
    (5, 64, 48, 4, (1,), (25,), (0,), 1, 2, 1, "bf16"),
    (20, 8, 16, 3, (3, 3), (4, 4), (1, 1), 1, 0, 1, "bf16"),     # many streams per tile
    (2, 33, 40, 3, (3, 3), (10, 9), (1, 1), 2, 1, 2, "f32"),     # temporal stride + dilation
    (1, 24, 24, 3, (3, 3), (56, 56), (1, 1), 1, 0, 1, "f32"),    # the 56x56 stem block
    (4, 96, 80, 5, (3, 3), (14, 14), (1, 1), 1, 2, 1, "bf16"),
    (3, 16, 16, 1, (3, 3), (8, 8), (1, 1), 1, 0, 1, "f32"),      # kT = 1: no ring
]


GEMM_WS_CASES = [
    # B, Cin, Cout, kT, (kH, kW), in_size, (pH, pW), sT, pT, dT, dtype -- the
    # warp-specialized configuration: bf16, 3x3, Ho*Wo a multiple of 4
    (3, 40, 24, 3, (3, 3), (8, 10), (1, 1), 1, 0, 1, "bf16"),    # ragged chunk and column tile
    (2, 32, 64, 2, (3, 3), (12, 9), (1, 1), 1, 1, 1, "bf16"),    # odd width: single-pixel loads
    (4, 64, 32, 3, (3, 3), (10, 10), (0, 0), 1, 0, 1, "bf16"),   # valid convolution, pH = 0
    (20, 16, 48, 3, (3, 3), (6, 6), (1, 1), 1, 2, 1, "bf16"),    # many images per tile, ragged tile
    (2, 33, 40, 3, (3, 3), (10, 8), (1, 1), 2, 1, 2, "bf16"),    # temporal stride and dilation
    (3, 24, 16, 1, (3, 3), (8, 8), (1, 1), 1, 0, 1, "bf16"),     # kT = 1: no ring
    (64, 96, 96, 3, (3, 3), (14, 14), (1, 1), 1, 0, 1, "bf16"),  # the 64-stream shape, fewer channels
]


@pytest.mark.parametrize("case", GEMM_WS_CASES, ids=lambda c: "ws_" + "_".join(map(str, c[:4])))
def test_gemm_ws_forced(case):
    """The warp-specialized GEMM step (producer waves stage the input,
    consumer waves stream the weights) against the oracle, stepping with
    update_state=False peeks, and forward_steps with end padding."""
    B, cin, cout, kT, ks, size, ps, sT, pT, dT, dt = case
    say("gemm ws", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=(kT,) + ks,
                          in_size=size, stride=(sT,) + (1,) * len(size),
                          padding=(pT,) + ps, dilation=(dT,) + (1,) * len(size), dtype=dt)
    x, w, b = synth.conv_inputs(spec, 9, 63000 + cin * 7 + cout, "kaiming")
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=spec.stride,
                      padding=spec.padding, dilation=spec.dilation, algo="gemm_ws")
    assert co.algo == "gemm_ws_bf16"
    ref = oracle_conv(w, b, spec.stride, spec.padding, spec.dilation, 1)
    xd = x.to(DEV)
    tdt = synth.torch_dtype(dt)
    outs, peeks = [], []
    for t in range(x.shape[2]):
        fr = xd[:, :, t].contiguous()
        pk = co.forward_step(fr, update_state=False)
        if pk is not None:
            peeks.append(pk.clone())
        y = co.forward_step(fr)
        if y is not None:
            outs.append(y.clone())
    r = ref.forward_steps(np64(x))
    if r is None:
        assert not outs
    else:
        got = np.stack([np64(o) for o in outs], axis=2)
        assert_close(got, r, tdt, "gemm_ws steps", terms=conv_terms(w))
        assert len(peeks) == len(outs)
        for a, bb in zip(peeks, outs):
            assert torch.equal(a, bb)
    co.clean_state()
    ref.clean_state()
    ys = co.forward_steps(xd, pad_end=True)
    rp = ref.forward_steps(np64(x), pad_end=True)
    if rp is None:
        assert ys is None
    else:
        assert_close(np64(ys), rp, tdt, "gemm_ws steps pad_end", terms=conv_terms(w))


@pytest.mark.parametrize("case", GEMM_CASES, ids=lambda c: "gemm_" + "_".join(map(str, c[:4])) + c[-1])
def test_gemm_forced(case):
    B, cin, cout, kT, ks, size, ps, sT, pT, dT, dt = case
    say("gemm", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=(kT,) + ks,
                          in_size=size, stride=(sT,) + (1,) * len(size),
                          padding=(pT,) + ps, dilation=(dT,) + (1,) * len(size), dtype=dt)
    x, w, b = synth.conv_inputs(spec, 11, 61000 + cin * 7 + cout, "kaiming")
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=spec.stride,
                      padding=spec.padding, dilation=spec.dilation, algo="gemm")
    assert co.algo.startswith("gemm")
    ref = oracle_conv(w, b, spec.stride, spec.padding, spec.dilation, 1)
    xd = x.to(DEV)
    tdt = synth.torch_dtype(dt)
    # steps through forward_step (with update_state=False peeks in between)
    outs, peeks = [], []
    for t in range(x.shape[2]):
        fr = xd[:, :, t].contiguous()
        pk = co.forward_step(fr, update_state=False)
        if pk is not None:
            peeks.append(pk.clone())
        y = co.forward_step(fr)
        if y is not None:
            outs.append(y.clone())
    r = ref.forward_steps(np64(x))
    if r is None:
        assert not outs
        return
    got = np.stack([np64(o) for o in outs], axis=2)
    assert_close(got, r, tdt, "gemm steps", terms=conv_terms(w))
    assert len(peeks) == len(outs)
    for a, bb in zip(peeks, outs):
        assert torch.equal(a, bb)
    # forward_steps with end padding from a clean state
    co.clean_state()
    ref.clean_state()
    ys = co.forward_steps(xd, pad_end=True)
    assert_close(np64(ys), ref.forward_steps(np64(x), pad_end=True), tdt, "gemm steps pad_end",
                 terms=conv_terms(w))


REG_CASES = [
    # B, Cin, Cout, kernel (time first), in_size, stride, padding, dilation, dtype
    (1, 24, 24, (3, 3, 3), (56, 56), (1, 1, 1), (0, 1, 1), (1, 1, 1), "f32"),   # 56x56 stem block
    (3, 7, 20, (2, 3, 3), (9, 11), (1, 1, 1), (1, 1, 1), (1, 1, 1), "f32"),     # ragged C and M
    (2, 10, 33, (3, 3, 2), (8, 7), (2, 2, 1), (2, 1, 0), (2, 1, 2), "f32"),     # strides, dilation
    (5, 64, 48, (4, 1), (25,), (1, 1), (0, 0), (1, 1), "f32"),                  # (kT, 1) over joints
    (5, 64, 48, (4, 1), (25,), (1, 1), (2, 0), (1, 1), "bf16"),
    (2, 40, 24, (3, 1, 3), (9, 11), (1, 1, 1), (0, 0, 1), (1, 1, 1), "bf16"),   # ragged channel block
    (4, 16, 16, (1, 3, 3), (8, 8), (1, 1, 1), (0, 1, 1), (1, 1, 1), "f32"),     # kT = 1: no ring
    (3, 5, 17, (3,), (), (1,), (0,), (1,), "f32"),                              # Conv1d, M = B
    (2, 100, 32, (2, 1, 1), (6, 5), (1, 1, 1), (1, 0, 0), (1, 1, 1), "bf16"),   # 4 channel blocks
    (3, 12, 40, (5, 3, 3), (7, 9), (2, 2, 2), (3, 1, 1), (1, 2, 1), "bf16"),    # stride 2 everywhere
    (8, 24, 24, (2, 3, 3), (28, 28), (1, 1, 1), (1, 1, 1), (1, 1, 1), "f32"),   # enough tiles: no split
]


@pytest.mark.parametrize("case", REG_CASES, ids=lambda c: "reg_" + "_".join(map(str, c[:3])) + c[-1])
def test_gemm_reg_forced(case):
    """Register-operand GEMM step (forced) against the oracle: forward_step with
    update_state=False peeks, then forward_steps with end padding."""
    B, cin, cout, k, size, s, p, dil, dt = case
    say("gemm_reg", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=k, in_size=size,
                          stride=s, padding=p, dilation=dil, dtype=dt)
    x, w, b = synth.conv_inputs(spec, 13, 71000 + cin * 7 + cout, "kaiming")
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=s, padding=p,
                      dilation=dil, algo="gemm_reg")
    assert co.algo.startswith("gemm_reg")
    ref = oracle_conv(w, b, s, p, dil, 1)
    xd = x.to(DEV)
    tdt = synth.torch_dtype(dt)
    outs, peeks = [], []
    for t in range(x.shape[2]):
        fr = xd[:, :, t].contiguous()
        pk = co.forward_step(fr, update_state=False)
        if pk is not None:
            peeks.append(pk.clone())
        y = co.forward_step(fr)
        if y is not None:
            outs.append(y.clone())
    r = ref.forward_steps(np64(x))
    if r is None:
        assert not outs
    else:
        got = np.stack([np64(o) for o in outs], axis=2)
        assert_close(got, r, tdt, "gemm_reg steps", terms=conv_terms(w))
        assert len(peeks) == len(outs)
        for a, bb in zip(peeks, outs):
            assert torch.equal(a, bb)
    co.clean_state()
    ref.clean_state()
    ys = co.forward_steps(xd, pad_end=True)
    rp = ref.forward_steps(np64(x), pad_end=True)
    if rp is None:
        assert ys is None
    else:
        assert_close(np64(ys), rp, tdt, "gemm_reg steps pad_end", terms=conv_terms(w))


DW_STEPS_CASES = [
    # B, C, kT, (kH, kW), in_size, (pT, pH, pW), dtype
    (3, 20, 3, (3, 3), (7, 7), (0, 1, 1), "bf16"),    # the X3D-style block, small
    (2, 12, 1, (3, 3), (6, 5), (0, 1, 1), "f32"),     # kT = 1: no ring
    (2, 9, 2, (3, 3), (5, 8), (1, 0, 1), "f32"),      # delay 0, valid rows
    (4, 16, 4, (1, 1), (3, 3), (3, 0, 0), "bf16"),    # pointwise taps, full padding
    (1, 33, 5, (3, 3), (9, 4), (2, 1, 1), "f32"),     # ragged, kT = 5
    (1, 3, 3, (3, 3), (5, 5), (1, 1, 1), "bf16"),     # clip bytes not a multiple of 16
    (2, 8, 3, (3, 3), (10, 9), (1, 1, 1), "bf16"),    # 90 output pixels: thread per output
    (2, 10, 3, (3, 3), (8, 8), (1, 1, 1), "bf16", (2, 2), (1, 1)),  # spatial stride 2
    (2, 7, 3, (3, 3), (7, 7), (0, 2, 2), "f32", (1, 1), (2, 2)),    # dilation 2: 11 x 11 tile
    (2, 6, 2, (3, 3), (8, 8), (0, 2, 2), "bf16", (1, 1), (2, 2)),   # 12 x 12 tile: thread per output
    (1, 5, 3, (3, 3), (6, 6), (2, 1, 1), "bf16", (1, 2), (1, 1)),   # stride in one axis only
    # temporal stride / dilation (plan-driven kernel): ..., sT, dT
    (2, 8, 3, (3, 3), (7, 7), (1, 1, 1), "bf16", (1, 1), (1, 1), 2, 1),  # temporal stride 2
    (2, 6, 3, (3, 3), (6, 6), (2, 1, 1), "f32", (1, 1), (1, 1), 1, 2),   # temporal dilation 2
    (1, 5, 5, (3, 3), (5, 5), (4, 0, 0), "bf16", (1, 1), (1, 1), 3, 1),  # stride 3, kT 5
    (2, 4, 2, (1, 1), (4, 4), (0, 0, 0), "f32", (1, 1), (1, 1), 2, 3),   # 1x1, stride 2, dilation 3
    (2, 9, 3, (3, 3), (7, 7), (1, 1, 1), "bf16", (1, 1), (1, 1), 2, 2),  # stride and dilation 2
]


@pytest.mark.parametrize("case", DW_STEPS_CASES, ids=lambda c: "dwsteps_" + "_".join(map(str, c[:3])) + (
    f"_s{c[9]}d{c[10]}" if len(c) > 9 else ""))
def test_depthwise_forward_steps_persistent(case):
    """The depthwise forward_steps runs as one persistent launch (partial sums
    in registers across frames).  Against the oracle with end padding, and
    bitwise against the per-frame step kernel (same arithmetic order), also
    when a clip continues a state left by single steps, after clean_state
    (stale ring contents) and with update_state=False."""
    B, C, kT, ks, size, p, dt = case[:7]
    st = (case[9] if len(case) > 9 else 1,) + (case[7] if len(case) > 7 else (1, 1))
    dil = (case[10] if len(case) > 10 else 1,) + (case[8] if len(case) > 8 else (1, 1))
    say("depthwise steps", case)
    spec = synth.ConvSpec(batch=B, in_channels=C, out_channels=C, kernel=(kT,) + ks, in_size=size,
                          stride=st, padding=p, dilation=dil, groups=C, dtype=dt)
    x, w, b = synth.conv_inputs(spec, 14, 91000 + 13 * C + kT, "kaiming")
    tdt = synth.torch_dtype(dt)
    xd = x.to(DEV)

    def make():
        return coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=st, padding=p,
                            dilation=dil, groups=C)

    co = make()
    assert co.algo == "depthwise" and co.steps_fused(x.shape[2])
    ref = oracle_conv(w, b, st, p, dil, C)
    ys = co.forward_steps(xd, pad_end=True)
    rp = ref.forward_steps(np64(x), pad_end=True)
    assert_close(np64(ys), rp, tdt, "persistent depthwise steps", terms=conv_terms(w))
    # bitwise against single steps
    co2 = make()
    outs = [co2.forward_step(xd[:, :, t].contiguous()) for t in range(x.shape[2])]
    outs = [o.clone() for o in outs if o is not None]
    co.clean_state()
    ys2 = co.forward_steps(xd)                      # after clean_state: stale ring contents
    if outs:
        assert torch.equal(ys2, torch.stack(outs, dim=2))
    # a clip that continues single steps, and single steps after a clip
    co3, co4 = make(), make()
    heads = [co3.forward_step(xd[:, :, t].contiguous()) for t in range(3)]
    mid = co3.forward_steps(xd[:, :, 3:9].contiguous())
    tail = [co3.forward_step(xd[:, :, t].contiguous()) for t in range(9, x.shape[2])]
    seq = [co4.forward_step(xd[:, :, t].contiguous()) for t in range(x.shape[2])]
    seq = [s_.clone() for s_ in seq if s_ is not None]
    got = ([mid[:, :, k] for k in range(mid.shape[2])] if mid is not None else []) + \
        [t_ for t_ in tail if t_ is not None]
    n_first = sum(1 for h_ in heads if h_ is not None)  # (a temporal stride skips steps)
    assert len(got) == len(seq) - n_first
    for g_, s_ in zip(got, seq[n_first:]):
        assert torch.equal(g_, s_)
    # update_state=False: same outputs, state bitwise unchanged
    torch.cuda.synchronize()
    before, n = co3.state.clone(), co3.steps
    peek = co3.forward_steps(xd[:, :, 2:10].contiguous(), update_state=False)
    torch.cuda.synchronize()
    assert co3.steps == n and torch.equal(co3.state, before)
    real = co3.forward_steps(xd[:, :, 2:10].contiguous())
    assert torch.equal(peek, real)


def _check_fused_steps(make, x, ref, tdt, what):
    """forward_steps as one persistent launch: against the oracle with end
    padding; bitwise against per-frame forward_step (same per-tap arithmetic
    order), also after clean_state (stale ring contents); a clip from the
    stream's start followed by single steps (the partial sums the clip
    leaves are those stepping leaves), a clip continuing a state left by
    single steps and single steps continuing a clip; and update_state=False
    (same outputs, state unchanged)."""
    xd = x.to(DEV)
    T = x.shape[2]
    co = make()
    assert co.steps_fused(T, pad_end=True), (what, co.algo)
    ys = co.forward_steps(xd, pad_end=True)
    rp = ref.forward_steps(np64(x), pad_end=True)
    assert_close(np64(ys), rp, tdt, what, terms=conv_terms(co.weight, co.bias is not None))
    co2 = make()
    outs = [co2.forward_step(xd[:, :, t].contiguous()) for t in range(T)]
    outs = [o.clone() for o in outs if o is not None]
    co.clean_state()
    ys2 = co.forward_steps(xd)
    if outs:
        assert torch.equal(ys2, torch.stack(outs, dim=2)), what
    co5 = make()
    head = co5.forward_steps(xd[:, :, :T - 5].contiguous())
    rest = [co5.forward_step(xd[:, :, t].contiguous()) for t in range(T - 5, T)]
    got = ([head[:, :, i] for i in range(head.shape[2])] if head is not None else []) + \
        [r_ for r_ in rest if r_ is not None]
    assert len(got) == len(outs), what
    for g_, s_ in zip(got, outs):
        assert torch.equal(g_, s_), what
    co3, co4 = make(), make()
    heads = [co3.forward_step(xd[:, :, t].contiguous()) for t in range(3)]
    mid = co3.forward_steps(xd[:, :, 3:9].contiguous())
    tail = [co3.forward_step(xd[:, :, t].contiguous()) for t in range(9, T)]
    seq = [co4.forward_step(xd[:, :, t].contiguous()) for t in range(T)]
    seq = [s_.clone() for s_ in seq if s_ is not None]
    got = ([mid[:, :, k] for k in range(mid.shape[2])] if mid is not None else []) + \
        [t_ for t_ in tail if t_ is not None]
    n_first = sum(1 for h_ in heads if h_ is not None)  # (a temporal stride skips steps)
    assert len(got) == len(seq) - n_first
    for g_, s_ in zip(got, seq[n_first:]):
        assert torch.equal(g_, s_), what
    torch.cuda.synchronize()
    before, n = co3.state.clone(), co3.steps
    peek = co3.forward_steps(xd[:, :, 2:10].contiguous(), update_state=False)
    torch.cuda.synchronize()
    assert co3.steps == n and torch.equal(co3.state, before), what
    real = co3.forward_steps(xd[:, :, 2:10].contiguous())
    assert (peek is None and real is None) or torch.equal(peek, real), what


REG_STEPS_CASES = [
    # B, C_in, C_out, kernel (time first), in_size, padding, dtype, frames
    (1, 24, 24, (3, 3, 3), (20, 20), (0, 1, 1), "f32", 12),   # 3x3, two waves per tile
    (2, 20, 32, (3, 3, 3), (40, 40), (1, 1, 1), "f32", 12),   # 3x3, one wave per tile
    (4, 12, 32, (3, 3, 3), (40, 40), (1, 1, 1), "f32", 12),   # 3x3, two columns per wave
    (4, 32, 32, (3, 3, 3), (40, 40), (2, 1, 1), "bf16", 12),  # bf16 3x3
    (3, 40, 20, (3, 1), (13,), (1, 0), "f32", 14),            # 1x1 spatial, small
    (32, 96, 128, (9, 1), (25,), (4, 0), "bf16", 14),         # deep temporal kernel, bf16
    (64, 64, 256, (5, 1), (25,), (2, 0), "bf16", 12),         # kT = 5 on the 9-tap shape (runtime kT)
    (64, 64, 256, (3, 1), (25,), (1, 0), "bf16", 12),         # 3-tap shape, eight staging waves
    (2, 7, 17, (1, 3, 3), (6, 9), (0, 1, 1), "f32", 12),      # kT = 1: no ring
]


@pytest.mark.parametrize("case", REG_STEPS_CASES, ids=lambda c: "regsteps_" + "_".join(
    map(str, c[:3])) + "_" + c[6])
def test_reg_forward_steps_persistent(case):
    """The register-GEMM forward_steps as one persistent launch (partial sums
    in accumulator registers across frames)."""
    B, cin, cout, k, size, p, dt, T = case
    say("reg steps", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=k, in_size=size,
                          padding=p, dtype=dt)
    x, w, b = synth.conv_inputs(spec, T, 93000 + 7 * cin + cout, "kaiming")
    tdt = synth.torch_dtype(dt)

    def make():
        return coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, padding=p)

    assert make().algo.startswith("gemm_reg")
    ones = (1,) * len(k)
    _check_fused_steps(make, x, oracle_conv(w, b, ones, p, ones, 1), tdt, "reg steps")


REG_STRIDED_CASES = [
    # B, C_in, C_out, kernel (time first), in_size, padding, dtype, frames, sT, dT
    # (sizes chosen so that the picker lands on the staged 1x1 shapes)
    (3, 40, 20, (3, 1), (13,), (1, 0), "f32", 14, 2, 1),             # temporal stride 2
    (32, 96, 128, (9, 1), (25,), (4, 0), "bf16", 14, 2, 1),          # skeleton-style, kT = 9
    (32, 64, 256, (3, 1), (25,), (2, 0), "bf16", 13, 1, 2),          # temporal dilation 2
    (2, 40, 32, (3, 1), (9,), (0, 0), "f32", 15, 3, 2),              # stride 3, dilation 2
    (2, 100, 72, (2, 1), (11,), (1, 0), "f32", 12, 2, 3),            # 32-channel-block shape
    (3, 40, 20, (3, 1), (13,), (1, 0), "f32", 64, 2, 1),             # long clip: time segments
    (32, 64, 256, (3, 1), (25,), (1, 0), "bf16", 64, 2, 1),          # segments, bf16
]


@pytest.mark.parametrize("case", REG_STRIDED_CASES, ids=lambda c: "regstrided_" + "_".join(
    map(str, c[:3])) + f"_{c[6]}_T{c[7]}_s{c[8]}d{c[9]}")
def test_reg_forward_steps_strided(case):
    """Temporal stride or dilation above 1 on the register GEMM's 1x1
    spatial shapes: forward_steps as one plan-driven persistent launch
    (partial sums in LDS slots, the host's step plans); the long clip is
    split into time segments, so the clip-then-steps check covers the last
    segment's write-back of the ring."""
    B, cin, cout, k, size, p, dt, T, sT, dT = case
    st = (sT,) + (1,) * (len(k) - 1)
    dil = (dT,) + (1,) * (len(k) - 1)
    say("reg strided steps", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=k, in_size=size,
                          stride=st, padding=p, dilation=dil, dtype=dt)
    x, w, b = synth.conv_inputs(spec, T, 98000 + 3 * cin + cout + T, "kaiming")

    def make():
        return coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=st, padding=p,
                            dilation=dil, algo="gemm_reg")

    assert make().algo.startswith("gemm_reg")
    _check_fused_steps(make, x, oracle_conv(w, b, st, p, dil, 1), synth.torch_dtype(dt),
                       "reg strided steps")


DIRECT_STEPS_CASES = [
    # B, C_in, C_out, groups, kernel (time first), in_size, stride, padding, dilation, dtype
    (1, 4, 8, 1, (3,), (), (1,), (0,), (1,), "f32"),                       # 1-D, no spatial axes
    (2, 6, 9, 3, (2, 3), (7,), (1, 1), (1, 1), (1, 1), "bf16"),            # grouped
    (3, 4, 4, 2, (4, 2, 2), (5, 6), (1, 1, 1), (3, 0, 1), (1, 1, 1), "f32"),  # kT = 4, delay 0
    (2, 16, 5, 1, (1, 1, 1), (4, 4), (1, 1, 1), (0, 0, 0), (1, 1, 1), "f32"),  # 16 positions, kT = 1
    (2, 1, 4, 1, (3, 3, 3), (9, 8), (1, 2, 1), (1, 1, 0), (1, 1, 2), "f32"),  # spatial stride, dilation
    # temporal stride / dilation (plan-driven form)
    (1, 4, 8, 1, (3,), (), (2,), (1,), (1,), "f32"),                       # 1-D, stride 2
    (2, 6, 9, 3, (2, 3), (7,), (1, 1), (1, 1), (2, 1), "bf16"),            # grouped, dilation 2
    (3, 4, 4, 2, (4, 2, 2), (5, 6), (3, 1, 1), (3, 0, 1), (1, 1, 1), "f32"),  # stride 3, kT = 4
    (2, 16, 5, 1, (3, 1, 1), (4, 4), (2, 1, 1), (2, 0, 0), (2, 1, 1), "f32"),  # stride and dilation 2
]


@pytest.mark.parametrize("case", DIRECT_STEPS_CASES, ids=lambda c: "dirsteps_" + "_".join(
    map(str, c[:4])) + "_" + c[9] + f"_s{c[6][0]}d{c[8][0]}")
def test_direct_forward_steps_persistent(case):
    """The direct family's forward_steps as one persistent launch (small
    layers: weights, partial sums and prefetched inputs in registers)."""
    B, cin, cout, G, k, size, st, p, dil, dt = case
    say("direct steps", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=k, in_size=size,
                          stride=st, padding=p, dilation=dil, groups=G, dtype=dt)
    x, w, b = synth.conv_inputs(spec, 13, 95000 + 11 * cin + cout, "normal")
    tdt = synth.torch_dtype(dt)

    def make():
        return coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=st, padding=p,
                            dilation=dil, groups=G, algo="direct")

    assert make().algo == "direct"
    _check_fused_steps(make, x, oracle_conv(w, b, st, p, dil, G), tdt, "direct steps")


GEMM_STEPS_CASES = [
    # B, C_in, C_out, kernel (time first), in_size, padding
    (3, 40, 80, (3, 3, 3), (9, 10), (1, 1, 1)),   # ragged channel chunk and channel tile
    (2, 32, 64, (2, 3, 3), (7, 7), (0, 1, 1)),    # odd width (single-pixel staging), kT = 2
    (4, 64, 48, (1, 1, 1), (6, 8), (0, 0, 0)),    # 1x1, kT = 1
    (2, 96, 64, (3, 1, 1), (5, 6), (2, 0, 0)),    # 1x1 spatial, delay 0
    (5, 32, 64, (3, 3, 3), (14, 14), (0, 1, 1)),  # tiles spanning streams
]


@pytest.mark.parametrize("case", GEMM_STEPS_CASES, ids=lambda c: "gemmsteps_" + "_".join(
    map(str, c[:3])) + f"_k{c[3][0]}")
def test_gemm_forward_steps_persistent(case):
    """The LDS-tiled GEMM's forward_steps as one persistent launch (bf16):
    a workgroup owns pixels x output channels x every temporal tap, the
    partial sums stay in its registers across frames."""
    B, cin, cout, k, size, p = case
    say("gemm steps", case)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=k, in_size=size,
                          padding=p, dtype="bf16")
    x, w, b = synth.conv_inputs(spec, 12, 97000 + 5 * cin + cout, "kaiming")

    def make():
        return coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, padding=p, algo="gemm")

    assert make().algo == "gemm_bf16"
    _check_fused_steps(make, x, oracle_conv(w, b, (1, 1, 1), p, (1, 1, 1), 1), torch.bfloat16,
                       "gemm steps")


REG_SEG_CASES = [
    # B, C_in, C_out, kernel (time first), in_size, padding, frames, dtype, oracle streams
    (32, 64, 256, (9, 1), (25,), (0, 0), 100, "bf16", (0, 31)),        # skeleton layer: 2 segments
    (1, 24, 24, (3, 3, 3), (28, 28), (0, 1, 1), 40, "f32", (0,)),      # 3x3 taps: 5 segments
    (2, 20, 36, (3, 3, 3), (14, 15), (2, 1, 1), 33, "f32", (1,)),      # start padding, ragged
]


@pytest.mark.parametrize("case", REG_SEG_CASES, ids=lambda c: f"regseg_{c[0]}_{c[1]}_{c[2]}_T{c[6]}")
def test_reg_forward_steps_time_segments(case):
    """The persistent register GEMM over a clip long enough to be split into
    time segments (each after the first replays kT - 1 frames and stores
    from its own first frame): against the oracle with end padding on
    sampled streams, bitwise against stepping on all, as a clip that
    continues single steps, and with update_state=False."""
    B, cin, cout, k, size, p, T, dt, sel = case
    say("reg segments", case)
    tdt = synth.torch_dtype(dt)
    spec = synth.ConvSpec(batch=B, in_channels=cin, out_channels=cout, kernel=k, in_size=size,
                          padding=p, dtype=dt)
    x, w, b = synth.conv_inputs(spec, T, 99000 + cin + cout + T, "kaiming")
    xd = x.to(DEV)

    def make():
        return coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, padding=p,
                            algo="gemm_reg")

    co = make()
    assert co.algo.startswith("gemm_reg") and co.steps_fused(T, pad_end=True)
    ones = (1,) * len(k)
    ys = co.forward_steps(xd, pad_end=True)
    sl = list(sel)
    rp = oracle_conv(w, b, ones, p, ones, 1).forward_steps(np64(x[sl]), pad_end=True)
    assert_close(np64(ys[sl]), rp, tdt, "reg segments", terms=conv_terms(w))
    # bitwise: the clip, stepping, and a clip between single steps
    seq = _run_steps(make(), xd)
    co.clean_state()
    assert torch.equal(co.forward_steps(xd), torch.stack(seq, dim=2))
    co3 = make()
    for t in range(3):
        co3.forward_step(xd[:, :, t].contiguous())
    mid = co3.forward_steps(xd[:, :, 3:T - 5].contiguous())
    tail = [co3.forward_step(xd[:, :, t].contiguous()) for t in range(T - 5, T)]
    got = [mid[:, :, i] for i in range(mid.shape[2])] + [t_ for t_ in tail if t_ is not None]
    n_first = sum(1 for t in range(3) if t >= co3.delay)
    assert len(got) == len(seq) - n_first
    for g_, s_ in zip(got, seq[n_first:]):
        assert torch.equal(g_, s_)
    # update_state=False: same outputs, state unchanged
    torch.cuda.synchronize()
    before, n = co3.state.clone(), co3.steps
    peek = co3.forward_steps(xd, update_state=False)
    torch.cuda.synchronize()
    assert co3.steps == n and torch.equal(co3.state, before)
    assert torch.equal(peek, co3.forward_steps(xd))


@pytest.mark.parametrize("name,streams", [
    ("conv3d_b64_c192_k3_14x14_bf16", (0, 37, 63)),
    ("dwconv3d_b16_c432_k3_7x7_avgpool_bf16", (0, 9, 15)),
    ("conv1d_b1_c4to8_k3_f32", None),
    ("conv3d_b1_c24_k3_56x56_f32", None),
    ("conv2d_b32_c64to256_k9x1_v25_f32", (0, 13, 31)),
    ("conv2d_b32_c64to256_k9x1_v25_bf16", (2, 29)),
])
def test_workload_forward_steps_fused(name, streams):
    """Full-size forward_steps as one launch over the workload's clip: the
    oracle recomputes every stream or sampled ones; bitwise against the
    per-frame step kernel."""
    wl = synth.WORKLOADS[name]
    c = wl.conv
    say("workload forward_steps", name)
    x, w, b = synth.workload_inputs(name)
    x = x[:, :, :40].contiguous()
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=c.batch, in_size=c.in_size, stride=c.stride,
                      padding=c.padding, dilation=c.dilation, groups=c.groups)
    assert co.steps_fused(x.shape[2])
    xd = x.to(DEV)
    ys = co.forward_steps(xd)
    co2 = coinf.CoConv(w.to(DEV), b.to(DEV), batch=c.batch, in_size=c.in_size, stride=c.stride,
                       padding=c.padding, dilation=c.dilation, groups=c.groups)
    outs = _run_steps(co2, xd)
    assert torch.equal(ys, torch.stack(outs, dim=2))
    sel = list(streams) if streams else list(range(c.batch))
    ref = oracle_conv(w, b, c.stride, c.padding, c.dilation, c.groups).forward_steps(np64(x[sel]))
    assert_close(np64(ys[sel]), ref, synth.torch_dtype(c.dtype), name, terms=conv_terms(w))


POOL_STEPS_CASES = [
    # kind, kernel (time first), in_size, stride, padding, count_include_pad, dtype
    ("avg", (4, 7, 7), (7, 7), (1, 7, 7), (0, 0, 0), True, "bf16"),   # the X3D-style pool
    ("avg", (3, 3, 2), (7, 6), (1, 2, 1), (1, 1, 0), False, "f32"),
    ("max", (5, 3, 3), (6, 5), (1, 1, 1), (2, 1, 1), True, "f32"),
    ("max", (1, 2, 2), (4, 4), (1, 2, 2), (0, 0, 0), True, "bf16"),
    # global spatial pools (frames in lanes), clips over several 32-frame blocks
    ("avg", (4, 7, 7), (7, 7), (1, 7, 7), (0, 0, 0), False, "bf16", 75),
    ("max", (3, 6, 6), (6, 6), (1, 1, 1), (1, 0, 0), True, "f32", 40),
    ("avg", (2, 5, 5), (5, 5), (1, 5, 5), (0, 0, 0), True, "bf16", 33),
    ("avg", (5, 8, 8), (8, 8), (1, 1, 1), (2, 0, 0), False, "f32", 70),
    ("max", (4, 7, 7), (7, 7), (1, 7, 7), (0, 0, 0), True, "bf16", 64),
    # temporal stride / dilation on the global pool: ..., frames, temporal dilation
    ("avg", (3, 7, 7), (7, 7), (2, 7, 7), (0, 0, 0), True, "bf16", 40, 1),
    ("avg", (4, 6, 6), (6, 6), (3, 1, 1), (2, 0, 0), False, "f32", 45, 1),
    ("max", (3, 5, 5), (5, 5), (1, 5, 5), (1, 0, 0), True, "bf16", 50, 3),
    ("max", (2, 7, 7), (7, 7), (2, 7, 7), (0, 0, 0), True, "bf16", 70, 4),
    # temporal stride on the lane-group pool (windows smaller than the frame)
    ("max", (3, 3, 3), (8, 8), (2, 2, 2), (1, 1, 1), True, "bf16", 21, 1),
    ("avg", (2, 3, 2), (7, 6), (3, 2, 1), (1, 1, 0), False, "f32", 26, 1),
    ("avg", (5, 2, 2), (4, 4), (2, 2, 2), (2, 0, 0), True, "bf16", 30, 1),
]


@pytest.mark.parametrize("case", POOL_STEPS_CASES, ids=lambda c: "poolsteps_" + c[0] + str(c[1][0]) + (
    f"_T{c[7]}" if len(c) > 7 else "") + (f"_s{c[3][0]}d{c[8]}" if len(c) > 8 else ""))
def test_pool_forward_steps_persistent(case):
    """Pool forward_steps as one persistent launch against the oracle (end
    padding), bitwise against per-frame steps, continuing a state left by
    single steps, and with update_state=False."""
    kind, ks, size, ss, ps, cip, dt = case[:7]
    T = case[7] if len(case) > 7 else 12
    dil = (case[8] if len(case) > 8 else 1, 1, 1)
    say("pool steps", case)
    tdt = synth.torch_dtype(dt)
    x = synth.normal((3, 6, T) + size, 7700 + ks[0] + T, dtype=dt)
    xd = x.to(DEV)

    def make():
        return coinf.CoPool(kind, batch=3, channels=6, kernel=ks, in_size=size, stride=ss,
                            padding=ps, dilation=dil, count_include_pad=cip, dtype=tdt)

    po = make()
    assert po.steps_fused(T)
    ys = po.forward_steps(xd, pad_end=True)
    r = oracle.ContinualPool(kind, ks, ss, ps, dil, cip, spatial_dims=2).forward_steps(
        np64(x), pad_end=True)
    assert_close(np64(ys), r, tdt, "persistent pool steps", terms=window_terms(ks))
    po2, po3 = make(), make()
    seq = [po2.forward_step(xd[:, :, t].contiguous()) for t in range(x.shape[2])]
    seq = [s_.clone() for s_ in seq if s_ is not None]
    heads = [po3.forward_step(xd[:, :, t].contiguous()) for t in range(2)]
    mid = po3.forward_steps(xd[:, :, 2:8].contiguous())
    tail = [po3.forward_step(xd[:, :, t].contiguous()) for t in range(8, x.shape[2])]
    got = ([mid[:, :, k] for k in range(mid.shape[2])] if mid is not None else []) + \
        [t_ for t_ in tail if t_ is not None]
    n_first = sum(1 for h_ in heads if h_ is not None)  # (a temporal stride skips steps)
    assert len(got) == len(seq) - n_first
    for g_, s_ in zip(got, seq[n_first:]):
        assert torch.equal(g_, s_)
    torch.cuda.synchronize()
    before, n = po3.state.clone(), po3.steps
    peek = po3.forward_steps(xd[:, :, 1:9].contiguous(), pad_end=True, update_state=False)
    torch.cuda.synchronize()
    assert po3.steps == n and torch.equal(po3.state, before)
    real = po3.forward_steps(xd[:, :, 1:9].contiguous(), pad_end=True)
    assert torch.equal(peek, real)


# what, B, C, (H, W), dtype, frames: (B*C - 1) planes of T*H*W elements reach past 2^31 bytes
LARGE_CLIP_CASES = [
    ("depthwise", 2, 32, (64, 64), "f32", 2100),
    ("avgpool", 2, 32, (64, 64), "f32", 2100),
    ("gemm", 2, 32, (64, 64), "f32", 2100),
    ("gemm_reg", 2, 24, (64, 64), "f32", 2800),
    ("gemm_ws", 8, 32, (14, 14), "bf16", 21504),
]


@pytest.mark.parametrize("case", LARGE_CLIP_CASES, ids=lambda c: c[0])
def test_forward_steps_clip_beyond_32bit_offsets(case):
    """forward_steps over a clip of more than 2^31 bytes: the persistent kernels
    decline it and the per-frame loop must still address every plane (the
    depthwise step hands such frames to the 64-bit direct kernel; the pool loop
    and the GEMM-family steps work from a contiguous copy of each frame, the
    GEMM family also emitting into a contiguous frame that is copied out).  The
    clip repeats a 7-frame seeded block, so the oracle recomputes sampled output
    frames from 3-frame windows."""
    what, B, C, (H, W), dt, T = case
    esz, P = (2 if dt == "bf16" else 4), 7
    assert (B * C - 1) * T * H * W * esz + H * W * esz >= 2 ** 31
    say("large clip", what, (B, C, T, H, W), dt)
    tdt = synth.torch_dtype(dt)
    base = synth.normal((B, C, P, H, W), 9100, dtype=dt)
    if what == "avgpool":
        mod = coinf.CoPool("avg", batch=B, channels=C, kernel=(3, 3, 3), in_size=(H, W),
                           stride=1, dtype=tdt)
    else:
        groups = C if what == "depthwise" else 1
        w = synth.normal((C, C // groups, 3, 3, 3), 9101, std=0.2 / (C // groups) ** 0.5,
                         dtype=dt)
        b = synth.normal((C,), 9102, dtype=dt)
        mod = coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=(H, W), padding=(0, 1, 1),
                           groups=groups, algo="auto" if what == "depthwise" else what)
        assert mod.algo.startswith(what)
    assert mod.delay == 2 and not mod.steps_fused(T)
    x = base.to(DEV).repeat(1, 1, T // P, 1, 1)
    y = mod.forward_steps(x)
    torch.cuda.synchronize()
    del x
    assert y.shape[2] == T - 2
    for k in (0, 1234, T - 3):
        win = np64(base[:, :, [(k + j) % P for j in range(3)]])
        if what == "avgpool":
            ref = oracle.pool_window("avg", win, np.ones(3, np.uint8), (3, 3, 3), (1, 1, 1),
                                     (0, 0), (1, 1, 1), True)
        else:
            ref = oracle.conv_window(win, np.ones(3, np.uint8), np64(w), np64(b), groups, 1,
                                     (1, 1), (1, 1), (1, 1, 1))
        assert_close(np64(y[:, :, k:k + 1]), ref, tdt, f"{what} frame {k}",
                     terms=27 if what == "avgpool" else conv_terms(w))


@pytest.mark.parametrize("algo,dt", [("gemm", "bf16"), ("gemm", "f32"), ("gemm_ws", "bf16")])
def test_misaligned_frame_is_staged(algo, dt):
    """A frame that starts one element past an aligned address: the GEMM-family
    step stages it into an aligned copy and still matches the oracle."""
    say("misaligned frame", algo, dt)
    spec = synth.ConvSpec(batch=2, in_channels=16, out_channels=24, kernel=(3, 3, 3),
                          in_size=(8, 8), padding=(1, 1, 1), dtype=dt)
    x, w, b = synth.conv_inputs(spec, 6, 9200, "kaiming")
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=2, in_size=(8, 8), padding=spec.padding,
                      algo=algo)
    assert co.algo.startswith(algo)
    n = 2 * 16 * 8 * 8
    buf = torch.zeros(n + 1, dtype=x.dtype, device=DEV)
    outs = []
    for t in range(x.shape[2]):
        buf[1:].copy_(x[:, :, t].reshape(-1).to(DEV))
        fr = buf[1:].view(2, 16, 8, 8)
        assert fr.data_ptr() % 16 != 0
        y = co.forward_step(fr)
        if y is not None:
            outs.append(y.clone())
    torch.cuda.synchronize()
    got = np.stack([np64(o) for o in outs], axis=2)
    ref = oracle_conv(w, b, spec.stride, spec.padding, spec.dilation, 1).forward_steps(np64(x))
    assert_close(got, ref, synth.torch_dtype(dt), f"{algo} misaligned", terms=conv_terms(w))


CLIP_WS_CASES = [
    # algo, B, Cin, Cout, kernel (time first), in_size, stride, padding, dilation, dtype
    ("gemm_ws", 3, 40, 24, (3, 3, 3), (8, 10), (1, 1, 1), (1, 1, 1), (1, 1, 1), "bf16"),
    ("gemm", 2, 20, 36, (2, 3, 3), (7, 6), (1, 1, 1), (1, 0, 1), (1, 1, 1), "f32"),
    ("gemm_reg", 4, 64, 48, (4, 1), (25,), (1, 1), (2, 0), (1, 1), "bf16"),
    ("gemm_reg", 3, 12, 40, (5, 3, 3), (7, 9), (2, 2, 2), (3, 1, 1), (1, 2, 1), "bf16"),
    ("depthwise", 3, 10, 10, (3, 3, 3), (7, 7), (1, 1, 1), (1, 1, 1), (1, 1, 1), "bf16"),
    ("direct", 1, 4, 8, (3,), (), (2,), (1,), (2,), "f32"),
]


@pytest.mark.parametrize("case", CLIP_WS_CASES, ids=lambda c: "clipws_" + c[0] + "_" + c[-1])
def test_clip_forward_on_step_kernels(case):
    """co_conv_forward_ws (clip mode on the step kernels, from a clean state
    in a scratch workspace): the regular convolution of the oracle, the
    direct clip kernel within the same bound, and forward_steps with end
    padding from a clean state bit for bit (Principles 2 and 4: a clip
    processed step by step with its end padding emits the regular output)."""
    algo, B, ci, co_, k, size, s, p, dil, dt = case
    say("clip ws", case)
    tdt = synth.torch_dtype(dt)
    spec = synth.ConvSpec(batch=B, in_channels=ci, out_channels=co_, kernel=k, in_size=size,
                          stride=s, padding=p, dilation=dil,
                          groups=ci if algo == "depthwise" else 1, dtype=dt)
    x, w, b = synth.conv_inputs(spec, 11, 99000 + ci * 3 + co_, "kaiming")
    xd = x.to(DEV)
    G = ci if algo == "depthwise" else 1

    def make():
        return coinf.CoConv(w.to(DEV), b.to(DEV), batch=B, in_size=size, stride=s, padding=p,
                            dilation=dil, groups=G, algo=algo)

    co = make()
    assert co.algo.startswith(algo)
    clip = co.forward(xd)
    ref = oracle.conv_forward(np64(x), np64(w), np64(b), s, p, dil, G)
    assert_close(np64(clip), ref, tdt, f"clip ws {algo}", terms=conv_terms(w))
    direct = coinf.conv_forward(co.desc, co.weight, co.bias, xd, direct=True)
    assert_close(np64(direct), ref, tdt, f"clip direct {algo}", terms=conv_terms(w))
    steps = make().forward_steps(xd, pad_end=True)
    assert torch.equal(clip, steps)


def test_clip_forward_on_step_kernels_64_streams():
    """The 64-stream layer's clip through co_conv_forward_ws (its steps run
    on the warp-specialized and persistent GEMM kernels): sampled streams
    against the oracle's regular convolution."""
    name = "conv3d_b64_c192_k3_14x14_bf16"
    wl = synth.WORKLOADS[name]
    c = wl.conv
    say("clip ws", name)
    x, w, b = synth.workload_inputs(name)
    x = x[:, :, :6].contiguous()
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=c.batch, in_size=c.in_size, stride=c.stride,
                      padding=c.padding, dilation=c.dilation, groups=c.groups)
    clip = co.forward(x.to(DEV))
    sel = [0, 31, 63]
    ref = oracle.conv_forward(np64(x[sel]), np64(w), np64(b), c.stride, c.padding, c.dilation,
                              c.groups)
    assert_close(np64(clip[sel]), ref, torch.bfloat16, "64-stream clip", terms=conv_terms(w))
