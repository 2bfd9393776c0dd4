"""Host-side tests of the C ABI (no GPU needed).

* libcoinf.so loads and exports every function include/coinf.h declares;
* descriptor validation returns the documented status codes;
* the step schedule (co_conv_plan_step / co_pool_plan_step) is checked
  symbolically on an exhaustive grid: replaying the plans on a model ring of
  "which (frame, tap) products each slot holds" must deliver, for every
  emitted output, exactly the set of real-frame taps that the ordinary
  convolution of its window sums -- and the emission steps must match the
  oracle's sliding-window driver.
"""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

from paper_2204_03418_amd import coinf as C
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "coinf.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(co_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 20
    lib = ctypes.CDLL(C.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings():
    for s in (C.CO_OK, C.CO_EMPTY, C.CO_EINVAL, C.CO_ENOTSUP, C.CO_ESTATE, C.CO_EHIP):
        assert C.co_status_str(s).decode().startswith("CO_")


def desc1d(k=3, s=1, p=0, d=1, cin=2, cout=3, groups=1, B=1, **kw):
    return C.conv_desc(B, cin, cout, (k,), (), (s,), (p,), (d,), groups, True, C.CO_F32, **kw)


def test_query_delay_and_receptive_field_example1():
    # Example 1: co.Conv3d(4, 8, 3) has delay 2 and receptive field 3
    d = C.conv_desc(2, 4, 8, (3, 3, 3), (6, 7))
    info = C.conv_query(d)
    assert (info.delay, info.receptive_field) == (2, 3)
    assert tuple(info.out_size) == (4, 5)


@pytest.mark.parametrize("k,p,dil,expect_d", [(3, 0, 1, 2), (3, 2, 1, 0), (3, 1, 1, 1),
                                               (3, 0, 2, 4), (1, 0, 1, 0), (9, 0, 1, 8)])
def test_query_principle4_delay(k, p, dil, expect_d):
    info = C.conv_query(desc1d(k=k, p=p, d=dil))
    assert info.delay == expect_d
    assert info.receptive_field == dil * (k - 1) + 1


def _status(desc):
    info = C.ConvInfo()
    return C.co_conv_query(ctypes.byref(desc), ctypes.byref(info))


def test_invalid_descriptors():
    assert _status(desc1d(p=3)) == C.CO_EINVAL              # negative delay
    assert _status(desc1d(cin=3, groups=2)) == C.CO_EINVAL  # groups do not divide
    assert _status(desc1d(cout=3, cin=2, groups=2)) == C.CO_EINVAL
    assert _status(desc1d(k=0)) == C.CO_EINVAL
    assert _status(desc1d(s=0)) == C.CO_EINVAL
    assert _status(desc1d(d=0)) == C.CO_EINVAL
    assert _status(desc1d(B=0)) == C.CO_EINVAL
    assert _status(desc1d(k=65)) == C.CO_EINVAL             # more taps than CO_MAX_TAPS
    d = desc1d()
    d.dtype = 7
    assert _status(d) == C.CO_EINVAL
    d = desc1d()
    d.in_size[1] = 2                                          # unused axis must be 1
    assert _status(d) == C.CO_EINVAL
    d = C.conv_desc(1, 2, 2, (3, 5), (4,))                    # spatial window does not fit
    assert _status(d) == C.CO_EINVAL
    d = desc1d()
    d.algo = 9
    assert _status(d) == C.CO_EINVAL


def test_forced_algorithm_not_supported():
    d = desc1d(cin=4, cout=4, groups=2, algo="depthwise")
    assert _status(d) == C.CO_ENOTSUP


def test_auto_algorithm_choice():
    dw = C.conv_desc(2, 8, 8, (3, 3, 3), (7, 7), padding=(0, 1, 1), groups=8)
    assert C.conv_query(dw).algo == C.CO_ALGO_DEPTHWISE
    g = C.conv_desc(1, 2, 3, (3,), ())
    assert C.conv_query(g).algo in (C.CO_ALGO_DIRECT, C.CO_ALGO_GEMM, C.CO_ALGO_GEMM_REG)


def test_frames_past_32bit_offsets_keep_to_64bit_kernels():
    """The GEMM-family kernels address one frame and the ring with 32-bit byte
    offsets: an input or output frame of 2^31 bytes (within the element limit)
    rules them out when the algorithm is chosen, one stream fewer keeps them."""
    f32 = dict(padding=(0, 1, 1), dtype=C.CO_F32)
    # input frame 128 x 256 x 128 x 128 fp32 = 2^31 bytes
    d = C.conv_desc(128, 256, 16, (1, 3, 3), (128, 128), algo="gemm", **f32)
    assert _status(d) == C.CO_ENOTSUP
    d = C.conv_desc(128, 256, 16, (1, 3, 3), (128, 128), **f32)
    assert C.conv_query(d).algo == C.CO_ALGO_DIRECT
    d = C.conv_desc(127, 256, 16, (1, 3, 3), (128, 128), algo="gemm", **f32)
    assert C.conv_query(d).algo == C.CO_ALGO_GEMM
    # output frame 128 x 256 x 128 x 128 fp32
    d = C.conv_desc(128, 16, 256, (1, 3, 3), (128, 128), algo="gemm", **f32)
    assert _status(d) == C.CO_ENOTSUP
    d = C.conv_desc(127, 16, 256, (1, 3, 3), (128, 128), algo="gemm", **f32)
    assert C.conv_query(d).algo == C.CO_ALGO_GEMM
    # register GEMM, bf16 1x1: input frame 1024 x 64 x 128 x 128 bf16 = 2^31 bytes
    d = C.conv_desc(1024, 64, 16, (1, 1, 1), (128, 128), dtype=C.CO_BF16, algo="gemm_reg")
    assert _status(d) == C.CO_ENOTSUP
    d = C.conv_desc(1023, 64, 16, (1, 1, 1), (128, 128), dtype=C.CO_BF16, algo="gemm_reg")
    assert C.conv_query(d).algo == C.CO_ALGO_GEMM_REG


def test_null_and_small_buffers_rejected_without_device():
    d = desc1d()
    info = C.conv_query(d)
    h = ctypes.c_void_p()
    fake = ctypes.c_void_p(0x1000)
    assert C.co_conv_init_state(ctypes.byref(d), fake, fake, None, info.state_bytes, None,
                                ctypes.byref(h)) == C.CO_EINVAL
    assert C.co_conv_init_state(ctypes.byref(d), None, fake, fake, info.state_bytes, None,
                                ctypes.byref(h)) == C.CO_EINVAL
    assert C.co_conv_init_state(ctypes.byref(d), fake, None, fake, info.state_bytes, None,
                                ctypes.byref(h)) == C.CO_EINVAL      # has_bias without bias
    assert C.co_conv_init_state(ctypes.byref(d), fake, fake, fake, info.state_bytes - 1, None,
                                ctypes.byref(h)) == C.CO_ESTATE
    assert C.co_conv_attach_state(ctypes.byref(d), fake, info.state_bytes - 4, 0, None,
                                  ctypes.byref(h)) == C.CO_ESTATE
    assert C.co_conv_attach_state(ctypes.byref(d), fake, info.state_bytes, -1, None,
                                  ctypes.byref(h)) == C.CO_EINVAL
    assert C.co_conv_forward_step(None, fake, fake, 1, None) == C.CO_EINVAL
    n = C.i32()
    assert C.co_conv_forward_steps(None, fake, 4, fake, 4, 0, 1, None, ctypes.byref(n)) == C.CO_EINVAL
    assert C.co_conv_destroy(None) == C.CO_EINVAL
    assert C.co_conv_forward(ctypes.byref(d), None, fake, fake, 5, fake, None) == C.CO_EINVAL
    # a clip too short for one window writes nothing and succeeds without the device
    assert C.co_conv_forward(ctypes.byref(d), fake, fake, fake, 2, fake, None) == C.CO_OK
    t = C.i32()
    assert C.co_conv_clip_frames(ctypes.byref(d), 7, ctypes.byref(t)) == C.CO_OK and t.value == 5


def _real_taps(tau, k, s, p, dil):
    """(real frame, tap) pairs that the ordinary convolution of output tau sums."""
    out = set()
    for j in range(k):
        r = tau * s + j * dil - p
        if r >= 0:
            out.add((r, j))
    return out


PLAN_GRID = [(k, s, dil, p) for k in (1, 2, 3, 4, 5) for s in (1, 2, 3) for dil in (1, 2, 3)
             for p in range(0, dil * (k - 1) + 1)]


@pytest.mark.parametrize("k,s,dil,p", PLAN_GRID)
def test_conv_plan_delivers_exact_window(k, s, dil, p):
    d = desc1d(k=k, s=s, p=p, d=dil)
    info = C.conv_query(d)
    R = info.ring_slots
    f = dil * (k - 1) + 1
    assert R == -(-(f - 1) // s) + 1
    ring = [None] * R           # slot -> (tau, set of (frame, tap)) or None
    steps = 40
    co = oracle.ContinualConv(np.ones((1, 1, k)), None, stride=s, padding=p, dilation=dil)
    for n in range(steps):
        plan = C.conv_plan(d, n, True)
        ref = co.forward_step(np.ones((1, 1)))
        assert bool(plan.emit) == (ref is not None), n
        emitted = None
        for j in range(k):
            a, slot, tau = plan.action[j], plan.slot[j], plan.target[j]
            if a == C.CO_TAP_NONE:
                assert slot == -1 and tau == -1
                continue
            assert tau * s + j * dil == n + p       # the frame really feeds tap j of tau
            if a == C.CO_TAP_START:
                assert ring[slot] is None, (n, j, "slot still live")
                ring[slot] = (tau, {(n, j)})
            elif a == C.CO_TAP_ACC:
                assert ring[slot] is not None and ring[slot][0] == tau
                ring[slot][1].add((n, j))
            elif a == C.CO_TAP_EMIT:
                assert j == k - 1 and ring[slot] is not None and ring[slot][0] == tau
                emitted = (tau, ring[slot][1] | {(n, j)})
                ring[slot] = None
            elif a == C.CO_TAP_EMIT_FRESH:
                assert j == k - 1 and slot == -1
                emitted = (tau, {(n, j)})
        if plan.emit:
            assert emitted is not None and emitted[0] == plan.out_index
            assert emitted[1] == _real_taps(plan.out_index, k, s, p, dil)
        else:
            assert emitted is None and plan.out_index == -1


@pytest.mark.parametrize("k,s,dil,p", PLAN_GRID[::3])
def test_conv_plan_update_state_false_keeps_only_completing_tap(k, s, dil, p):
    d = desc1d(k=k, s=s, p=p, d=dil)
    for n in range(20):
        a = C.conv_plan(d, n, True)
        b = C.conv_plan(d, n, False)
        assert a.emit == b.emit and a.out_index == b.out_index
        for j in range(k):
            if j == k - 1:
                assert a.action[j] == b.action[j] and a.slot[j] == b.slot[j]
            else:
                assert b.action[j] == C.CO_TAP_NONE


STRIDED_GRID = [g for g in PLAN_GRID if g[1] > 1 or g[2] > 1]


@pytest.mark.parametrize("k,s,dil,p", STRIDED_GRID)
def test_strided_plan_tables_and_segment_warmup(k, s, dil, p):
    """The bookkeeping of the plan-driven persistent kernels (temporal stride
    or dilation above 1), against the step plans themselves: (a) after a
    stream's first (k - 1) dil steps the plan of step n + s R equals that
    of step n, so explicit plans for a call's frames before that point plus
    one period of s R plans cover any call; (b) a time segment that starts
    max((k - 1) dil, s R) frames before its first stored frame, with every
    ring slot unknown, completes every output it stores from slots it
    started itself, and ends with every slot started inside it (k >= 2;
    with k = 1 no slot is ever written), so the last segment's write-back
    is the state stepping leaves; (c) the
    emission count at a segment's first frame follows from the call's
    first emitting frame."""
    d = desc1d(k=k, s=s, p=p, d=dil)
    R = C.conv_query(d).ring_slots
    delay = C.conv_query(d).delay
    period, warm = s * R, max((k - 1) * dil, s * R)

    def key(n):
        pl = C.conv_plan(d, n, True)
        return tuple((pl.action[j], pl.slot[j]) for j in range(k)), bool(pl.emit)

    for n0 in (0, 1, 5, 37):
        count = 24 * warm
        n_start = max(0, min(count, (k - 1) * dil - n0))
        for t in range(n_start, count):
            assert key(n0 + t) == key(n0 + n_start + (t - n_start) % period), (n0, t)
        emits = [t for t in range(count) if key(n0 + t)[1]]
        t_e0 = (s - (n0 - delay) % s) % s if n0 >= delay else delay - n0
        assert not emits or emits[0] == min(t_e0, count)
        for s0 in range(4 * warm, count, 3):
            tw = s0 - warm
            before = sum(1 for t in emits if t < tw)
            assert before == ((tw - t_e0 + s - 1) // s if tw > t_e0 else 0), (n0, s0)
            known = [False] * R
            for t in range(tw, count):
                pl = C.conv_plan(d, n0 + t, True)
                for j in range(k):
                    a, sl = pl.action[j], pl.slot[j]
                    if a == C.CO_TAP_START:
                        known[sl] = True
                    elif a == C.CO_TAP_EMIT and t >= s0:
                        assert known[sl], (n0, s0, t, j)
            assert all(known) if k > 1 else not any(known), (n0, s0)


POOL_PLAN_GRID = [(k, s, dil, p) for k in (1, 2, 3, 4, 7) for s in (1, 2, 3) for dil in (1, 2)
                  for p in range(0, k // 2 + 1)]


@pytest.mark.parametrize("k,s,dil,p", POOL_PLAN_GRID)
def test_pool_plan_reads_the_window(k, s, dil, p):
    d = C.pool_desc("max", 1, 1, (k,), (), (s,), (p,), (dil,))
    info = C.pool_query(d)
    f = dil * (k - 1) + 1
    assert info.fifo_slots == f and info.delay == f - p - 1
    fifo = {}
    for n in range(40):
        plan = C.pool_plan(d, n)
        if plan.emit:
            tau = plan.out_index
            assert tau * s + f - 1 - p == n
            for j in range(k):
                r = tau * s + j * dil - p
                src = plan.src[j]
                if r < 0:
                    assert src == -1
                elif r == n:
                    assert src == -2
                else:
                    assert fifo.get(src) == r, (n, j)
        fifo[plan.write_slot] = n


def test_pool_validation():
    info = C.PoolInfo()
    bad = C.pool_desc("avg", 1, 1, (3, 3, 3), (5, 5), (1, 1, 1), (0, 2, 0))  # pad > k/2
    assert C.co_pool_query(ctypes.byref(bad), ctypes.byref(info)) == C.CO_EINVAL
    bad = C.pool_desc("avg", 1, 1, (3,), (), (1,), (0,), (2,))               # avg dilation
    assert C.co_pool_query(ctypes.byref(bad), ctypes.byref(info)) == C.CO_ENOTSUP
    ok = C.pool_desc("avg", 16, 432, (4, 7, 7), (7, 7), (1, 7, 7))
    assert C.co_pool_query(ctypes.byref(ok), ctypes.byref(info)) == C.CO_OK
    assert info.delay == 3 and tuple(info.out_size) == (1, 1)


def test_emission_count_matches_oracle_formula():
    for k, s, p in itertools.product((1, 3, 4), (1, 2, 3), (0, 1, 2)):
        if p > k - 1:
            continue
        d = desc1d(k=k, s=s, p=p)
        # forward_steps over T frames emits floor((T + p - f)/s) + 1 outputs
        for T in range(0, 12):
            emitted = sum(C.conv_plan(d, n).emit for n in range(T))
            expect = (T + p - k) // s + 1 if T + p >= k else 0
            assert emitted == expect


def test_gemm_state_and_algorithm_for_named_workloads():
    """Every named workload resolves to its intended kernel family and a
    state size that holds the packed weights and the ring."""
    from paper_2204_03418_amd import synth
    expect = {"conv1d_b1_c4to8_k3_f32": C.CO_ALGO_DIRECT,
              "dwconv3d_b16_c432_k3_7x7_avgpool_bf16": C.CO_ALGO_DEPTHWISE,
              "conv3d_b1_c24_k3_56x56_f32": C.CO_ALGO_GEMM_REG,
              "conv2d_b32_c64to256_k9x1_v25_f32": C.CO_ALGO_GEMM_REG,
              "conv2d_b32_c64to256_k9x1_v25_bf16": C.CO_ALGO_GEMM_REG}
    for name, w in synth.WORKLOADS.items():
        c = w.conv
        d = C.conv_desc(c.batch, c.in_channels, c.out_channels, c.kernel, c.in_size, c.stride,
                        c.padding, c.dilation, c.groups, True,
                        C.CO_BF16 if c.dtype == "bf16" else C.CO_F32)
        info = C.conv_query(d)
        assert info.algo == expect.get(name, C.CO_ALGO_GEMM), name
        esz = 2 if c.dtype == "bf16" else 4
        So = 1
        for s in info.out_size[:len(c.in_size)]:
            So *= s
        ring = info.ring_slots * c.batch * c.out_channels * So * 4
        assert info.state_bytes >= ring + c.out_channels * 4, name


def test_register_gemm_shapes():
    """The register-operand GEMM holds K = kH*kW*C_in in registers: it takes
    small-K layers with C_out >= 16 and refuses the rest when forced."""
    ok = C.conv_desc(1, 24, 24, (3, 3, 3), (56, 56), padding=(0, 1, 1), algo="gemm_reg")
    assert C.conv_query(ok).algo == C.CO_ALGO_GEMM_REG
    bf = C.conv_desc(32, 64, 256, (9, 1), (25,), dtype=C.CO_BF16, algo="gemm_reg")
    assert C.conv_query(bf).algo == C.CO_ALGO_GEMM_REG
    deep = C.conv_desc(2, 192, 192, (3, 3, 3), (14, 14), padding=(0, 1, 1), algo="gemm_reg")
    assert _status(deep) == C.CO_ENOTSUP          # K = 1728: too deep for registers
    narrow = C.conv_desc(1, 4, 8, (3,), (), algo="gemm_reg")
    assert _status(narrow) == C.CO_ENOTSUP        # C_out < 16
    grouped = C.conv_desc(1, 32, 32, (3, 3, 3), (8, 8), groups=2, algo="gemm_reg")
    assert _status(grouped) == C.CO_ENOTSUP


def _chain(f, s, p):
    n = len(f)
    arr = ctypes.c_int32 * n
    out = [ctypes.c_int64() for _ in range(4)]
    st = C.co_chain_delay(n, arr(*f), arr(*s), arr(*p), *[ctypes.byref(o) for o in out])
    return st, tuple(o.value for o in out)


def test_chain_delay_principle6():
    """co_chain_delay against the worked example (printed values) and the
    oracle's chain formula, itself pinned by stepped chains."""
    assert _chain([3, 3], [2, 1], [2, 0]) == (C.CO_OK, (7, 2, 2, 4))
    assert _chain([3, 4], [1, 1], [0, 0]) == (C.CO_OK, (6, 0, 1, 5))   # conv then pool: d = 5
    rng = np.random.default_rng(17)
    for _ in range(200):
        n = int(rng.integers(1, 5))
        f = [int(v) for v in rng.integers(1, 8, n)]
        s = [int(v) for v in rng.integers(1, 4, n)]
        p = [int(rng.integers(0, fi)) for fi in f]
        st, got = _chain(f, s, p)
        assert st == C.CO_OK and got == oracle.chain_delay(f, s, p)
    assert _chain([3, 0], [1, 1], [0, 0])[0] == C.CO_EINVAL
    assert _chain([3], [0], [0])[0] == C.CO_EINVAL
    assert _chain([3], [1], [-1])[0] == C.CO_EINVAL


def test_delay_query_and_validation():
    d = C.DelayDesc(2, 3, 5, 4, C.CO_BF16)
    nb = ctypes.c_int64()
    assert C.co_delay_query(ctypes.byref(d), ctypes.byref(nb)) == C.CO_OK
    assert nb.value == 256 + 4 * 2 * 3 * 5 * 2
    for bad in (C.DelayDesc(0, 3, 5, 1, C.CO_F32), C.DelayDesc(1, 3, 5, -1, C.CO_F32),
                C.DelayDesc(1, 3, 0, 1, C.CO_F32), C.DelayDesc(1, 3, 5, 1, 7)):
        assert C.co_delay_query(ctypes.byref(bad), ctypes.byref(nb)) == C.CO_EINVAL
    # a state buffer that is too small is rejected before any device work
    h = ctypes.c_void_p()
    buf = ctypes.create_string_buffer(16)
    assert C.co_delay_init_state(ctypes.byref(d), buf, 16, None, ctypes.byref(h)) == C.CO_ESTATE
    # clip merge: shape and argument checks happen on the host
    assert C.co_add_frames(None, None, None, 4, 3, 0, 5, 0, C.CO_F32, None) == C.CO_OK
    assert C.co_add_frames(None, None, None, 4, 3, 4, 5, 2, C.CO_F32, None) == C.CO_EINVAL
    assert C.co_add_frames(None, None, None, 4, 0, 1, 5, 0, C.CO_F32, None) == C.CO_EINVAL


def _oracle_count(mod, n0, T, pad_end):
    """Outputs the oracle's sliding-window driver emits over T frames (plus
    its end padding) after n0 earlier frames: the count is counted, not
    computed."""
    x = np.zeros((1, 1, n0 + T))
    for t in range(n0):
        mod.forward_step(x[:, :, t])
    y = mod.forward_steps(x[:, :, n0:], pad_end=pad_end)
    return 0 if y is None else y.shape[2]


@pytest.mark.parametrize("k,s,p,dil", [(k, s, p, dil) for k, s, p, dil in
                                       itertools.product((1, 2, 3, 5), (1, 2, 3), (0, 1, 2, 4),
                                                         (1, 2))
                                       if p <= dil * (k - 1)])
def test_out_frames_calls_match_oracle_driver(k, s, p, dil):
    """co_conv_out_frames / co_pool_out_frames (Principles 4-5, the capacity a
    forward_steps call needs) against the number of outputs the oracle's
    driver emits for the same call, from several step counters."""
    d = desc1d(k=k, s=s, p=p, d=dil, cin=1, cout=1)
    w = np.ones((1, 1, k))
    for n0, T, pad_end in itertools.product((0, 1, 2, 5, 9), (0, 1, 3, 7, 12), (False, True)):
        if n0 + T == 0:
            continue  # no real frame at all: the oracle defines no output over padding only
        got = C.conv_out_frames(d, n0, T, pad_end)
        ref = _oracle_count(oracle.ContinualConv(w, None, stride=s, padding=p, dilation=dil),
                            n0, T, pad_end)
        assert got == ref, (k, s, p, dil, n0, T, pad_end)
        if 2 * p <= k and dil == 1:  # PyTorch's pool padding rule
            pd = C.pool_desc("max", 1, 1, (k,), (), (s,), (p,))
            got = C.pool_out_frames(pd, n0, T, pad_end)
            ref = _oracle_count(oracle.ContinualPool("max", (k,), (s,), (p,), spatial_dims=0),
                                n0, T, pad_end)
            assert got == ref, ("pool", k, s, p, n0, T, pad_end)


def test_out_frames_rejects_bad_arguments():
    d = desc1d()
    n = C.i32()
    assert C.co_conv_out_frames(ctypes.byref(d), -1, 4, 0, ctypes.byref(n)) == C.CO_EINVAL
    assert C.co_conv_out_frames(ctypes.byref(d), 0, -1, 0, ctypes.byref(n)) == C.CO_EINVAL
    assert C.co_conv_out_frames(ctypes.byref(d), (1 << 62) - 2, 4, 0,
                                ctypes.byref(n)) == C.CO_EINVAL   # past the step limit
    assert C.co_conv_out_frames(ctypes.byref(desc1d(p=3)), 0, 4, 0,
                                ctypes.byref(n)) == C.CO_EINVAL   # invalid descriptor


@pytest.mark.parametrize("k,p,dil", [(k, p, dil) for k, p, dil in
                                     itertools.product((1, 2, 3, 4, 5, 7), range(0, 4), (1, 2))
                                     if p <= dil * (k - 1)])
def test_residual_align_matches_oracle_residual(k, p, dil):
    """co_residual_align (section 3.1.1, Principle 7) against the oracle's
    residual connection: its delay line, its clip-mode shrink, and the step
    of its first non-empty output, counted by stepping it."""
    f = dil * (k - 1) + 1
    mod = oracle.ContinualConv(np.ones((1, 1, k)), None, padding=p, dilation=dil)
    al = C.residual_align(f, 1, p, mod.delay)
    if 2 * p > f - 1:
        assert al is None
        with pytest.raises(ValueError):
            oracle.ContinualResidual(mod)
        return
    d_res, shrink, delay = al
    res = oracle.ContinualResidual(mod)
    assert res.b.d == d_res and res.shrink == shrink
    x = np.ones((1, 1, 3 * f + 4))
    first = next(t for t in range(x.shape[2]) if res.forward_step(x[:, :, t]) is not None)
    assert first == delay
    # clip mode: the module's output is the input less `shrink` frames at the
    # start and at the end (one more at the end for an even receptive field,
    # whose centre falls between two frames)
    y = res.forward(x)
    assert x.shape[2] - 2 * shrink - y.shape[2] == (1 - f % 2)
    assert C.residual_align(f, 2, p, mod.delay) is None  # strided modules have no residual


def test_stale_and_foreign_handles_rejected_without_device():
    """A pointer the library never made (or one already destroyed) is not
    dereferenced: every call returns CO_EINVAL."""
    bogus = ctypes.c_void_p(0x1234)
    n = C.i64()
    assert C.co_conv_forward_step(bogus, bogus, bogus, 1, None) == C.CO_EINVAL
    assert C.co_conv_get_steps(bogus, ctypes.byref(n)) == C.CO_EINVAL
    assert C.co_conv_destroy(bogus) == C.CO_EINVAL
    assert C.co_pool_destroy(bogus) == C.CO_EINVAL
    assert C.co_delay_destroy(bogus) == C.CO_EINVAL
    assert C.co_convpool_destroy(bogus) == C.CO_EINVAL
    assert C.co_bneck_destroy(bogus) == C.CO_EINVAL
    out = ctypes.c_void_p()
    assert C.co_bneck_bind(bogus, 0, bogus, 0, bogus, ctypes.byref(out)) == C.CO_EINVAL
    assert C.co_bneck_forward_step(bogus, bogus, bogus, 1, None) == C.CO_EINVAL
    n32 = C.i32()
    assert C.co_bneck_forward_steps(bogus, bogus, 1, bogus, 1, 1, None,
                                    ctypes.byref(n32)) == C.CO_EINVAL
    assert C.co_conv_algo_name(bogus) == b"none"


def test_step_counter_limit_without_device():
    """Step counters stay below 2^62 (the schedule's n + pT and n + count
    cannot overflow): plans and attaches past it are rejected on the host."""
    d = desc1d(p=2)
    plan = C.StepPlan()
    assert C.co_conv_plan_step(ctypes.byref(d), 1 << 62, 1, ctypes.byref(plan)) == C.CO_EINVAL
    assert C.co_conv_plan_step(ctypes.byref(d), (1 << 62) - 1, 1, ctypes.byref(plan)) == C.CO_OK
    assert plan.emit == 1 and plan.out_index == (1 << 62) - 1
    h = ctypes.c_void_p()
    assert C.co_conv_attach_state(ctypes.byref(d), ctypes.c_void_p(0x1000), 1 << 20,
                                  (1 << 62) + 1, None, ctypes.byref(h)) == C.CO_EINVAL
    pd = C.pool_desc("avg", 1, 1, (3,), (), (1,), (1,))
    pplan = C.PoolPlan()
    assert C.co_pool_plan_step(ctypes.byref(pd), 1 << 62, ctypes.byref(pplan)) == C.CO_EINVAL


def test_pool_frames_of_2GiB_are_rejected():
    """The pool step kernels address a frame with 32-bit buffer offsets: a
    frame of 2^31 bytes or more is rejected when the descriptor is queried."""
    info = C.PoolInfo()
    big = C.pool_desc("avg", 1, 1, (2, 1, 1), (32768, 16384), (1, 1, 1), dtype=C.CO_F32)
    assert C.co_pool_query(ctypes.byref(big), ctypes.byref(info)) == C.CO_EINVAL
    half = C.pool_desc("avg", 1, 1, (2, 1, 1), (32768, 16384), (1, 1, 1), dtype=C.CO_BF16)
    assert C.co_pool_query(ctypes.byref(half), ctypes.byref(info)) == C.CO_OK


def test_warp_specialized_gemm_selection():
    """CO_ALGO_GEMM_WS: granted for bf16 3x3 layers with Ho*Wo % 4 == 0 and
    spatial padding <= 1, refused otherwise.  AUTO takes the register GEMM
    below 3e8 multiply-accumulates per step and the warp-specialized GEMM
    above it where it applies (the 64-stream layer, a 16-stream 128-channel
    layer), else the LDS-tiled GEMM."""
    def q(B, cin, cout, size, pad=(0, 1, 1), dtype=C.CO_BF16, algo=C.CO_ALGO_GEMM_WS, k=(3, 3, 3)):
        d = C.conv_desc(B, cin, cout, k, size, (1, 1, 1), pad, (1, 1, 1), 1, True, dtype,
                        algo=algo)
        info = C.ConvInfo()
        return C.co_conv_query(ctypes.byref(d), ctypes.byref(info)), info
    st, info = q(3, 40, 24, (8, 10))
    assert st == C.CO_OK and info.algo == C.CO_ALGO_GEMM
    assert q(3, 40, 24, (9, 11))[0] == C.CO_ENOTSUP                    # Ho*Wo = 99
    assert q(3, 40, 24, (8, 10), dtype=C.CO_F32)[0] == C.CO_ENOTSUP    # fp32
    assert q(3, 40, 24, (8, 10), pad=(0, 2, 2))[0] == C.CO_ENOTSUP     # spatial padding 2
    assert q(3, 40, 24, (8, 10), k=(3, 1, 1))[0] == C.CO_ENOTSUP       # 1x1 taps
    # the 64-stream layer's state holds the ws kernel's packed weights
    st, big = q(64, 192, 192, (14, 14), algo=C.CO_ALGO_AUTO)
    st2, forced = q(64, 192, 192, (14, 14))
    assert st == st2 == C.CO_OK and big.state_bytes == forced.state_bytes
    # AUTO by the work of a step
    assert q(3, 40, 24, (8, 10), algo=C.CO_ALGO_AUTO)[1].algo == C.CO_ALGO_GEMM_REG
    st, mid = q(16, 128, 128, (14, 14), algo=C.CO_ALGO_AUTO)
    assert st == C.CO_OK and mid.state_bytes == q(16, 128, 128, (14, 14))[1].state_bytes
    st, wide = q(4, 256, 256, (28, 28), pad=(0, 0, 0), k=(3, 1, 1), algo=C.CO_ALGO_AUTO)
    assert st == C.CO_OK and wide.algo == C.CO_ALGO_GEMM                # 617 M: LDS-tiled


def test_batch_norm_and_activation_validation_without_device():
    """co_conv_init_state_bn / co_conv_fold_bn reject missing statistics and
    a negative or non-finite eps, and co_act_forward an unknown activation or
    dtype, all before anything is launched; zero elements is a no-op."""
    d = desc1d(p=2)
    dev = ctypes.c_void_p(0x1000)
    h = ctypes.c_void_p()
    for eps in (-1e-5, float("nan"), float("inf")):
        assert C.co_conv_init_state_bn(ctypes.byref(d), dev, dev, dev, dev, dev, dev, eps, dev,
                                       1 << 20, None, ctypes.byref(h)) == C.CO_EINVAL
        assert C.co_conv_fold_bn(ctypes.byref(d), dev, dev, dev, dev, dev, dev, eps, dev, dev,
                                 None) == C.CO_EINVAL
    assert C.co_conv_init_state_bn(ctypes.byref(d), dev, dev, None, dev, dev, dev, 1e-5, dev,
                                   1 << 20, None, ctypes.byref(h)) == C.CO_EINVAL
    assert C.co_conv_fold_bn(ctypes.byref(d), dev, dev, dev, dev, dev, None, 1e-5, dev, dev,
                             None) == C.CO_EINVAL
    assert C.co_conv_init_state_bn(ctypes.byref(d), dev, dev, dev, dev, dev, dev, 1e-5, dev,
                                   16, None, ctypes.byref(h)) == C.CO_ESTATE
    assert C.co_act_forward(dev, dev, 4, C.CO_F32, 7, None) == C.CO_EINVAL
    assert C.co_act_forward(dev, dev, 4, 9, C.CO_ACT_RELU, None) == C.CO_EINVAL
    assert C.co_act_forward(dev, dev, -1, C.CO_F32, C.CO_ACT_RELU, None) == C.CO_EINVAL
    assert C.co_act_forward(None, None, 0, C.CO_BF16, C.CO_ACT_RELU, None) == C.CO_OK
    assert C.co_act_forward(None, dev, 4, C.CO_F32, C.CO_ACT_RELU, None) == C.CO_EINVAL


def test_clip_forward_ws_validation_without_device():
    """co_conv_forward_ws: a missing workspace or buffer is CO_EINVAL, a
    workspace below state_bytes CO_ESTATE, a clip too short to emit is a
    no-op; nothing is launched in these cases."""
    d = desc1d(k=3, p=0, cin=2, cout=3)
    info = C.conv_query(d)
    dev = ctypes.c_void_p(0x1000)
    assert C.co_conv_forward_ws(ctypes.byref(d), dev, dev, None, dev, 2, dev, dev,
                                info.state_bytes, None) == C.CO_OK  # T_out = 0
    assert C.co_conv_forward_ws(ctypes.byref(d), dev, dev, None, dev, 5, dev, None,
                                info.state_bytes, None) == C.CO_EINVAL
    assert C.co_conv_forward_ws(ctypes.byref(d), dev, dev, None, None, 5, dev, dev,
                                info.state_bytes, None) == C.CO_EINVAL
    assert C.co_conv_forward_ws(ctypes.byref(d), dev, dev, None, dev, 5, dev, dev,
                                info.state_bytes - 1, None) == C.CO_ESTATE
    assert C.co_conv_forward_ws(ctypes.byref(d), None, dev, None, dev, 5, dev, dev,
                                info.state_bytes, None) == C.CO_EINVAL
