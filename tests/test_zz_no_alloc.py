"""co_conv_forward_steps_noalloc (the entry point for callers that cannot
allocate device memory) against co_conv_forward_steps, through the C ABI.

The two run the same kernels; the no-allocation one keeps the ring backup
(update_state = 0 on the looping path) and staged frame copies in the
library's per-GPU scratch instead of stream-ordered allocations.  Outputs and
states must be bitwise equal, and both within the parity bar of the oracle.
Every case makes two calls in a row, the second with a smaller input.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2204_03418_amd import coinf, synth
from parity_util import assert_close, conv_terms, np64, oracle_conv, say

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _layer(spec, algo, seed):
    x, w, b = synth.conv_inputs(spec, frames=16, seed_base=seed)
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=spec.batch, in_size=spec.in_size,
                      stride=spec.stride, padding=spec.padding, dilation=spec.dilation,
                      groups=spec.groups, algo=algo)
    return co, x, w, b


def _call(fn, co, x, pad_end, update):
    """One forward_steps call through the C ABI on device clip x; returns
    (status, emitted frames)."""
    T = x.shape[2]
    cap = T + co.t_padding + 1
    y = torch.full((co.batch, co.out_channels, cap) + co.out_size, float("nan"),
                   dtype=co.torch_dtype, device=DEV)
    n = coinf.i32()
    st = fn(co.handle, ctypes.c_void_p(x.data_ptr()), T, ctypes.c_void_p(y.data_ptr()), cap,
            1 if pad_end else 0, 1 if update else 0,
            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), ctypes.byref(n))
    torch.cuda.synchronize()
    return st, y[:, :, :n.value]


def _oracle(co, w, b, x_cpu, pad_end):
    ref = oracle_conv(w, b, co.desc.stride[:co.desc.spatial_dims + 1],
                      co.desc.padding[:co.desc.spatial_dims + 1],
                      co.desc.dilation[:co.desc.spatial_dims + 1], co.desc.groups)
    return ref.forward_steps(np64(x_cpu), pad_end=pad_end)


CASES = [
    # (name, spec, algo, misaligned frames) -- temporal stride 2 keeps every
    # call on the looping path, where update_state = 0 needs the ring backup
    ("gemm_bf16", synth.ConvSpec(batch=4, in_channels=32, out_channels=32, kernel=(3, 3, 3),
                                 in_size=(8, 8), stride=(2, 1, 1), padding=(1, 1, 1),
                                 dtype="bf16"), "gemm", False),
    ("gemm_bf16_misaligned", synth.ConvSpec(batch=4, in_channels=32, out_channels=32,
                                            kernel=(3, 3, 3), in_size=(8, 8), stride=(2, 1, 1),
                                            padding=(1, 1, 1), dtype="bf16"), "gemm", True),
    ("reg_f32", synth.ConvSpec(batch=2, in_channels=16, out_channels=32, kernel=(3, 3, 3),
                               in_size=(10, 10), stride=(2, 1, 1), padding=(2, 1, 1),
                               dtype="f32"), "gemm_reg", False),
    ("direct_f32", synth.ConvSpec(batch=2, in_channels=4, out_channels=8, kernel=(3,),
                                  stride=(2,), padding=(1,), dtype="f32"), "direct", False),
    ("depthwise_bf16_dilated", synth.ConvSpec(batch=2, in_channels=24, out_channels=24,
                                              kernel=(3, 3, 3), in_size=(7, 7),
                                              dilation=(2, 1, 1), padding=(1, 1, 1),
                                              groups=24, dtype="bf16"), "auto", False),
]


def _clip(x_cpu, misaligned):
    """Device copy of the clip; misaligned: starting one element past an
    aligned address (the GEMM kernels' frames are then staged)."""
    if not misaligned:
        return x_cpu.to(DEV)
    flat = torch.empty(x_cpu.numel() + 1, dtype=x_cpu.dtype, device=DEV)
    v = flat[1:].view(x_cpu.shape)
    v.copy_(x_cpu.to(DEV))
    return v


@pytest.mark.parametrize("name,spec,algo,misaligned", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("update", [False, True], ids=["keep_state", "update_state"])
def test_noalloc_matches_allocating_entry_point(name, spec, algo, misaligned, update):
    say(f"noalloc case {name} update={update}")
    co_a, x, w, b = _layer(spec, algo, seed=7100)
    co_b, _, _, _ = _layer(spec, algo, seed=7100)
    assert co_a.algo == co_b.algo
    # init leaves the ring unwritten (each partial sum is started before it is
    # read): start both handles from the same bytes
    co_b.state.copy_(co_a.state)
    for T, pad_end in ((11, True), (5, False)):  # second call: a smaller input
        xs = x[:, :, :T].contiguous()
        xd = _clip(xs, misaligned)
        s0 = co_b.state.clone()
        st_a, y_a = _call(coinf.co_conv_forward_steps, co_a, xd, pad_end, update)
        st_b, y_b = _call(coinf.co_conv_forward_steps_noalloc, co_b, xd, pad_end, update)
        assert st_a == coinf.CO_OK and st_b == coinf.CO_OK, (st_a, st_b)
        assert torch.equal(y_a, y_b), f"{name}: outputs differ between the entry points"
        assert torch.equal(co_a.state, co_b.state), f"{name}: states differ"
        assert co_a.steps == co_b.steps
        if not update:
            assert torch.equal(co_b.state, s0), f"{name}: update_state=0 changed the state"
            assert co_b.steps == 0
            ref = _oracle(co_b, w, b, xs, pad_end)
            if ref is None:
                assert y_b.shape[2] == 0
            else:
                assert_close(np64(y_b), ref, co_b.torch_dtype, f"{name} T={T}", terms=conv_terms(w))


def test_noalloc_rejects_calls_beyond_the_scratch():
    """A looping call with update_state = 0 whose ring exceeds the scratch:
    CO_ESCRATCH, nothing enqueued, the handle unchanged."""
    cap = coinf.i64()
    assert coinf.co_conv_scratch_bytes(ctypes.byref(cap)) == coinf.CO_OK
    # temporal dilation 4 with kT = 3: nine ring slots, beyond the persistent
    # kernels' plan tables, so the call loops over step launches; ring:
    # 9 slots x 2048 channels x 4096 positions x 4 B = 288 MiB > 64 MiB
    spec = synth.ConvSpec(batch=1, in_channels=1, out_channels=2048, kernel=(3, 1),
                          in_size=(4096,), dilation=(4, 1), dtype="f32")
    say("noalloc rejection case")
    co, x, _, _ = _layer(spec, "direct", seed=7200)
    assert co.info.ring_slots == 9 and not co.steps_fused(10)
    assert co.info.ring_slots * 2048 * 4096 * 4 > cap.value
    xd = x[:, :, :10].contiguous().to(DEV)
    y = torch.empty((1, 2048, 10, 4096), dtype=torch.float32, device=DEV)
    n = coinf.i32(-7)
    st = coinf.co_conv_forward_steps_noalloc(
        co.handle, ctypes.c_void_p(xd.data_ptr()), 10, ctypes.c_void_p(y.data_ptr()), 10, 0, 0,
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), ctypes.byref(n))
    assert st == coinf.CO_ESCRATCH, coinf.co_status_str(st)
    assert n.value == -7 and co.steps == 0
    # with update_state = 1 no backup is needed: the same call runs (delay 8:
    # steps 8 and 9 emit)
    st = coinf.co_conv_forward_steps_noalloc(
        co.handle, ctypes.c_void_p(xd.data_ptr()), 10, ctypes.c_void_p(y.data_ptr()), 10, 0, 1,
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), ctypes.byref(n))
    torch.cuda.synchronize()
    assert st == coinf.CO_OK and n.value == 2 and co.steps == 10
