"""C-ABI behaviour that needs live handles (device state): the handle
registry and the step-counter limit."""
import ctypes

import pytest
import torch

from paper_2204_03418_amd import coinf, synth
from parity_util import say

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _conv(**kw):
    spec = synth.ConvSpec(batch=2, in_channels=4, out_channels=8, kernel=(3, 3, 3),
                          in_size=(6, 7), dtype="f32", **kw)
    x, w, b = synth.conv_inputs(spec, 6, 4242)
    co = coinf.CoConv(w.to(DEV), b.to(DEV), batch=2, in_size=(6, 7), stride=spec.stride,
                      padding=spec.padding)
    return co, x.to(DEV)


def test_destroyed_handle_is_rejected():
    say("destroyed handle")
    co, x = _conv()
    h = ctypes.c_void_p(co.handle.value)
    y = co.new_output()
    x0 = x[:, :, 0].contiguous()
    assert coinf.co_conv_forward_step(h, ctypes.c_void_p(x0.data_ptr()),
                                      ctypes.c_void_p(y.data_ptr()), 1, None) == coinf.CO_EMPTY
    assert coinf.co_conv_destroy(h) == coinf.CO_OK
    co.handle = None
    assert coinf.co_conv_destroy(h) == coinf.CO_EINVAL             # second destroy
    assert coinf.co_conv_forward_step(h, ctypes.c_void_p(x0.data_ptr()),
                                      ctypes.c_void_p(y.data_ptr()), 1, None) == coinf.CO_EINVAL
    n = coinf.i64()
    assert coinf.co_conv_get_steps(h, ctypes.byref(n)) == coinf.CO_EINVAL
    # a handle of another kind is rejected too
    po = coinf.CoPool("avg", batch=2, channels=8, kernel=(2, 1, 1), in_size=(4, 5),
                      stride=(1, 1, 1), dtype=torch.float32, device=DEV)
    assert coinf.co_conv_get_steps(po.handle, ctypes.byref(n)) == coinf.CO_EINVAL
    assert coinf.co_pool_get_steps(po.handle, ctypes.byref(n)) == coinf.CO_OK


def test_step_counter_limit():
    """A handle resumed just below 2^62 steps takes one more step, then every
    call that would pass the limit is rejected with the handle unchanged."""
    say("step counter limit")
    co, x = _conv(padding=(2, 1, 1))
    limit = 1 << 62
    late = coinf.CoConv(co.weight, co.bias, batch=2, in_size=(6, 7), padding=(2, 1, 1),
                        state=co.state.clone(), attach_steps=limit - 1)
    x0 = x[:, :, 0].contiguous()
    assert late.forward_step(x0) is not None                       # step 2^62 - 1 emits
    assert late.steps == limit
    with pytest.raises(RuntimeError):
        late.forward_step(x0)
    assert late.steps == limit
    back = coinf.CoConv(co.weight, co.bias, batch=2, in_size=(6, 7), padding=(2, 1, 1),
                        state=co.state.clone(), attach_steps=limit - 1)
    with pytest.raises(RuntimeError):
        back.forward_steps(x[:, :, :2].contiguous())               # would pass the limit
    assert back.steps == limit - 1
    torch.cuda.synchronize()
