"""The parity measure itself (tests/parity_util.py), on the CPU: the
elementwise bound catches a bias-sized slip on one output channel of a
64-stream-sized bf16 layer that the normwise bound alone lets through, and
accepts the rounding a correct bf16 result carries."""
import numpy as np
import pytest
import torch

from parity_util import TOL, elementwise_excess, relerr


def _ref(shape=(4, 192, 3, 14, 14), seed=11):
    rng = np.random.default_rng(seed)
    # outputs of a 5185-term bf16 convolution: about N(0, 1.4^2)
    return rng.normal(0.0, 1.4, shape)


def test_bias_slip_on_one_channel_is_caught():
    ref = _ref()
    got = ref.copy()
    got[:, 17] += 0.1                      # one output channel off by a bias-sized 0.1
    assert relerr(got, ref) <= TOL[torch.bfloat16]   # the normwise bound lets it pass
    r, _, _, _ = elementwise_excess(got, ref, torch.bfloat16, terms=5185)
    assert r > 1.0


def test_correct_bf16_rounding_passes():
    ref = _ref()
    got = torch.from_numpy(ref).to(torch.bfloat16).double().numpy()   # rounded once (RNE)
    r, _, _, _ = elementwise_excess(got, ref, torch.bfloat16, terms=5185)
    assert r <= 1.0            # half an ulp is at most 2^-8 |o|, the rtol allowance


@pytest.mark.parametrize("terms", [4, 28, 649, 5185])
def test_float32_accumulation_within_bound(terms):
    """A float32 sum of `terms` random products against float64: inside the
    bound, with room to spare."""
    rng = np.random.default_rng(terms)
    a = rng.normal(size=(2000, terms)).astype(np.float32)
    b = rng.normal(size=(2000, terms)).astype(np.float32) / np.sqrt(terms)
    ref = (a.astype(np.float64) * b.astype(np.float64)).sum(axis=1)
    acc = np.zeros(2000, dtype=np.float32)
    for k in range(terms):                 # sequential float32 accumulation
        acc = (acc + a[:, k] * b[:, k]).astype(np.float32)
    r, _, _, _ = elementwise_excess(acc.astype(np.float64), ref, torch.float32, terms=terms)
    assert r <= 0.5
