"""Pins of the oracle's batch normalisation (evaluation mode) and ReLU, the
stateless modules a continual network composes with its convolutions
(section 3.2; the paper's Inception listing wraps each convolution as conv ->
BatchNorm3d -> ReLU).  Checked against PyTorch in float64, closed forms, a
conv -> BN -> ReLU chain stepped against the clip computed by PyTorch, the
identity that folding BN into a convolution's weights and bias preserves the
result, and planted mistakes that the pins must catch."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _bn_params(C, seed):
    rng = np.random.default_rng(seed)
    return (rng.normal(1.0, 0.3, C), rng.normal(0.0, 0.2, C), rng.normal(0.0, 0.5, C),
            rng.uniform(0.2, 2.0, C))


@pytest.mark.parametrize("shape", [(2, 5), (3, 4, 9), (2, 6, 5, 7), (2, 3, 4, 5, 6)])
def test_batchnorm_matches_torch(shape):
    rng = np.random.default_rng(len(shape))
    x = rng.normal(size=shape)
    g, b, m, v = _bn_params(shape[1], 3)
    bn = oracle.BatchNormEval(g, b, m, v, eps=1e-3)
    ref = F.batch_norm(torch.from_numpy(x), torch.from_numpy(m), torch.from_numpy(v),
                       torch.from_numpy(g), torch.from_numpy(b), training=False, eps=1e-3)
    np.testing.assert_allclose(bn.forward(x), ref.numpy(), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(bn.forward_step(x), ref.numpy(), rtol=1e-13, atol=1e-13)


def test_batchnorm_closed_forms():
    C = 4
    x = np.random.default_rng(1).normal(size=(2, C, 3, 3))
    # unit statistics and affine: the identity (var = 1 - eps)
    ident = oracle.BatchNormEval(np.ones(C), np.zeros(C), np.zeros(C), np.full(C, 1 - 1e-5))
    np.testing.assert_allclose(ident.forward(x), x, rtol=1e-12, atol=1e-12)
    # an input equal to the running mean maps to beta
    g, b, m, v = _bn_params(C, 2)
    xm = np.broadcast_to(m.reshape(1, C, 1, 1), x.shape)
    np.testing.assert_allclose(oracle.BatchNormEval(g, b, m, v).forward(xm),
                               np.broadcast_to(b.reshape(1, C, 1, 1), x.shape), atol=1e-12)


def test_relu_matches_torch():
    x = np.random.default_rng(5).normal(size=(3, 4, 5))
    np.testing.assert_array_equal(oracle.ReLU().forward(x), torch.relu(torch.from_numpy(x)).numpy())


def test_conv_bn_relu_chain_matches_torch_clip():
    """The chain steps through the clip; its outputs equal PyTorch's conv3d ->
    batch_norm -> relu on the clip (temporal padding 0: the outputs after the
    delay are the valid ones)."""
    rng = np.random.default_rng(11)
    B, Ci, C, T = 2, 3, 5, 7
    x = rng.normal(size=(B, Ci, T, 6, 5))
    w = rng.normal(0, 0.3, size=(C, Ci, 3, 3, 3))
    bias = rng.normal(0, 0.1, C)
    g, b, m, v = _bn_params(C, 4)
    ch = oracle.ContinualChain(oracle.ContinualConv(w, bias, padding=(0, 1, 1)),
                               oracle.BatchNormEval(g, b, m, v), oracle.ReLU())
    got = ch.forward_steps(x)
    t = lambda a: torch.from_numpy(np.asarray(a))
    ref = F.relu(F.batch_norm(F.conv3d(t(x), t(w), t(bias), padding=(0, 1, 1)), t(m), t(v), t(g),
                              t(b), training=False))
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ch.forward(x), ref.numpy(), rtol=1e-12, atol=1e-12)


def test_batchnorm_folds_into_conv_weights():
    """conv(x; W, b) followed by BN equals conv(x; W s, (b - mean) s + beta)
    with s = gamma / sqrt(var + eps) per output channel: the identity the
    library's BN-folded initialisation relies on (float64, PyTorch conv)."""
    rng = np.random.default_rng(12)
    x = rng.normal(size=(2, 4, 5, 6, 6))
    w = rng.normal(0, 0.3, size=(6, 4, 3, 3, 3))
    bias = rng.normal(0, 0.1, 6)
    g, b, m, v = _bn_params(6, 5)
    s = g / np.sqrt(v + 1e-5)
    t = lambda a: torch.from_numpy(np.asarray(a))
    direct = oracle.BatchNormEval(g, b, m, v).forward(F.conv3d(t(x), t(w), t(bias)).numpy())
    folded = F.conv3d(t(x), t(w * s.reshape(-1, 1, 1, 1, 1)), t((bias - m) * s + b)).numpy()
    np.testing.assert_allclose(folded, direct, rtol=1e-11, atol=1e-11)


class _BNsqrtMissing(oracle.BatchNormEval):
    def forward(self, x):   # planted: divides by var + eps instead of its square root
        x = np.asarray(x, dtype=np.float64)
        sh = (1, -1) + (1,) * (x.ndim - 2)
        return ((x - self.mean.reshape(sh)) / (self.var + self.eps).reshape(sh)
                * self.gamma.reshape(sh) + self.beta.reshape(sh))


class _BNaffineSwapped(oracle.BatchNormEval):
    def forward(self, x):   # planted: gamma and beta exchanged
        x = np.asarray(x, dtype=np.float64)
        sh = (1, -1) + (1,) * (x.ndim - 2)
        return ((x - self.mean.reshape(sh)) / np.sqrt(self.var + self.eps).reshape(sh)
                * self.beta.reshape(sh) + self.gamma.reshape(sh))


class _BNlastAxis(oracle.BatchNormEval):
    def forward(self, x):   # planted: normalises along the last axis instead of channels
        x = np.asarray(x, dtype=np.float64)
        return (x - self.mean) / np.sqrt(self.var + self.eps) * self.gamma + self.beta


@pytest.mark.parametrize("bad", [_BNsqrtMissing, _BNaffineSwapped, _BNlastAxis])
def test_planted_batchnorm_mistakes_fail_the_torch_pin(bad):
    C = 5
    x = np.random.default_rng(9).normal(size=(2, C, 4, C))
    g, b, m, v = _bn_params(C, 6)
    t = lambda a: torch.from_numpy(np.asarray(a))
    ref = F.batch_norm(t(x), t(m), t(v), t(g), t(b), training=False).numpy()
    assert not np.allclose(bad(g, b, m, v).forward(x), ref, rtol=1e-6, atol=1e-6)
