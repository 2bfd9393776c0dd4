"""Seeded synthetic inputs and the named workloads.

This module only draws random numbers and describes shapes.  It holds none of
the method's arithmetic, so both the oracle-based tests and the HIP path can
take their inputs from it.

The streams stand in for the paper's video (X3D-like 3D CNN blocks on
Kinetics-400), skeleton (ST-GCN-like temporal convolution on NTU RGB+D 60,
T = 300 frames of V = 25 joints) and 1-D signal workloads: the datasets and
trained weights are not used.  Frames are i.i.d. N(0, 1); the kernels are
data-oblivious, so the distribution affects numerics only, never cost.

Draws are float32 from ``torch.Generator('cpu')`` seeded per workload number
c = 1..5 (in the order listed below; both skeleton precisions share 5): x with
``1000*c + 0``, weights ``1000*c + 1``, bias ``1000*c + 2``.  bfloat16
workloads round the float32 draws to nearest-even on the host, so the oracle
and the GPU consume identical values.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class ConvSpec:
    """One continual convolution layer (kernel/stride/padding/dilation time first)."""
    batch: int
    in_channels: int
    out_channels: int
    kernel: tuple
    in_size: tuple = ()            # spatial sizes (S1[, S2]); () for Conv1d
    stride: tuple = None
    padding: tuple = None
    dilation: tuple = None
    groups: int = 1
    bias: bool = True
    dtype: str = "f32"             # "f32" | "bf16"

    def __post_init__(self):
        nd = 1 + len(self.in_size)
        assert len(self.kernel) == nd
        for name, fill in (("stride", 1), ("padding", 0), ("dilation", 1)):
            if getattr(self, name) is None:
                object.__setattr__(self, name, (fill,) * nd)

    @property
    def spatial_dims(self):
        return len(self.in_size)

    @property
    def weight_shape(self):
        return (self.out_channels, self.in_channels // self.groups) + tuple(self.kernel)


@dataclass(frozen=True)
class PoolSpec:
    """One continual pooling layer."""
    kind: str                      # "avg" | "max"
    batch: int
    channels: int
    kernel: tuple
    in_size: tuple = ()
    stride: tuple = None
    padding: tuple = None
    dilation: tuple = None
    count_include_pad: bool = True
    dtype: str = "f32"

    def __post_init__(self):
        nd = 1 + len(self.in_size)
        assert len(self.kernel) == nd
        if self.stride is None:
            object.__setattr__(self, "stride", tuple(self.kernel))
        if self.padding is None:
            object.__setattr__(self, "padding", (0,) * nd)
        if self.dilation is None:
            object.__setattr__(self, "dilation", (1,) * nd)

    @property
    def spatial_dims(self):
        return len(self.in_size)


@dataclass(frozen=True)
class Workload:
    name: str
    index: int                     # workload number 1..5; seed base 1000 * index
    frames: int                    # T of the synthetic clip
    conv: ConvSpec
    pool: PoolSpec = None
    weight_init: str = "kaiming"   # "kaiming" | "normal"
    note: str = ""


WORKLOADS = {
    w.name: w for w in [
        Workload(
            name="conv1d_b1_c4to8_k3_f32", index=1, frames=64,
            conv=ConvSpec(batch=1, in_channels=4, out_channels=8, kernel=(3,), dtype="f32"),
            weight_init="normal",
            note="CoConv1d single stream, 1-D signal"),
        Workload(
            name="conv3d_b1_c24_k3_56x56_f32", index=2, frames=16,
            conv=ConvSpec(batch=1, in_channels=24, out_channels=24, kernel=(3, 3, 3),
                          in_size=(56, 56), padding=(0, 1, 1), dtype="f32"),
            note="CoConv3d single stream, X3D-S-like stem block"),
        Workload(
            name="conv3d_b64_c192_k3_14x14_bf16", index=3, frames=32,
            conv=ConvSpec(batch=64, in_channels=192, out_channels=192, kernel=(3, 3, 3),
                          in_size=(14, 14), padding=(0, 1, 1), dtype="bf16"),
            note="CoConv3d, 64 independent streams"),
        Workload(
            name="dwconv3d_b16_c432_k3_7x7_avgpool_bf16", index=4, frames=64,
            conv=ConvSpec(batch=16, in_channels=432, out_channels=432, kernel=(3, 3, 3),
                          in_size=(7, 7), padding=(0, 1, 1), groups=432, dtype="bf16"),
            pool=PoolSpec(kind="avg", batch=16, channels=432, kernel=(4, 7, 7),
                          in_size=(7, 7), stride=(1, 7, 7), dtype="bf16"),
            note="X3D-style depthwise CoConv3d followed by continual AvgPool3d (4,7,7)"),
        Workload(
            name="conv2d_b32_c64to256_k9x1_v25_f32", index=5, frames=300,
            conv=ConvSpec(batch=32, in_channels=64, out_channels=256, kernel=(9, 1),
                          in_size=(25,), dtype="f32"),
            note="ST-GCN-like temporal conv over T=300 frames of V=25 joints (fp32)"),
        Workload(
            name="conv2d_b32_c64to256_k9x1_v25_bf16", index=5, frames=300,
            conv=ConvSpec(batch=32, in_channels=64, out_channels=256, kernel=(9, 1),
                          in_size=(25,), dtype="bf16"),
            note="ST-GCN-like temporal conv over T=300 frames of V=25 joints (bf16)"),
    ]
}


def torch_dtype(name: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def normal(shape, seed: int, std: float = 1.0, dtype: str = "f32") -> torch.Tensor:
    """float32 N(0, std^2) draws on the CPU, rounded to ``dtype`` (RNE for bf16)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    t = torch.randn(tuple(shape), generator=g, dtype=torch.float32) * std
    return t.to(torch_dtype(dtype)).contiguous()


def kaiming_std(weight_shape) -> float:
    """PyTorch's kaiming_normal_ default: fan_in mode, ReLU gain sqrt(2)."""
    fan_in = 1
    for s in weight_shape[1:]:
        fan_in *= s
    return math.sqrt(2.0 / fan_in)


def conv_inputs(spec: ConvSpec, frames: int, seed_base: int, weight_init: str = "kaiming"):
    """(x clip (B, C_in, T, *S), weight, bias or None), CPU tensors in spec.dtype."""
    x = normal((spec.batch, spec.in_channels, frames) + tuple(spec.in_size), seed_base + 0,
               dtype=spec.dtype)
    std = kaiming_std(spec.weight_shape) if weight_init == "kaiming" else 1.0
    w = normal(spec.weight_shape, seed_base + 1, std=std, dtype=spec.dtype)
    b = normal((spec.out_channels,), seed_base + 2, std=0.1, dtype=spec.dtype) if spec.bias else None
    return x, w, b


def pool_inputs(spec: PoolSpec, frames: int, seed_base: int):
    return normal((spec.batch, spec.channels, frames) + tuple(spec.in_size), seed_base + 0,
                  dtype=spec.dtype)


def workload_inputs(name: str):
    """Inputs of a named workload (seeds 1000*index + {0, 1, 2})."""
    w = WORKLOADS[name]
    return conv_inputs(w.conv, w.frames, 1000 * w.index, w.weight_init)


@dataclass(frozen=True)
class BottleneckSpec:
    """The front of an X3D bottleneck block: pointwise conv + BN + ReLU,
    depthwise CoConv3d + BN + ReLU, continual average pool over the plane."""
    name: str
    batch: int
    in_channels: int
    channels: int
    in_size: tuple
    kernel: tuple        # depthwise kernel, time first
    padding: tuple       # depthwise padding, time first
    pool_kernel: tuple   # (kT, H, W) over the depthwise output plane
    frames: int
    seed: int
    dtype: str = "bf16"


# X3D-M's last stage at 7x7 (192 channels in, expanded to 432), the same
# depthwise and pool shapes as the depthwise workload, 16 streams.
BOTTLENECK = BottleneckSpec(name="bneck_b16_c192to432_k3_7x7_avgpool_bf16", batch=16,
                            in_channels=192, channels=432, in_size=(7, 7), kernel=(3, 3, 3),
                            padding=(0, 1, 1), pool_kernel=(4, 7, 7), frames=16, seed=6000)


def bottleneck_inputs(spec: BottleneckSpec = BOTTLENECK):
    """CPU tensors: x (B, C_in, T, H, W); pointwise weight (C, C_in, 1, 1, 1)
    and bias; depthwise weight (C, 1, kT, kH, kW); two sets of evaluation
    statistics (gamma, beta, mean, var) as float32.  Seeds spec.seed + i."""
    s0, dt = spec.seed, spec.dtype
    C = spec.channels
    x = normal((spec.batch, spec.in_channels, spec.frames) + tuple(spec.in_size), s0, dtype=dt)
    w1_shape = (C, spec.in_channels, 1, 1, 1)
    w1 = normal(w1_shape, s0 + 1, std=kaiming_std(w1_shape), dtype=dt)
    b1 = normal((C,), s0 + 2, std=0.1, dtype=dt)
    w2_shape = (C, 1) + tuple(spec.kernel)
    w2 = normal(w2_shape, s0 + 3, std=kaiming_std(w2_shape), dtype=dt)

    def stats(k):
        return (1.0 + 0.1 * normal((C,), k), 0.1 * normal((C,), k + 1),
                0.1 * normal((C,), k + 2), 0.5 + normal((C,), k + 3).abs())

    return x, w1, b1, w2, stats(s0 + 10), stats(s0 + 20)
