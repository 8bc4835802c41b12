"""Workload definitions and seeded synthetic inputs.

This module holds no convolution or halo arithmetic: it only names the layer
shapes that are run and draws their input tensors.  It is shared by the test
suite, the benchmark and the smoke check, and feeds both the GPU library and
the CPU oracle with bit-identical values.

Shapes follow the paper's workloads (Dryden et al., Sec. VI): ResNet-50 layers
on 224x224x3 ImageNet-sized samples, and the 2048x2048x18 mesh-tangling
samples in fp32.  Neither dataset is available, so every tensor is drawn from
a seeded generator with the stated distribution (the paper itself benchmarks
the mesh model on synthetic data).

Seeding: workload ``seed``; tensor t (x=0, w=1, dy=2) of sub-layer ``sub``
draws from ``np.random.default_rng(SeedSequence([seed, sub, t]))``.  Uniform
values are ``rng.uniform(-1, 1)``, Gaussian ones ``rng.standard_normal()``,
both cast to fp32; bf16 workloads then round each fp32 value to bf16 with
round-to-nearest-even, and the rounded values (widened back, exactly, to fp32)
are what the oracle sees.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    N: int
    C: int
    K: int
    H: int          # global input height
    W: int          # global input width
    R: int
    S: int
    stride: int
    pad: int
    P: int          # spatial grid rows
    Q: int          # spatial grid cols
    halo: int       # margin width on every side of every tile
    dtype: str      # "f32" or "bf16": dtype of x, w, dy
    dist: str       # "uniform" or "normal"
    seed: int
    sub: int = 0
    tiles: tuple = ()   # tiles checked at full size (row-major index); () = all
    desc: str = ""

    @property
    def Ht(self):
        return self.H // self.P

    @property
    def Wt(self):
        return self.W // self.Q

    @property
    def Ho(self):
        return (self.H + 2 * self.pad - self.R) // self.stride + 1

    @property
    def Wo(self):
        return (self.W + 2 * self.pad - self.S) // self.stride + 1

    @property
    def Hot(self):
        return self.Ho // self.P

    @property
    def Wot(self):
        return self.Wo // self.Q

    def flops_per_pass_tile(self) -> int:
        return 2 * self.N * self.K * self.C * self.R * self.S * self.Hot * self.Wot


LAYERS = {
    # 1: a single undecomposed 3x3 layer, fp32
    "c1": Layer("c1", 1, 4, 4, 32, 32, 3, 3, 1, 1, 1, 1, 1, "f32", "uniform", 1000,
                desc="3x3 s1 p1, N=1, C=K=4, 32x32, fp32, no decomposition"),
    # 2: the same conv on a 2x2 grid of 16x16 tiles, fp32
    "c2": Layer("c2", 2, 8, 8, 32, 32, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 1001,
                desc="3x3 s1 p1, N=2, C=K=8, 32x32 on a 2x2 grid (16x16 tiles), h=1, fp32"),
    # 3: ResNet-50 layer shapes at N=32, bf16 inputs
    "c3a": Layer("c3a", 32, 3, 64, 224, 224, 7, 7, 2, 3, 1, 1, 3, "bf16", "uniform", 1002, 0,
                 desc="ResNet-50 conv1: 7x7 s2 p3, C=3->K=64, 224x224, N=32, bf16"),
    "c3b": Layer("c3b", 32, 64, 64, 56, 56, 3, 3, 1, 1, 1, 1, 1, "bf16", "uniform", 1002, 1,
                 desc="ResNet-50 3x3 s1 p1, C=K=64, 56x56, N=32, bf16"),
    "c3c": Layer("c3c", 32, 256, 64, 56, 56, 1, 1, 1, 0, 1, 1, 0, "bf16", "uniform", 1002, 2,
                 desc="ResNet-50 1x1, C=256->K=64, 56x56, N=32, bf16"),
    # 4: one 512x512 tile of a 2048x2048x18 mesh sample on a 4x4 grid, fp32
    "c4": Layer("c4", 1, 18, 32, 2048, 2048, 3, 3, 1, 1, 4, 4, 1, "f32", "normal", 1003,
                tiles=(5, 0),
                desc="mesh-2K-like 3x3 s1 p1, C=18->K=32, 512x512 tile of 2048x2048 (4x4 grid), h=1, fp32"),
    # 5: hybrid sample+spatial: N=4 per GPU, one 256x256 tile of 1024x1024 on a 4x4 grid, bf16
    "c5a": Layer("c5a", 4, 64, 64, 1024, 1024, 3, 3, 1, 1, 4, 4, 1, "bf16", "uniform", 1004, 0,
                 tiles=(5, 0),
                 desc="3x3 s1 p1, C=K=64, N=4, 256x256 tile of 1024x1024 (4x4 grid), h=1, bf16"),
    "c5b": Layer("c5b", 4, 32, 32, 1024, 1024, 5, 5, 1, 2, 4, 4, 2, "bf16", "uniform", 1004, 1,
                 tiles=(5, 0),
                 desc="5x5 s1 p2, C=K=32, N=4, 256x256 tile of 1024x1024 (4x4 grid), h=2, bf16"),
    # decomposed stride-2 layers (Sec. III-A: one-sided halos at stride > 1)
    "c3a_2x2": Layer("c3a_2x2", 32, 3, 64, 224, 224, 7, 7, 2, 3, 2, 2, 3, "bf16", "uniform", 1002, 3,
                     tiles=(3, 0),
                     desc="ResNet-50 conv1 7x7 s2 p3, C=3->K=64, 224x224 on a 2x2 grid (112x112 tiles, "
                          "56x56 outputs), h=3, N=32, bf16"),
    "c4s2": Layer("c4s2", 1, 32, 32, 2048, 2048, 3, 3, 2, 1, 4, 4, 1, "f32", "normal", 1003, 1,
                  tiles=(5, 0),
                  desc="mesh-2K-like stride-2 3x3 p1 block entry, C=K=32, 512x512 tile of 2048x2048 "
                       "(4x4 grid, 256x256 outputs), h=1, fp32"),
}

# The layer the benchmark times: the largest conv tile by flops and bytes.
BENCH_LAYER = "c5a"


def _rng(seed: int, sub: int, t: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, sub, t]))


def _draw(rng, shape, dist):
    if dist == "uniform":
        return rng.uniform(-1.0, 1.0, size=shape).astype(np.float32)
    if dist == "normal":
        return rng.standard_normal(size=shape, dtype=np.float32)
    if dist == "int":
        return rng.integers(-2, 3, size=shape).astype(np.float32)
    raise ValueError(dist)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 -> nearest-even bf16 -> fp32 (exact widening)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).to(torch.float32).numpy()


def draw(layer: Layer, which: str, dist: str | None = None) -> np.ndarray:
    """Global tensor 'x' [N,C,H,W], 'w' [K,C,R,S] or 'dy' [N,K,Ho,Wo] (fp32 values,
    already bf16-representable for bf16 layers)."""
    shapes = {"x": (layer.N, layer.C, layer.H, layer.W),
              "w": (layer.K, layer.C, layer.R, layer.S),
              "dy": (layer.N, layer.K, layer.Ho, layer.Wo)}
    t = {"x": 0, "w": 1, "dy": 2}[which]
    a = _draw(_rng(layer.seed, layer.sub, t), shapes[which], dist or layer.dist)
    if layer.dtype == "bf16":
        a = round_to_bf16(a)
    return a


def small(name: str, **kw) -> Layer:
    """A copy of a layer with some fields replaced (for reduced-size cases)."""
    return dataclasses.replace(LAYERS[name], **kw)
