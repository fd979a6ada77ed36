"""Synthetic workloads for checksum-protected convolution layers.

This module is shared by the CPU oracle, the tests and the benchmark.  It
holds only layer shapes and seeded random draws; it contains none of the
protection method's arithmetic (no convolution, no checksum, no threshold).

Layer shapes follow the networks the paper evaluates (Sec. 6, "CNN models and
dataset": AlexNet, VGG-19, ResNet-18 and YOLOv2), each layer taken in
isolation with a fresh input at its own input shape.  The paper measures on
the ImageNet validation set with pretrained models; neither is available, so
seeded synthetic tensors with the layer's shape stand in for both:

* feature maps ``D`` are drawn from U(0, 1) (a non-negative stand-in for
  post-activation maps), except the tiny single-layer case, which uses N(0, 1);
* kernels ``W`` are He-normal, standard deviation sqrt(2 / (Ch*R*S)), except
  the tiny case, which uses N(0, 1/27);
* bf16 tensors are the fp32 draw rounded once to bf16 (round to nearest even),
  so both sides of any comparison consume identical bits.

Random streams are ``numpy.random.Generator(PCG64(SeedSequence([12203, cfg,
layer, tensor])))`` with tensor ids 0 = D, 1 = W, 2 = fault draws.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

SEED_ROOT = 12203
T_D, T_W, T_FAULT = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class LayerSpec:
    """Shape of one convolution layer: D[n][ch][h][w] (x) W[m][ch][r][s]."""
    name: str
    n: int
    ch: int
    h: int
    w: int
    m: int
    r: int
    s: int
    stride: int
    pad: int
    dtype: str  # "f32" or "bf16"

    def with_(self, **kw) -> "LayerSpec":
        return dataclasses.replace(self, **kw)


@dataclasses.dataclass(frozen=True)
class Config:
    cid: int
    name: str
    layers: tuple
    d_dist: str  # "uniform" or "normal"
    w_dist: str  # "he" or "tiny"


def _sq(name, n, ch, hw, m, rs, u, p, dt):
    return LayerSpec(name, n, ch, hw, hw, m, rs, rs, u, p, dt)


def _tiny() -> Config:
    return Config(0, "tiny", (_sq("c", 4, 3, 32, 16, 3, 1, 1, "f32"),), "normal", "tiny")


def _alexnet() -> Config:
    n = 64
    layers = (
        _sq("conv1", n, 3, 227, 96, 11, 4, 0, "f32"),
        _sq("conv2", n, 96, 27, 256, 5, 1, 2, "f32"),
        _sq("conv3", n, 256, 13, 384, 3, 1, 1, "f32"),
        _sq("conv4", n, 384, 13, 384, 3, 1, 1, "f32"),
        _sq("conv5", n, 384, 13, 256, 3, 1, 1, "f32"),
    )
    return Config(1, "alexnet", layers, "uniform", "he")


def _vgg19(dtype: str) -> Config:
    n = 32
    plan = [(3, 64, 224), (64, 64, 224), (64, 128, 112), (128, 128, 112),
            (128, 256, 56), (256, 256, 56), (256, 256, 56), (256, 256, 56),
            (256, 512, 28), (512, 512, 28), (512, 512, 28), (512, 512, 28),
            (512, 512, 14), (512, 512, 14), (512, 512, 14), (512, 512, 14)]
    layers = tuple(_sq(f"v{i + 1}", n, c, hw, m, 3, 1, 1, dtype)
                   for i, (c, m, hw) in enumerate(plan))
    return Config(2, "vgg19" + ("" if dtype == "f32" else "_bf16"), layers, "uniform", "he")


def _resnet18() -> Config:
    n, dt = 128, "bf16"
    L = [_sq("stem", n, 3, 224, 64, 7, 2, 3, dt)]
    L += [_sq(f"l1.{i}", n, 64, 56, 64, 3, 1, 1, dt) for i in range(4)]
    for stage, (cin, cout, hin) in enumerate([(64, 128, 56), (128, 256, 28), (256, 512, 14)], start=2):
        L.append(_sq(f"l{stage}.down", n, cin, hin, cout, 3, 2, 1, dt))
        L.append(_sq(f"l{stage}.proj", n, cin, hin, cout, 1, 2, 0, dt))
        L += [_sq(f"l{stage}.{i}", n, cout, hin // 2, cout, 3, 1, 1, dt) for i in range(3)]
    return Config(3, "resnet18", tuple(L), "uniform", "he")


def _darknet19() -> Config:
    n, dt = 16, "f32"
    plan = [(3, 32, 416, 3), (32, 64, 208, 3),
            (64, 128, 104, 3), (128, 64, 104, 1), (64, 128, 104, 3),
            (128, 256, 52, 3), (256, 128, 52, 1), (128, 256, 52, 3),
            (256, 512, 26, 3), (512, 256, 26, 1), (256, 512, 26, 3), (512, 256, 26, 1), (256, 512, 26, 3),
            (512, 1024, 13, 3), (1024, 512, 13, 1), (512, 1024, 13, 3), (1024, 512, 13, 1), (512, 1024, 13, 3)]
    layers = tuple(_sq(f"c{i + 1}", n, c, hw, m, r, 1, r // 2, dt)
                   for i, (c, m, hw, r) in enumerate(plan))
    return Config(4, "darknet19", layers, "uniform", "he")


def configs() -> List[Config]:
    """The five workloads, in order: tiny, AlexNet, VGG-19 (fp32), ResNet-18, Darknet-19.

    VGG-19 also runs in bf16; ``vgg19_bf16()`` returns that variant.
    """
    return [_tiny(), _alexnet(), _vgg19("f32"), _resnet18(), _darknet19()]


def vgg19_bf16() -> Config:
    return _vgg19("bf16")


def config(cid: int) -> Config:
    return configs()[cid]


def rng(cid: int, layer: int, tensor: int, extra: int = 0) -> np.random.Generator:
    words = [SEED_ROOT, cid, layer, tensor] + ([extra] if extra else [])
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(words)))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(x)
    rounded = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    if nan.any():
        rounded[nan] = 0x7FC0
    return rounded


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def gen_d(cfg: Config, li: int, spec: Optional[LayerSpec] = None) -> np.ndarray:
    """Feature map D[n][ch][h][w] as float32 (already bf16-representable for bf16 layers)."""
    spec = spec or cfg.layers[li]
    g = rng(cfg.cid, li, T_D)
    shape = (spec.n, spec.ch, spec.h, spec.w)
    if cfg.d_dist == "normal":
        x = g.standard_normal(shape, dtype=np.float32)
    else:
        x = g.random(shape, dtype=np.float32)
    if spec.dtype == "bf16":
        x = bf16_bits_to_f32(f32_to_bf16_bits(x)).reshape(shape)
    return x


def gen_w(cfg: Config, li: int, spec: Optional[LayerSpec] = None) -> np.ndarray:
    """Kernels W[m][ch][r][s] as float32 (bf16-representable for bf16 layers)."""
    spec = spec or cfg.layers[li]
    g = rng(cfg.cid, li, T_W)
    shape = (spec.m, spec.ch, spec.r, spec.s)
    if cfg.w_dist == "tiny":
        std = np.float32(np.sqrt(1.0 / 27.0))
    else:
        std = np.float32(np.sqrt(2.0 / (spec.ch * spec.r * spec.s)))
    x = g.standard_normal(shape, dtype=np.float32) * std
    if spec.dtype == "bf16":
        x = bf16_bits_to_f32(f32_to_bf16_bits(x)).reshape(shape)
    return x


def gen_int_d(spec: LayerSpec, seed: int, hi: int = 3) -> np.ndarray:
    """Integer-valued feature map in {0..hi}: every fp32 sum of products stays exact."""
    g = rng(99, seed, T_D)
    return g.integers(0, hi + 1, size=(spec.n, spec.ch, spec.h, spec.w)).astype(np.float32)


def gen_int_w(spec: LayerSpec, seed: int, lim: int = 2) -> np.ndarray:
    """Integer-valued kernels in {-lim..lim}."""
    g = rng(99, seed, T_W)
    return g.integers(-lim, lim + 1, size=(spec.m, spec.ch, spec.r, spec.s)).astype(np.float32)


def fault_draws(cid: int, li: int, count: int, variant: int = 0) -> np.ndarray:
    """``count`` rows of seven U(0,1) draws for the fault harness to interpret.

    Columns: position (n, m, x, y) selectors, bit/kind selector, magnitude,
    sign.  The harness maps them onto concrete faults.
    """
    g = rng(cid, li, T_FAULT, variant)
    return g.random((count, 7))
