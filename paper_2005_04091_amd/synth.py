"""Seeded synthetic layers for the fused sparse convolution.

This module only draws random inputs; it holds none of the convolution's
arithmetic, so both the GPU path's tests/benchmark and the CPU oracle can be fed
from it. The paper evaluates on pruned VGG-16 / ResNet-20 blocks (section
"Evaluation"; layer densities in Table 1), which are not available here: these
layers stand in for them with Bernoulli weight masks at the densities of that
table's range.

Draw order for one layer, from ``numpy.random.default_rng(seed)``: per-row
densities (skewed layers only) -> mask -> weight values -> input -> bias.
Distributions: mask Bernoulli(d), weights U[-1, 1), input U[0, 1), bias
U[-0.1, 0.1).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 409100


@dataclass
class Layer:
    """One synthetic conv layer: NCHW input, masked KCRS filter, bias and flags."""
    name: str
    x: np.ndarray            # [N, C, H, W] float32
    w: np.ndarray            # [K, C, R, S] float32, zero where mask is 0
    mask: np.ndarray         # [K, C, R, S] uint8
    bias: np.ndarray | None  # [K] float32
    stride: int = 1
    pad: int = 1
    relu: bool = True
    pool: bool = False
    meta: dict = field(default_factory=dict)

    @property
    def shape(self):
        N, C, H, W = self.x.shape
        K, _, R, S = self.w.shape
        return N, C, H, W, K, R, S


# Named layers (all 3x3, stride 1, pad 1, fused bias + ReLU; 'pool' adds the 2x2 max-pool).
CONFIGS = {
    "tiny":      dict(N=1, C=16, K=16, H=16, W=16, density=0.2, pool=False, seed=SEED_BASE + 1),
    "resnet":    dict(N=32, C=64, K=64, H=56, W=56, density=0.2, pool=False, seed=SEED_BASE + 2),
    "conv_pool": dict(N=32, C=128, K=128, H=28, W=28, density=0.1, pool=True, seed=SEED_BASE + 3),
    "narrow_d0.05": dict(N=32, C=256, K=256, H=14, W=14, density=0.05, pool=False, skew=True, seed=SEED_BASE + 40),
    "narrow_d0.2":  dict(N=32, C=256, K=256, H=14, W=14, density=0.2, pool=False, skew=True, seed=SEED_BASE + 41),
    "narrow_d0.5":  dict(N=32, C=256, K=256, H=14, W=14, density=0.5, pool=False, skew=True, seed=SEED_BASE + 42),
}

# The VGG-style block: two chained 3x3 layers at 224x224 (the second one pooled).
VGG_BLOCK = dict(N=32, C_real=3, C=64, K=64, H=224, W=224, density=0.2, seed=SEED_BASE + 5)


def _row_densities(rng, K: int, target: float) -> np.ndarray:
    """Per-output-channel densities: Beta(2, 5) draws rescaled so their mean
    (2/7) maps to ``target``, clipped at 1."""
    b = rng.beta(2.0, 5.0, size=K)
    return np.minimum(1.0, b * (target / (2.0 / 7.0)))


def _mask(rng, K, C, R, S, density) -> np.ndarray:
    d = np.asarray(density, dtype=np.float64)
    if d.ndim == 1:
        d = d[:, None, None, None]
    return (rng.random((K, C, R, S)) < d).astype(np.uint8)


def _weights(rng, mask) -> np.ndarray:
    vals = rng.uniform(-1.0, 1.0, size=mask.shape).astype(np.float32)
    return np.where(mask != 0, vals, np.float32(0.0)).astype(np.float32)


def _input(rng, N, C, H, W) -> np.ndarray:
    return rng.random((N, C, H, W), dtype=np.float32)


def _bias(rng, K) -> np.ndarray:
    return rng.uniform(-0.1, 0.1, size=K).astype(np.float32)


def make_layer(name: str) -> Layer:
    """The named synthetic layer (see ``CONFIGS``)."""
    cfg = CONFIGS[name]
    rng = np.random.default_rng(cfg["seed"])
    N, C, K, H, W = cfg["N"], cfg["C"], cfg["K"], cfg["H"], cfg["W"]
    R = S = 3
    density = cfg["density"]
    meta = {"target_density": density}
    if cfg.get("skew"):
        dk = _row_densities(rng, K, density)
        meta["row_density_mean"] = float(dk.mean())
        density = dk
    mask = _mask(rng, K, C, R, S, density)
    w = _weights(rng, mask)
    x = _input(rng, N, C, H, W)
    b = _bias(rng, K)
    return Layer(name, x, w, mask, b, stride=1, pad=1, relu=True, pool=cfg["pool"], meta=meta)


def make_vgg_block():
    """Input and the two layers of the VGG-style block.

    The block input has 3 real channels zero-padded to 64 (channels 3..63 are 0).
    Returns ``(x, layer1, layer2)``; each layer's ``x`` is the block input for
    layer 1 and, for layer 2, a seeded U[0, 1) tensor of layer 2's input shape
    (used when layer 2 is exercised on its own; in the chained block it reads
    layer 1's output instead).
    """
    cfg = VGG_BLOCK
    rng = np.random.default_rng(cfg["seed"])
    N, C, K, H, W, d = cfg["N"], cfg["C"], cfg["K"], cfg["H"], cfg["W"], cfg["density"]
    m1 = _mask(rng, K, C, 3, 3, d)
    m2 = _mask(rng, K, K, 3, 3, d)
    w1 = _weights(rng, m1)
    w2 = _weights(rng, m2)
    x = np.zeros((N, C, H, W), np.float32)
    x[:, :cfg["C_real"]] = _input(rng, N, cfg["C_real"], H, W)
    b1 = _bias(rng, K)
    b2 = _bias(rng, K)
    x2 = _input(rng, N, K, H, W)
    l1 = Layer("vgg_conv1", x, w1, m1, b1, stride=1, pad=1, relu=True, pool=False)
    l2 = Layer("vgg_conv2_pool", x2, w2, m2, b2, stride=1, pad=1, relu=True, pool=True)
    return x, l1, l2


# A ResNet basic block at the ResNet layer's shape: relu(conv2(relu(conv1(x))) + x).
RESNET_BLOCK = dict(N=32, C=64, H=56, W=56, density=0.2, seed=SEED_BASE + 6)


def make_resnet_block():
    """Input and the two layers of a ResNet basic block (the shortcut is the
    block input, added before the second layer's ReLU). Draw order: mask 1,
    mask 2, weights 1, weights 2, input, bias 1, bias 2. Returns ``(x, layer1,
    layer2)``; layer 2's ``x`` is a seeded U[0, 1) tensor of its input shape."""
    cfg = RESNET_BLOCK
    rng = np.random.default_rng(cfg["seed"])
    N, C, H, W, d = cfg["N"], cfg["C"], cfg["H"], cfg["W"], cfg["density"]
    m1 = _mask(rng, C, C, 3, 3, d)
    m2 = _mask(rng, C, C, 3, 3, d)
    w1 = _weights(rng, m1)
    w2 = _weights(rng, m2)
    x = _input(rng, N, C, H, W)
    b1 = _bias(rng, C)
    b2 = _bias(rng, C)
    x2 = _input(rng, N, C, H, W)
    l1 = Layer("resnet_block_conv1", x, w1, m1, b1, stride=1, pad=1, relu=True, pool=False)
    l2 = Layer("resnet_block_conv2", x2, w2, m2, b2, stride=1, pad=1, relu=True, pool=False)
    return x, l1, l2


# Resize-Conv-ReLU-Maxpool: the Conv-ReLU-Maxpool layer (28x28, C=K=128, density
# 0.1, pool to 14x14) fed by a bilinear resize of a 42x42 source (a 1.5x
# downscale, so every output pixel interpolates between two source pixels on
# each axis, at fractions 1/4 and 3/4).
RESIZE_BLOCK = dict(N=32, C=128, K=128, Hin=42, Win=42, H=28, W=28, density=0.1, seed=SEED_BASE + 7)


def make_resize_block():
    """Source image batch and the layer of the Resize-Conv-ReLU-Maxpool block.
    Draw order: mask, weights, source, bias. Returns ``(src, layer)``; the
    layer's ``x`` is a seeded U[0, 1) tensor of its own input shape (for the
    layer alone; in the block it reads the resized source)."""
    cfg = RESIZE_BLOCK
    rng = np.random.default_rng(cfg["seed"])
    N, C, K, H, W, d = cfg["N"], cfg["C"], cfg["K"], cfg["H"], cfg["W"], cfg["density"]
    m = _mask(rng, K, C, 3, 3, d)
    w = _weights(rng, m)
    src = _input(rng, N, C, cfg["Hin"], cfg["Win"])
    b = _bias(rng, K)
    x = _input(rng, N, C, H, W)
    return src, Layer("resize_conv_relu_maxpool", x, w, m, b, stride=1, pad=1, relu=True, pool=True)


def random_layer(seed: int, N: int, C: int, K: int, H: int, W: int, R: int = 3, S: int = 3, stride: int = 1,
                 pad: int = 1, density: float = 0.2, relu: bool = True, pool: bool = False, bias: bool = True,
                 skew: bool = False) -> Layer:
    """A small seeded layer with the same distributions, for shape sweeps."""
    rng = np.random.default_rng(seed)
    d = _row_densities(rng, K, density) if skew else density
    mask = _mask(rng, K, C, R, S, d)
    w = _weights(rng, mask)
    x = _input(rng, N, C, H, W)
    b = _bias(rng, K) if bias else None
    return Layer(f"random_{seed}", x, w, mask, b, stride=stride, pad=pad, relu=relu, pool=pool)
