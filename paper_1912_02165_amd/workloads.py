"""Seeded synthetic layers shaped like the paper's VGG/ResNet 3x3 layers.

The paper benchmarks single 3x3, pad-1 layers of VGG and ResNet at batch 64
(Sec. 6).  No dataset or trained weights are involved, so the inputs here are
seeded random tensors with the same shapes:

* x ~ U[-1, 1), except the ResNet-style post-ReLU layer, where x = max(0, N(0, 1));
* w ~ N(0, std = sqrt(2 / (9 C)))  (He initialisation of a 3x3 kernel);
* NumPy ``Generator(PCG64(seed))``, drawn in float64 and rounded to float32;
  seeds are 1000 * id + 1 for x and 1000 * id + 2 for w.

This module only draws numbers; it holds none of the convolution arithmetic and
is shared by the tests, the benchmark and the smoke check.
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Layer:
    id: int
    name: str
    N: int
    C: int
    K: int
    H: int
    W: int
    ms: tuple           # Winograd output-tile sizes this layer is run with
    x_dist: str = "uniform"   # "uniform" or "relu_normal"

    @property
    def direct_flops(self):
        """2 * N * C * K * H * W * 9: multiply-adds of the direct convolution."""
        return 2.0 * self.N * self.C * self.K * self.H * self.W * 9

    def tag(self, m):
        return f"{self.name}/F({m}x{m},3x3)"


LAYERS = (
    Layer(1, "N1_C64_K64_56x56", 1, 64, 64, 56, 56, (2, 4)),
    Layer(2, "N32_C64_K64_224x224", 32, 64, 64, 224, 224, (4,)),
    Layer(3, "N32_C128_K128_112x112", 32, 128, 128, 112, 112, (4, 6)),
    Layer(4, "N64_C128_K128_28x28_relu", 64, 128, 128, 28, 28, (4,), "relu_normal"),
    Layer(5, "N64_C512_K512_14x14", 64, 512, 512, 14, 14, (6,)),
)

LAYER_BY_ID = {l.id: l for l in LAYERS}

# Every (layer, m) pair the library is checked and measured on.
PAIRS = tuple((l, m) for l in LAYERS for m in l.ms)


def draw_x(shape, seed, dist="uniform"):
    rng = np.random.Generator(np.random.PCG64(seed))
    if dist == "uniform":
        v = rng.uniform(-1.0, 1.0, size=shape)
    elif dist == "relu_normal":
        v = np.maximum(0.0, rng.standard_normal(size=shape))
    else:
        raise ValueError(dist)
    return v.astype(np.float32)


def draw_w(shape, seed):
    C = shape[1]
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.normal(0.0, np.sqrt(2.0 / (9.0 * C)), size=shape).astype(np.float32)


def layer_inputs(layer, n_images=None):
    """(x, w) float32 for ``layer``; ``n_images`` keeps only the first images of x."""
    # PCG64 draws are sequential in C order, so a shorter draw is exactly the
    # first images of the full tensor.
    N = layer.N if n_images is None else min(n_images, layer.N)
    x = draw_x((N, layer.C, layer.H, layer.W), 1000 * layer.id + 1, layer.x_dist)
    w = draw_w((layer.K, layer.C, 3, 3), 1000 * layer.id + 2)
    return x, w


def random_inputs(N, C, K, H, W, seed, dist="uniform"):
    """(x, w) for an arbitrary shape, same distributions as the layers."""
    x = draw_x((N, C, H, W), 2 * seed + 1, dist)
    w = draw_w((K, C, 3, 3), 2 * seed + 2)
    return x, w
