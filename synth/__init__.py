"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark.

This module only draws random numbers and lays them out; it holds none of the
kernel-quantization arithmetic (no distances, means, quantizers or packing).

The paper quantizes the 3x3 convolution kernels of ImageNet-trained VGG-16 and
ResNet-18 models (Sec. 4.1).  Those weights are not available here, so layers
of the same shapes are drawn from Kaiming-style distributions instead:

* VGG-16-shaped stack: 13 layers, weights ~ N(0, sigma), sigma = sqrt(2 / (9 C_in)).
* ResNet-18-shaped stack: 16 layers, weights ~ Laplace(0, sigma / sqrt(2))
  (same variance as the normal above).
* Stress layer: 1024 x 1024 kernels drawn from a mixture of 4096 Gaussian
  clusters in R^9 (centres ~ N(0, 1), within-cluster std 0.1).

Each layer's weight tensor is OIHW, so kernel i = o * C_in + c and the 9 values
of a kernel are contiguous (Sec. 3.1 reshapes the weight tensor into n = p q
kernels of omega^2 values).

The initial codebook is k distinct kernels of the layer picked in a seeded
random order (the paper does not say how k-means is initialised).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

DIM = 9  # omega^2 for 3x3 kernels

# (C_in, C_out) of the 3x3 convolutions of VGG-16 (13 layers).
VGG16_LAYERS = [(3, 64), (64, 64), (64, 128), (128, 128), (128, 256), (256, 256), (256, 256),
                (256, 512), (512, 512), (512, 512), (512, 512), (512, 512), (512, 512)]
# (C_in, C_out) of the 3x3 convolutions of ResNet-18 (16 layers).
RESNET18_LAYERS = [(64, 64)] * 4 + [(64, 128)] + [(128, 128)] * 3 + [(128, 256)] + \
    [(256, 256)] * 3 + [(256, 512)] + [(512, 512)] * 3


def kaiming_std(c_in: int) -> float:
    return math.sqrt(2.0 / (DIM * c_in))


def normal_layer(c_in: int, c_out: int, seed: int) -> np.ndarray:
    """[C_out*C_in, 9] float32 kernels, N(0, sqrt(2/(9 C_in)))."""
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((c_out * c_in, DIM), dtype=np.float64) * kaiming_std(c_in)
    return np.ascontiguousarray(w.astype(np.float32))


def laplace_layer(c_in: int, c_out: int, seed: int) -> np.ndarray:
    """[C_out*C_in, 9] float32 kernels, Laplace(0, sqrt(2/(9 C_in))/sqrt(2))."""
    rng = np.random.default_rng(seed)
    w = rng.laplace(0.0, kaiming_std(c_in) / math.sqrt(2.0), (c_out * c_in, DIM))
    return np.ascontiguousarray(w.astype(np.float32))


def mixture_layer(n: int, n_centers: int, within_std: float, seed: int) -> np.ndarray:
    """[n, 9] float32 kernels from a seeded Gaussian mixture with N(0,1) centres."""
    rng = np.random.default_rng(seed)
    centers = rng.standard_normal((n_centers, DIM))
    labels = rng.integers(0, n_centers, n)
    x = centers[labels] + within_std * rng.standard_normal((n, DIM))
    return np.ascontiguousarray(x.astype(np.float32))


def distinct_init(X: np.ndarray, k: int, seed: int) -> np.ndarray:
    """Indices of k distinct kernels of X, taken in a seeded random order.

    Kernels are compared bit for bit after mapping -0.0 to +0.0.  Raises
    ValueError when X has fewer than k distinct kernels.
    """
    n = X.shape[0]
    rng = np.random.default_rng(seed)
    order = rng.permutation(n)
    canon = np.where(X == 0, np.float32(0), X).view(np.uint32)
    seen = set()
    sel = []
    for i in order:
        key = canon[i].tobytes()
        if key in seen:
            continue
        seen.add(key)
        sel.append(int(i))
        if len(sel) == k:
            return np.asarray(sel, dtype=np.int64)
    raise ValueError(f"only {len(sel)} distinct kernels, k={k}")


def n_distinct(X: np.ndarray) -> int:
    canon = np.where(X == 0, np.float32(0), X).view(np.uint32)
    return int(np.unique(canon, axis=0).shape[0])


@dataclass
class Layer:
    name: str
    X: np.ndarray      # [n, 9] float32
    k: int
    C0: np.ndarray     # [k, 9] float32 initial codebook

    @property
    def n(self) -> int:
        return int(self.X.shape[0])


def make_layer(name: str, X: np.ndarray, k: int, init_seed: int) -> Layer:
    k_eff = min(k, n_distinct(X)) if k >= X.shape[0] else k
    sel = distinct_init(X, k_eff, init_seed)
    return Layer(name, X, k_eff, np.ascontiguousarray(X[sel]))


# ---- the workloads ---------------------------------------------------------------

def single_layer(k: int = 256, seed: int = 1) -> list[Layer]:
    """One 64x64 3x3 layer (4096 kernels), N(0, sqrt(2/(9*64)))."""
    X = normal_layer(64, 64, seed)
    return [make_layer("conv64x64", X, k, seed)]


def vgg16_stack(k: int = 256, layers: int | None = None) -> list[Layer]:
    """The 13 VGG-16 3x3 layers; k is clamped to the layer's distinct kernels."""
    out = []
    for li, (ci, co) in enumerate(VGG16_LAYERS[:layers]):
        X = normal_layer(ci, co, 1000 + li)
        out.append(make_layer(f"vgg.conv{li + 1}", X, k, 1000 + li))
    return out


def resnet18_stack(k: int = 256, layers: int | None = None) -> list[Layer]:
    """The 16 ResNet-18 3x3 layers, Laplace-distributed; same data for every k."""
    out = []
    for li, (ci, co) in enumerate(RESNET18_LAYERS[:layers]):
        X = laplace_layer(ci, co, 2000 + li)
        out.append(make_layer(f"resnet18.conv{li + 1}", X, k, 2000 + li))
    return out


def stress_layer(n: int = 1 << 20, k: int = 4096, n_centers: int = 4096, seed: int = 4000) -> list[Layer]:
    X = mixture_layer(n, n_centers, 0.1, seed)
    return [make_layer("stress", X, k, seed)]


def shrink(layers: list[Layer], max_n: int, seed: int = 7) -> list[Layer]:
    """A bounded sample of each layer (seeded row subset), for oracle-sized runs."""
    rng = np.random.default_rng(seed)
    out = []
    for L in layers:
        if L.n <= max_n:
            out.append(L)
            continue
        rows = np.sort(rng.choice(L.n, max_n, replace=False))
        X = np.ascontiguousarray(L.X[rows])
        out.append(make_layer(L.name + f"[{max_n}]", X, min(L.k, max_n // 2), seed))
    return out


def random_codebook_state(X: np.ndarray, k: int, seed: int, jitter: float = 0.25) -> np.ndarray:
    """A codebook that is not made of data points: k data kernels plus seeded noise."""
    rng = np.random.default_rng(seed)
    sel = rng.choice(X.shape[0], k, replace=X.shape[0] < k)
    scale = float(np.std(X)) if X.size else 1.0
    C = X[sel].astype(np.float64) + jitter * scale * rng.standard_normal((k, DIM))
    return np.ascontiguousarray(C.astype(np.float32))


def random_indices(n: int, k: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, k, n).astype(np.int32)


def moved_codebook(C: np.ndarray, frac: float, scale: float, seed: int) -> np.ndarray:
    """C with a seeded random fraction of its entries moved by N(0, scale^2) noise
    (a codebook sequence with controlled movement between rounds)."""
    rng = np.random.default_rng(seed)
    k = C.shape[0]
    out = C.astype(np.float64).copy()
    moved = rng.random(k) < frac
    out[moved] += scale * rng.standard_normal((int(moved.sum()), C.shape[1]))
    return np.ascontiguousarray(out.astype(np.float32))
