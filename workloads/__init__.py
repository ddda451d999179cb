"""Seeded synthetic inputs shared by the GPU path's callers and the oracle's.

This module holds none of the method's arithmetic: it only draws images,
labels and initial weights, and names the workloads.  The paper trains on
MNIST, CIFAR-10 and ILSVRC-2012 (Table 1); those datasets are not used.  The
draws below stand in for them with the same image shapes and label
cardinalities: images ~ N(0, 1) in float32, labels uniform over the classes
in int32, both from numpy's PCG64 generator.

Initial weights are He-normal, N(0, 2 / fan_in), for conv and FC weights,
zero for biases, 1 for batch-norm gamma and 0 for beta.  The caller passes
the parameter layout (a list of ``(offset, kind, shape)``) obtained from
whichever implementation it drives, so the layout itself lives here nowhere.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    arch: str              # "lenet5" | "resnet32" | "resnet50"
    in_c: int
    in_h: int
    in_w: int
    num_classes: int
    k: int                 # learners
    b: int                 # images per learner
    lr: float = 0.01
    momentum: float = 0.9
    iters: int = 1
    seed: int = 0
    sweep_k: tuple = field(default_factory=tuple)

    @property
    def alpha(self) -> float:
        return 1.0 / self.k

    @property
    def n_images(self) -> int:
        return self.k * self.b

    def with_k(self, k: int) -> "Workload":
        d = dict(self.__dict__)
        d["k"] = k
        return Workload(**d)


# The five workloads of the method's evaluation, at their full sizes.
LENET_K2 = Workload("lenet5_k2_b4", "lenet5", 1, 28, 28, 10, k=2, b=4, iters=10, seed=0)
LENET_K8 = Workload("lenet5_k8_b16", "lenet5", 1, 28, 28, 10, k=8, b=16, iters=1000, seed=1)
RESNET32_K4 = Workload("resnet32_k4_b32", "resnet32", 3, 32, 32, 10, k=4, b=32, iters=200, seed=2)
RESNET32_SWEEP = Workload("resnet32_b16_ksweep", "resnet32", 3, 32, 32, 10, k=4, b=16, iters=200,
                          seed=3, sweep_k=(1, 2, 4, 8, 16, 32))
RESNET50_K2 = Workload("resnet50_k2_b32", "resnet50", 3, 224, 224, 1000, k=2, b=32, iters=20,
                       seed=4)
# SMA-only microbenchmark: ResNet-50's parameter count, 32 replicas.
SMA_MICRO_P = 25_557_032
SMA_MICRO_K = 32

ALL = {w.name: w for w in (LENET_K2, LENET_K8, RESNET32_K4, RESNET32_SWEEP, RESNET50_K2)}


def batch(n_images: int, in_c: int, in_h: int, in_w: int, num_classes: int, seed: int,
          step: int = 0):
    """Images [n][c][h][w] float32 ~ N(0,1) and labels [n] int32 ~ U{0..classes-1}.

    Each (seed, step) pair gives an independent draw, so successive steps
    see distinct images."""
    rng = np.random.default_rng([seed, step])
    x = rng.standard_normal((n_images, in_c, in_h, in_w), dtype=np.float32)
    y = rng.integers(0, num_classes, size=n_images, dtype=np.int32)
    return x, y


def workload_batch(w: Workload, step: int = 0):
    return batch(w.n_images, w.in_c, w.in_h, w.in_w, w.num_classes, w.seed, step)


def init_w0(layout, seed: int) -> np.ndarray:
    """Initial model, float32, from a parameter layout [(offset, kind, shape)].

    kind is one of "conv_w", "fc_w", "bias", "bn_gamma", "bn_beta"."""
    rng = np.random.default_rng(seed + 1)
    total = max(off + int(np.prod(shape)) for off, _, shape in layout)
    w = np.zeros(total, dtype=np.float32)
    for off, kind, shape in layout:
        n = int(np.prod(shape))
        if kind in ("conv_w", "fc_w"):
            fan_in = int(np.prod(shape[1:]))
            w[off:off + n] = (rng.standard_normal(n) * np.sqrt(2.0 / fan_in)).astype(np.float32)
        elif kind == "bn_gamma":
            w[off:off + n] = 1.0
        else:
            w[off:off + n] = 0.0
    return w


def random_state(k: int, P: int, seed: int, scale: float = 0.05):
    """Replicas W [k][P], gradients G [k][P], z and z_prev [P] ~ N(0,1)*scale,
    float32: the inputs of the SMA-only microbenchmark and its parity tests."""
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((k, P), dtype=np.float32) * scale)
    G = (rng.standard_normal((k, P), dtype=np.float32) * scale)
    Z = (rng.standard_normal(P, dtype=np.float32) * scale)
    Zp = (rng.standard_normal(P, dtype=np.float32) * scale)
    return W, G, Z, Zp
