"""Seeded synthetic inputs and workload presets for the parallel neural network (PNN).

This module is shared input, not shared method: it draws the data, labels and the
initial parameter vector that both the CPU oracle and the GPU library are fed, and
it holds none of the method's arithmetic (no forward pass, no gradient, no merge).

The paper trains on MNIST (28x28 grey images, 10 classes, 60,000 train / 10,000 test;
section "MNIST Dataset").  MNIST is not available here, so every workload uses a
stand-in with the same shapes: each sample is one of a few seeded random prototype
images plus Gaussian pixel noise (standard deviation 0.15), clipped to [0, 1]; its
label is the class of the prototype.

Seeds: base 230409590 + workload index; independent streams come from
``PCG64(seed).jumped(stream)``: 0 = prototypes, 1 = training set, 2 = held-out set,
3 = initial parameters.

The paper initialises weights from a time-seeded N(0,1) draw (section "Implementation
Details"); that is not reproducible, so the initial parameters here are uniform Xavier
per layer, W ~ U(-a, a) with a = sqrt(6 / (fan_in + fan_out)), and zero biases.  One
parameter vector is cloned to every child network, as the paper does when it compares
an SNN and a PNN started from the same random net (section "Accuracy and Confidence").
"""
from __future__ import annotations

import dataclasses
from typing import List, Tuple

import numpy as np

BASE_SEED = 230409590
N_PIXELS = 784
N_CLASSES = 10
NOISE_STD = 0.15

# activation codes (shared numbering of the C interfaces)
SIGMOID, TANH, RELU, LEAKY_RELU, SOFTMAX = 0, 1, 2, 3, 4
# loss codes: which output-error rule is used
LOSS_MSE, LOSS_XENT = 0, 1
# precision codes
FP32, BF16_MIXED = 0, 1

ACT_NAMES = {SIGMOID: "sigmoid", TANH: "tanh", RELU: "relu", LEAKY_RELU: "leaky_relu", SOFTMAX: "softmax"}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One training workload: net shape, schedule and synthetic data recipe."""
    name: str
    index: int                 # seed offset
    sizes: Tuple[int, ...]     # layer widths, sizes[0] = 784 inputs, sizes[-1] = 10 outputs
    acts: Tuple[int, ...]      # activation per weight layer
    loss: int
    precision: int
    replicas: int              # K child networks
    batch: int                 # B, 1 = per-sample SGD
    lr: float
    epochs: int
    merge_every_epoch: bool    # True: average + broadcast after every epoch; False: average once at the end
    n_train: int
    n_test: int
    protos_per_class: int

    @property
    def n_layers(self) -> int:
        return len(self.sizes) - 1

    def param_count(self) -> int:
        return sum(self.sizes[l + 1] * self.sizes[l] + self.sizes[l + 1] for l in range(self.n_layers))

    def scaled(self, **kw) -> "Workload":
        """Same recipe with some fields replaced (smaller parity cases)."""
        return dataclasses.replace(self, **kw)


WORKLOADS: List[Workload] = [
    Workload("mlp784-16-10_sigmoid_fp32_k1_sgd", 0, (784, 16, 10), (SIGMOID, SIGMOID), LOSS_MSE, FP32,
             1, 1, 0.1, 1, False, 2_000, 10_000, 1),
    Workload("mlp784-128-10_sigmoid_fp32_k4_sgd", 1, (784, 128, 10), (SIGMOID, SIGMOID), LOSS_MSE, FP32,
             4, 1, 0.05, 1, False, 60_000, 10_000, 1),
    Workload("mlp784-256-10_tanh_sigmoid_fp32_k16_b32", 2, (784, 256, 10), (TANH, SIGMOID), LOSS_MSE, FP32,
             16, 32, 0.05, 5, False, 60_000, 10_000, 20),
    Workload("mlp784-512-256-10_relu_softmax_bf16_k64_b64", 3, (784, 512, 256, 10), (RELU, RELU, SOFTMAX),
             LOSS_XENT, BF16_MIXED, 64, 64, 0.05, 3, True, 240_000, 10_000, 1),
    Workload("mlp784-1024-10_sigmoid_fp32_k256_b128", 4, (784, 1024, 10), (SIGMOID, SIGMOID), LOSS_MSE, FP32,
             256, 128, 0.02, 2, True, 600_000, 10_000, 1),
]


def _rng(index: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(BASE_SEED + index).jumped(stream))


def prototypes(w: Workload) -> np.ndarray:
    """[10 * protos_per_class, 784] float32 prototype images, pixels i.i.d. U(0, 1)."""
    return _rng(w.index, 0).random((N_CLASSES * w.protos_per_class, N_PIXELS), dtype=np.float32)


def _samples(w: Workload, n: int, stream: int) -> Tuple[np.ndarray, np.ndarray]:
    protos = prototypes(w)
    rng = _rng(w.index, stream)
    labels = rng.integers(0, N_CLASSES, size=n, dtype=np.int64)
    if w.protos_per_class > 1:
        which = labels * w.protos_per_class + rng.integers(0, w.protos_per_class, size=n, dtype=np.int64)
    else:
        which = labels
    x = np.empty((n, N_PIXELS), dtype=np.float32)
    step = 65536
    for s in range(0, n, step):
        e = min(n, s + step)
        noise = rng.standard_normal((e - s, N_PIXELS), dtype=np.float32)
        noise *= np.float32(NOISE_STD)
        noise += protos[which[s:e]]
        np.clip(noise, 0.0, 1.0, out=noise)
        x[s:e] = noise
    return x, labels.astype(np.int32)


def train_set(w: Workload, n: int | None = None) -> Tuple[np.ndarray, np.ndarray]:
    """Training images [n, 784] float32 in [0, 1] and labels [n] int32 (default n = w.n_train)."""
    return _samples(w, w.n_train if n is None else n, 1)


def test_set(w: Workload, n: int | None = None) -> Tuple[np.ndarray, np.ndarray]:
    """Held-out images and labels drawn from the same recipe on an independent stream."""
    return _samples(w, w.n_test if n is None else n, 2)


def init_params(w: Workload, seed_stream: int = 3) -> np.ndarray:
    """Flat float32 parameter vector theta0 = [W1, b1, W2, b2, ...], W_l row-major [out][in]."""
    rng = _rng(w.index, seed_stream)
    parts = []
    for l in range(w.n_layers):
        fan_in, fan_out = w.sizes[l], w.sizes[l + 1]
        a = np.sqrt(6.0 / (fan_in + fan_out))
        parts.append(rng.uniform(-a, a, size=fan_out * fan_in).astype(np.float32))
        parts.append(np.zeros(fan_out, dtype=np.float32))
    return np.concatenate(parts)


def random_params(sizes, seed: int, scale: float = 0.5) -> np.ndarray:
    """Small seeded parameter vector with non-zero biases, for tiny test nets."""
    rng = np.random.Generator(np.random.PCG64(seed))
    parts = []
    for l in range(len(sizes) - 1):
        parts.append(rng.uniform(-scale, scale, size=sizes[l + 1] * sizes[l]).astype(np.float32))
        parts.append(rng.uniform(-scale, scale, size=sizes[l + 1]).astype(np.float32))
    return np.concatenate(parts)


def random_batch(n_in: int, n_out: int, n: int, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """Seeded inputs in [0, 1] and labels in [0, n_out), for tiny test nets."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.random((n, n_in), dtype=np.float32)
    y = rng.integers(0, n_out, size=n).astype(np.int32)
    return x, y
