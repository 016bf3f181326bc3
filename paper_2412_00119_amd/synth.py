"""Seeded synthetic workloads for the binary MLP train step.

This module only makes inputs: ±1 samples, labels and the five workload
definitions.  It holds none of the training method's arithmetic, so both the
GPU path and the CPU oracle can be fed from it without sharing any of the
method's code.

The recipe follows the paper's Random Prototypes dataset (Section 4.1.1): one
random ±1 prototype per class, and each sample is its class prototype with
every entry flipped independently with probability ``flip``.  The paper
discards duplicate samples; at the sizes used here (at least 784 bits, flip
>= 0.2) the chance of a duplicate is far below 1e-100, so that step is
skipped.  Image-shaped workloads (3072 = 3x32x32 inputs, standing in for
CIFAR-10-sized inputs) can use spatially correlated prototypes: a Gaussian
random field per channel, blurred with a circular separable Gaussian and then
thresholded at zero.

Labels are 0-based (the paper numbers classes 1..c).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Iterator, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    """One binary-MLP training workload.

    widths     K_0..K_L (input width first).
    n_classes  c.
    bound      B, the odd bound on the hidden integer weights.
    batch      mini-batch size bs.
    n_train    training samples per epoch (streamed when ``streamed``).
    n_test     held-out samples.
    flip       per-bit flip probability of the prototype recipe.
    proto      "iid" (i.i.d. ±1 prototypes) or "field" (blurred random field).
    epochs     epochs of the workload's schedule.
    group_size gamma (0 asks the library for the paper's gamma* rule).
    robustness r; p_r the initial reinforcement probability.
    index      workload number, used to derive the seeds.
    """

    name: str
    widths: Tuple[int, ...]
    n_classes: int
    bound: int
    batch: int
    n_train: int
    n_test: int
    flip: float
    proto: str = "iid"
    epochs: int = 1
    group_size: int = 64
    robustness: float = 0.25
    p_r: float = 0.5
    index: int = 1
    streamed: bool = False

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    @property
    def steps_per_epoch(self) -> int:
        return self.n_train // self.batch

    @property
    def seed_train(self) -> int:
        return 1000 * self.index + 1

    @property
    def seed_test(self) -> int:
        return 1000 * self.index + 2

    @property
    def seed_model(self) -> int:
        return 1000 * self.index + 3

    def fwd_macs(self) -> int:
        """Binary multiply-accumulates of one forward pass over one batch:
        hidden layers plus their local classifiers, at logical sizes."""
        w = self.widths
        per_sample = sum(w[l] * (w[l - 1] + self.n_classes) for l in range(1, len(w)))
        return per_sample * self.batch


# The five workloads.  Hidden-weight bounds not fixed by the workload text
# take 127, the largest odd value of an 8-bit integer.
TINY = Workload("tiny-784-256", (784, 256), 10, 15, 128, 2048, 512, 0.2,
                epochs=1, index=1)
SMALL = Workload("bmlp-784-1024x2", (784, 1024, 1024), 10, 127, 256, 60000, 10000, 0.25,
                 epochs=5, index=2)
FIELD = Workload("bmlp-3072-2048x3", (3072, 2048, 2048, 2048), 10, 127, 512, 50000, 10000, 0.3,
                 proto="field", epochs=1, index=3)
HEADLINE = Workload("bmlp-3072-4096x4", (3072, 4096, 4096, 4096, 4096), 100, 31, 1024, 50000, 10000,
                    0.3, epochs=1, index=4)
STRESS = Workload("bmlp-8192-8192x8", (8192,) + (8192,) * 8, 1000, 63, 4096, 1_000_000, 10000, 0.3,
                  epochs=1, index=5, streamed=True)

WORKLOADS = {w.name: w for w in (TINY, SMALL, FIELD, HEADLINE, STRESS)}
ORDERED = (TINY, SMALL, FIELD, HEADLINE, STRESS)


def _blur_circular(img: np.ndarray, sigma: float) -> np.ndarray:
    """Separable Gaussian blur with wrap-around boundary on the last two axes."""
    rad = int(np.ceil(4 * sigma))
    xs = np.arange(-rad, rad + 1)
    ker = np.exp(-0.5 * (xs / sigma) ** 2)
    ker /= ker.sum()
    out = np.zeros_like(img)
    for s, wgt in zip(xs, ker):
        out += wgt * np.roll(img, s, axis=-1)
    img2 = out
    out = np.zeros_like(img2)
    for s, wgt in zip(xs, ker):
        out += wgt * np.roll(img2, s, axis=-2)
    return out


def prototypes(w: Workload, rng: np.random.Generator) -> np.ndarray:
    """Class prototypes, int8 ±1 of shape [c][K_0]."""
    k0 = w.widths[0]
    if w.proto == "iid":
        return np.where(rng.random((w.n_classes, k0)) < 0.5, 1, -1).astype(np.int8)
    if w.proto == "field":
        side = int(round((k0 // 3) ** 0.5))
        assert 3 * side * side == k0, "field prototypes need K_0 = 3*s*s"
        f = rng.standard_normal((w.n_classes, 3, side, side))
        f = _blur_circular(f, 2.0)
        return np.where(f >= 0, 1, -1).astype(np.int8).reshape(w.n_classes, k0)
    raise ValueError(w.proto)


def samples(protos: np.ndarray, labels: np.ndarray, flip: float,
            rng: np.random.Generator) -> np.ndarray:
    """Noisy copies of the prototypes: each entry flipped with probability flip."""
    base = protos[labels]
    flips = rng.random(base.shape) < flip
    return np.where(flips, -base, base).astype(np.int8)


def balanced_labels(n: int, c: int, rng: np.random.Generator) -> np.ndarray:
    return rng.permutation(np.arange(n) % c).astype(np.int32)


@dataclass
class Dataset:
    """A materialised split: x int8 ±1 [N][K_0], y int32 [N]."""

    x: np.ndarray
    y: np.ndarray
    protos: np.ndarray = field(repr=False)

    def batches(self, bs: int) -> Iterator[Tuple[np.ndarray, np.ndarray]]:
        for s in range(0, len(self.y) - bs + 1, bs):
            yield self.x[s:s + bs], self.y[s:s + bs]


def make_split(w: Workload, split: str = "train", n: int | None = None) -> Dataset:
    """Materialise ``n`` samples (default: the workload's split size).

    Prototypes are drawn from the training seed, so both splits share them;
    the held-out split draws its labels and flips from its own seed.
    """
    prng = np.random.default_rng(w.seed_train)
    protos = prototypes(w, prng)
    if split == "train":
        n = w.n_train if n is None else n
        rng = np.random.default_rng([w.seed_train, 1])
    elif split == "test":
        n = w.n_test if n is None else n
        rng = np.random.default_rng(w.seed_test)
    else:
        raise ValueError(split)
    y = balanced_labels(n, w.n_classes, rng)
    x = samples(protos, y, w.flip, rng)
    return Dataset(x, y, protos)


def stream_batch(w: Workload, step: int, bs: int | None = None) -> Tuple[np.ndarray, np.ndarray]:
    """Batch ``step`` of a streamed workload, generated on demand."""
    bs = w.batch if bs is None else bs
    prng = np.random.default_rng(w.seed_train)
    protos = prototypes(w, prng)
    rng = np.random.default_rng([w.seed_train, 2, step])
    y = rng.integers(0, w.n_classes, size=bs).astype(np.int32)
    x = samples(protos, y, w.flip, rng)
    return x, y


def random_pm1(shape, rng: np.random.Generator) -> np.ndarray:
    """Uniform ±1 int8 array."""
    return np.where(rng.random(shape) < 0.5, 1, -1).astype(np.int8)


def epoch_order(w: Workload, epoch: int, n: int) -> np.ndarray:
    """Seeded per-epoch permutation of the training set."""
    return np.random.default_rng([w.seed_train, 3, epoch]).permutation(n)
