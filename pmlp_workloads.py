"""Seeded synthetic workloads for ParallelMLPs training.

This module only *generates inputs*: model grids (hidden sizes and
activation ids), sample matrices, labels and batch boundaries.  It holds
none of the method's arithmetic, so both the HIP path's tests/benchmark and
the CPU oracle can draw identical inputs from it without sharing any code
that computes a result.

The paper's experiments (Section 4.2, Section 4.3) use a grid of hidden
sizes times activation functions and unpublished "controlled" synthetic
datasets whose generator is not described.  The stand-in here:

* X ~ N(0, 1), fp32, shape [S, F];
* labels from a random linear teacher T ~ N(0, 1) of shape [F, O]:
  y = argmax_o (X T + eps), eps ~ N(0, 0.1^2), ties to the lowest index;
* numpy PCG64 streams: data seed 1000 + config index, the teacher drawn
  from an independent child stream of the same seed; weight-init seed
  3000 + config index (consumed by the library's counter-based init).

Model order inside the pack is activation-major, size-ascending, which is
how Section 3 (last paragraph) describes repeating the size grid once per
activation function.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

# Activation ids shared by the C ABI and the oracle's documentation.
ACT_NAMES = (
    "identity", "relu", "tanh", "sigmoid", "elu", "leaky_relu",
    "gelu", "silu", "softplus", "swish2",
    "selu", "hardshrink", "mish",
)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int
    sizes: Tuple[int, int]          # hidden sizes sizes[0]..sizes[1] inclusive
    acts: Tuple[int, ...]           # activation ids, outer loop of the grid
    repeats: int                    # copies of each (size, activation) pair
    F: int
    O: int
    S: int
    B: int
    epochs: int
    lr: float = 0.01

    def model_grid(self) -> Tuple[np.ndarray, np.ndarray]:
        hs: List[int] = []
        acts: List[int] = []
        for a in self.acts:
            for h in range(self.sizes[0], self.sizes[1] + 1):
                for _ in range(self.repeats):
                    hs.append(h)
                    acts.append(a)
        return np.asarray(hs, dtype=np.int32), np.asarray(acts, dtype=np.int32)

    @property
    def M(self) -> int:
        return len(self.acts) * (self.sizes[1] - self.sizes[0] + 1) * self.repeats

    @property
    def N(self) -> int:
        per = sum(range(self.sizes[0], self.sizes[1] + 1))
        return len(self.acts) * per * self.repeats

    @property
    def data_seed(self) -> int:
        return 1000 + self.index

    @property
    def init_seed(self) -> int:
        return 3000 + self.index

    def batches(self) -> List[Tuple[int, int]]:
        return batch_bounds(self.S, self.B)


ALL10 = tuple(range(10))

WORKLOADS = {
    # 60 models: h = 1..10 x 6 activations, F=10, O=2, 1,000 samples, B=32.
    "w60_f10": Workload("w60_f10", 0, (1, 10), (0, 1, 2, 3, 4, 5), 1, 10, 2, 1000, 32, 1),
    # 1,000 models: h = 1..100 x 10 activations, F=50, O=2, 10,000 samples, B=128.
    "w1k_f50": Workload("w1k_f50", 1, (1, 100), ALL10, 1, 50, 2, 10000, 128, 10),
    # 10,000 models: h = 1..1000 x 10 activations (N = 5,005,000), F=100, O=2, B=256.
    "w10k_f100": Workload("w10k_f100", 2, (1, 1000), ALL10, 1, 100, 2, 10000, 256, 1),
    # Same models, F=1000, B=1024, 100,000 samples (GEMM-dominated).
    "w10k_f1000": Workload("w10k_f1000", 3, (1, 1000), ALL10, 1, 1000, 2, 100000, 1024, 1),
    # Same models, F=32, O=10, B=32, 50,000 samples (reduction-dominated).
    "w10k_f32_o10": Workload("w10k_f32_o10", 4, (1, 1000), ALL10, 1, 32, 10, 50000, 32, 1),
    # Paper-shaped grid (Section 4.2): h = 1..100 x 10 activations x 10 repeats.
    "paper_10k": Workload("paper_10k", 5, (1, 100), ALL10, 10, 100, 2, 10000, 256, 1),
}


def batch_bounds(S: int, B: int) -> List[Tuple[int, int]]:
    """Contiguous batches in sample order; the last partial batch is kept."""
    return [(s, min(B, S - s)) for s in range(0, S, B)]


def make_dataset(F: int, O: int, S: int, seed: int,
                 noise: float = 0.1) -> Tuple[np.ndarray, np.ndarray]:
    """X ~ N(0,1) [S,F] fp32 and teacher labels y [S] int32 (see module doc)."""
    root = np.random.default_rng(seed)
    teacher_rng = np.random.default_rng(root.bit_generator.seed_seq.spawn(1)[0])
    X = root.standard_normal((S, F), dtype=np.float32)
    T = teacher_rng.standard_normal((F, O))
    eps = teacher_rng.standard_normal((S, O)) * noise
    scores = X.astype(np.float64) @ T + eps
    y = np.argmax(scores, axis=1).astype(np.int32)
    return np.ascontiguousarray(X), y


def make_regression_dataset(F: int, O: int, S: int, seed: int,
                            noise: float = 0.1) -> Tuple[np.ndarray, np.ndarray]:
    """X ~ N(0,1) [S,F] fp32 and real targets Y [S,O] fp32 from the same
    seeded linear teacher: Y = X T / sqrt(F) + eps, eps ~ N(0, noise^2)
    (for the regression head; the paper names regression as the method's
    other use but describes no regression data)."""
    root = np.random.default_rng(seed)
    teacher_rng = np.random.default_rng(root.bit_generator.seed_seq.spawn(1)[0])
    X = root.standard_normal((S, F), dtype=np.float32)
    T = teacher_rng.standard_normal((F, O))
    eps = teacher_rng.standard_normal((S, O)) * noise
    Y = (X.astype(np.float64) @ T / np.sqrt(F) + eps).astype(np.float32)
    return np.ascontiguousarray(X), np.ascontiguousarray(Y)


def workload_dataset(w: Workload, S: Optional[int] = None):
    return make_dataset(w.F, w.O, w.S if S is None else S, w.data_seed)


def random_models(rng: np.random.Generator, M: int, hmax: int,
                  acts: Sequence[int] = ALL10) -> Tuple[np.ndarray, np.ndarray]:
    """Random hidden sizes in [1, hmax] and random activation ids."""
    hs = rng.integers(1, hmax + 1, size=M).astype(np.int32)
    ac = rng.choice(np.asarray(acts, dtype=np.int32), size=M).astype(np.int32)
    return hs, ac


def random_params(rng: np.random.Generator, N: int, F: int, O: int,
                  scale1: float = 0.3, scale2: float = 0.5):
    """Uniform fp32 weights for tests that do not go through the library init."""
    W1 = rng.uniform(-scale1, scale1, size=(N, F)).astype(np.float32)
    W2 = rng.uniform(-scale2, scale2, size=(O, N)).astype(np.float32)
    return W1, W2
