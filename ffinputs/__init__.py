"""Seeded synthetic inputs for the Forward-Forward workloads.

This module only draws random numbers: it holds none of the method's
arithmetic (no normalisation, no label embedding, no forward pass).  Both the
CPU oracle's tests and the HIP path's tests and benchmark take their inputs
from here, so the two sides always see the same bytes.

Recipe (all draws from ``numpy.random.default_rng``, in float64, then cast to
float32 in a fixed draw order):

* data: ``zero = rng.random((N, D)) < p_zero``; ``vals = 1 - rng.random((N, D))``
  (values in (0, 1]); ``x = where(zero, 0, vals)``.  ``p_zero`` is 0.8 for the
  MNIST-shaped sets (sparse, like handwritten digits on a black background)
  and 0 for the CIFAR-shaped set (dense pixels).  The stand-ins take the
  shapes of MNIST (784 = 28x28 features, 10 classes, 60 000 training and
  10 000 test images) and CIFAR-10 (3072 = 32x32x3 features, 50 000 images);
  no item of either dataset is used.
* labels: ``y = rng.integers(0, C, N)``; the fixed negative label (the
  paper's FixedNEG choice, drawn once) is ``(y + rng.integers(1, C, N)) % C``,
  i.e. uniform over the C-1 wrong classes.
* weights (a separate generator seeded ``seed_w``): per layer
  ``W = rng.uniform(-a, a, (d_out, d_in))`` with ``a = 1/sqrt(d_in)``, ``b = 0``.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

N_CLASSES = 10


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: data shape, net shape, hyper-parameters, schedule."""
    name: str
    n: int                      # number of base vectors
    dims: Tuple[int, ...]       # layer widths, input first
    seed_data: int
    seed_w: int
    p_zero: float               # probability that a feature is 0
    theta: float = 2.0
    lr: float = 0.03
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    norm_eps: float = 1e-8
    chunk_pairs: int = 0        # positive (= negative) rows per step; 0 = full batch
    epochs: int = 1             # passes over the data per layer
    schedule: str = "sequential"
    dtype: str = "f32"
    n_classes: int = N_CLASSES

    @property
    def n_layers(self) -> int:
        return len(self.dims) - 1

    def chunks(self) -> List[Tuple[int, int]]:
        """(first pair, pairs) of every chunk: full chunks, then one ragged tail."""
        b = self.chunk_pairs or self.n
        return [(s, min(b, self.n - s)) for s in range(0, self.n, b)]


WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    # Tiny MNIST-shaped net: 512 vectors, 784->500->500, full batch, 5 steps per layer.
    Workload("mnist_tiny_784_500x2", n=512, dims=(784, 500, 500), seed_data=0, seed_w=1,
             p_zero=0.8, lr=0.03, chunk_pairs=512, epochs=5),
    # Label scoring of 10 000 MNIST-shaped vectors through 784->2000x4.
    Workload("mnist_score_784_2000x4", n=10000, dims=(784, 2000, 2000, 2000, 2000),
             seed_data=10, seed_w=11, p_zero=0.8),
    # Full MNIST-shaped training set, 784->2000x4, 1024+1024 rows per step, layer by layer.
    Workload("mnist_784_2000x4", n=60000, dims=(784, 2000, 2000, 2000, 2000),
             seed_data=20, seed_w=21, p_zero=0.8, lr=0.03, chunk_pairs=1024),
    Workload("mnist_784_2000x4_bf16", n=60000, dims=(784, 2000, 2000, 2000, 2000),
             seed_data=20, seed_w=21, p_zero=0.8, lr=0.03, chunk_pairs=1024, dtype="bf16"),
    # Same data and net, one HIP stream per layer handing chunks down the pipeline.
    Workload("mnist_784_2000x4_pipelined", n=60000, dims=(784, 2000, 2000, 2000, 2000),
             seed_data=20, seed_w=21, p_zero=0.8, lr=0.03, chunk_pairs=1024,
             schedule="pipelined"),
    # CIFAR-shaped: 50 000 dense 3072-vectors, 3072x5 widths, bf16 operands, pipelined.
    Workload("cifar_3072x4_bf16_pipelined", n=50000, dims=(3072, 3072, 3072, 3072, 3072),
             seed_data=40, seed_w=41, p_zero=0.0, lr=0.01, chunk_pairs=2048,
             schedule="pipelined", dtype="bf16"),
]}


def make_data(seed: int, n: int, d: int, p_zero: float = 0.8,
              n_classes: int = N_CLASSES) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Base vectors x[n, d] float32, true labels y[n] int32, wrong labels y_neg[n] int32."""
    rng = np.random.default_rng(seed)
    zero = rng.random((n, d)) < p_zero if p_zero > 0 else None
    vals = 1.0 - rng.random((n, d))
    if zero is not None:
        vals[zero] = 0.0
    x = vals.astype(np.float32)
    y = rng.integers(0, n_classes, n)
    y_neg = (y + rng.integers(1, n_classes, n)) % n_classes
    return x, y.astype(np.int32), y_neg.astype(np.int32)


def make_weights(seed: int, dims) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Per layer (W[d_out, d_in] float32, b[d_out] float32), W ~ U(+-1/sqrt(d_in)), b = 0."""
    rng = np.random.default_rng(seed)
    out = []
    for d_in, d_out in zip(dims[:-1], dims[1:]):
        a = 1.0 / np.sqrt(d_in)
        w = rng.uniform(-a, a, (d_out, d_in)).astype(np.float32)
        out.append((w, np.zeros(d_out, np.float32)))
    return out


def make_workload(w: Workload, n: int | None = None):
    """Data and initial weights of a workload; ``n`` truncates the set (same prefix)."""
    x, y, y_neg = make_data(w.seed_data, w.n, w.dims[0], w.p_zero, w.n_classes)
    if n is not None:
        x, y, y_neg = x[:n], y[:n], y_neg[:n]
    return x, y, y_neg, make_weights(w.seed_w, w.dims)


def random_matrix(seed: int, rows: int, cols: int, lo: float = -1.0, hi: float = 1.0,
                  p_zero: float = 0.0) -> np.ndarray:
    """Generic seeded float32 matrix for shape sweeps and edge cases."""
    rng = np.random.default_rng(seed)
    m = rng.uniform(lo, hi, (rows, cols))
    if p_zero > 0:
        m[rng.random((rows, cols)) < p_zero] = 0.0
    return m.astype(np.float32)


def random_labels(seed: int, n: int, n_classes: int = N_CLASSES) -> Tuple[np.ndarray, np.ndarray]:
    """Seeded true and wrong labels for ``n`` rows."""
    rng = np.random.default_rng(seed)
    y = rng.integers(0, n_classes, n)
    y_neg = (y + rng.integers(1, n_classes, n)) % n_classes
    return y.astype(np.int32), y_neg.astype(np.int32)
