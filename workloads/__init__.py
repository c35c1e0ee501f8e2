"""Seeded synthetic workloads for the AGN hot path.

This module is shared by the CPU oracle and by the GPU path's tests and
benchmark.  It holds no arithmetic of the method itself (no forward or
backward pass, no update, no commit): only the shapes of the five
workloads, the synthetic inputs that stand in for the paper's MNIST runs
(Section 4), the labels drawn from seeded random teachers, and the seeded
commit orders that simulate the asynchronous FIFO arrival of commits
(Section 1, caption of the asynchronous data-parallelism figure).

Inputs are generated on the host once and handed byte-identical to both
sides.  Everything is deterministic given the workload's seed.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import List, Sequence

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "workload", "make_data", "make_heldout", "HELDOUT_ROWS", "commit_orders",
    "random_params",
    "bf16_bits_from_f32", "f32_from_bf16_bits", "data_digest", "small_workload",
]

SEED_BASE = 20171000
TEACHER_HIDDEN = 256      # hidden width of the two-layer label teacher
_CHUNK_ROWS = 8192        # rows generated per draw (fixed so the stream is reproducible)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One AGN training configuration.

    dims      layer widths d_0..d_L (d_0 inputs, d_L = C classes)
    n         number of workers
    lam       local steps per round (lambda)
    m         mini-batch size
    eta       learning rate (constant: Section 4 applies no decay)
    rounds    number of AGN rounds the configuration runs
    order     "sequential" (0..n-1 every round) or "permutation" (seeded
              random permutation per round)
    N         number of samples; worker k owns rows [k*S, (k+1)*S), S = N // n
    data      "gauss_linear" (x ~ N(0,1), labels = argmax of a linear teacher)
              or "sparse_teacher2" (x = Bernoulli(0.2) * U[0,1), labels =
              argmax of a two-layer ReLU teacher with per-class centred logits)
    seed      base seed; data, teacher and orders use independent streams
    dtype     "fp32" or "bf16" (bf16 GEMM inputs, fp32 master weights)
    data_seed seed of the data/teacher streams (config 3 shares config 2's data)
    """
    name: str
    dims: tuple
    n: int
    lam: int
    m: int
    eta: float
    rounds: int
    order: str
    N: int
    data: str
    seed: int
    dtype: str = "fp32"
    data_seed: int | None = None

    @property
    def num_layers(self) -> int:
        return len(self.dims) - 1

    @property
    def num_params(self) -> int:
        return sum(self.dims[l] * self.dims[l + 1] + self.dims[l + 1]
                   for l in range(self.num_layers))

    @property
    def shard(self) -> int:
        return self.N // self.n

    @property
    def worker_samples_per_round(self) -> int:
        return self.n * self.lam * self.m

    @property
    def flops_per_round(self) -> int:
        """Algorithmic FLOPs of one round: forward, input-gradient (not for
        the first layer) and weight-gradient products, 2 flops per MAC."""
        d = self.dims
        macs = sum(d[l] * d[l + 1] for l in range(self.num_layers))
        per_sample = 6 * macs - 2 * d[0] * d[1]
        return per_sample * self.worker_samples_per_round


def _s(c: int) -> int:
    return SEED_BASE + c


# The five workloads.  Synthetic data stands in for MNIST (784 inputs,
# 10 classes) and for a wider 3072-input / 100-class problem.
WORKLOADS = {
    "tiny": Workload("tiny", (784, 64, 10), n=2, lam=4, m=32, eta=0.05, rounds=1,
                     order="sequential", N=4096, data="gauss_linear", seed=_s(1)),
    "mlp1000_n8": Workload("mlp1000_n8", (784, 1000, 1000, 10), n=8, lam=15, m=128,
                           eta=0.01, rounds=10, order="sequential", N=60000,
                           data="sparse_teacher2", seed=_s(2)),
    "mlp1000_n20": Workload("mlp1000_n20", (784, 1000, 1000, 10), n=20, lam=15, m=128,
                            eta=0.01, rounds=10, order="permutation", N=60000,
                            data="sparse_teacher2", seed=_s(3), data_seed=_s(2)),
    "mlp2000_n40": Workload("mlp2000_n40", (784, 2000, 2000, 2000, 10), n=40, lam=30,
                            m=128, eta=0.005, rounds=5, order="permutation", N=120000,
                            data="sparse_teacher2", seed=_s(4)),
    "wide_bf16": Workload("wide_bf16", (3072, 2048, 2048, 2048, 100), n=32, lam=10,
                          m=256, eta=0.005, rounds=5, order="permutation", N=262144,
                          data="gauss_linear", seed=_s(5), dtype="bf16"),
}
WORKLOAD_ORDER = ["tiny", "mlp1000_n8", "mlp1000_n20", "mlp2000_n40", "wide_bf16"]


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def small_workload(name, dims, n, lam, m, eta, rounds, N, data="gauss_linear",
                   order="permutation", seed=12345, dtype="fp32") -> Workload:
    """A reduced workload for tests (same generators, smaller shapes)."""
    return Workload(name, tuple(dims), n=n, lam=lam, m=m, eta=eta, rounds=rounds,
                    order=order, N=N, data=data, seed=seed, dtype=dtype)


# ---------------------------------------------------------------------------
# bf16 encoding of the input matrix (storage format of the bf16 workload)
# ---------------------------------------------------------------------------

def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16, round-to-nearest-even, return the 16-bit
    patterns as uint16.  NaN is not expected in synthetic inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------------------
# data and labels
# ---------------------------------------------------------------------------

def _teacher_logits(wl: Workload, X_chunks: Sequence[np.ndarray], rng_t) -> np.ndarray:
    """Logits of the workload's teacher on the float32 inputs (float64)."""
    d0, C = wl.dims[0], wl.dims[-1]
    if wl.data == "gauss_linear":
        T = rng_t.standard_normal((d0, C))
        return np.concatenate([xc.astype(np.float64) @ T for xc in X_chunks])
    # two-layer ReLU teacher
    A = rng_t.standard_normal((d0, TEACHER_HIDDEN)) / np.sqrt(d0)
    B = rng_t.standard_normal((TEACHER_HIDDEN, C)) / np.sqrt(TEACHER_HIDDEN)
    return np.concatenate([np.maximum(xc.astype(np.float64) @ A, 0.0) @ B for xc in X_chunks])


def _teacher_labels(wl: Workload, X_chunks: Sequence[np.ndarray], rng_t,
                    centre: np.ndarray | None = None) -> np.ndarray:
    """Labels = argmax of the teacher's logits (ties to the lowest class).
    The two-layer teacher's logits are centred per class over the training
    set so that the classes come out roughly balanced; ``centre`` passes the
    training set's per-class means for other rows."""
    z = _teacher_logits(wl, X_chunks, rng_t)
    if wl.data != "gauss_linear":
        z = z - (z.mean(axis=0) if centre is None else centre)
    return np.argmax(z, axis=1).astype(np.int32)


def _draw(wl: Workload, rng_x, N: int):
    """N input rows from the stream rng_x: (stored X, float32 chunks)."""
    d0 = wl.dims[0]
    bf16 = wl.dtype == "bf16"
    X = np.empty((N, d0), dtype=np.uint16 if bf16 else np.float32)
    chunks = []
    for r0 in range(0, N, _CHUNK_ROWS):
        rows = min(_CHUNK_ROWS, N - r0)
        if wl.data == "gauss_linear":
            xc = rng_x.standard_normal((rows, d0), dtype=np.float32)
        elif wl.data == "sparse_teacher2":
            keep = rng_x.random((rows, d0), dtype=np.float32) < np.float32(0.2)
            val = rng_x.random((rows, d0), dtype=np.float32)
            xc = np.where(keep, val, np.float32(0.0)).astype(np.float32)
        else:
            raise ValueError(f"unknown data kind {wl.data!r}")
        X[r0:r0 + rows] = bf16_bits_from_f32(xc) if bf16 else xc
        chunks.append(xc)
    return X, chunks


def make_data(wl: Workload):
    """Return (X, y).

    X is float32 [N][d_0] for fp32 workloads and uint16 bf16 bit patterns
    [N][d_0] for bf16 workloads; y is int32 [N] with labels in [0, C).
    Labels are computed from the float32 inputs (before bf16 rounding);
    argmax ties go to the lowest class index.
    """
    ds = wl.data_seed if wl.data_seed is not None else wl.seed
    X, chunks = _draw(wl, np.random.default_rng([ds, 0]), wl.N)
    y = _teacher_labels(wl, chunks, np.random.default_rng([ds, 1]))
    return X, y


HELDOUT_ROWS = 10000      # stands in for the size of MNIST's test set


def make_heldout(wl: Workload, rows: int = HELDOUT_ROWS):
    """A held-out set (X, y) in make_data's format: inputs from a stream of
    their own, labelled by the training set's teacher (for the two-layer
    teacher, centred by the training set's per-class means).  It stands in
    for the validation set of Section 4's figures."""
    ds = wl.data_seed if wl.data_seed is not None else wl.seed
    centre = None
    if wl.data != "gauss_linear":
        _, train = _draw(wl, np.random.default_rng([ds, 0]), wl.N)
        centre = _teacher_logits(wl, train, np.random.default_rng([ds, 1])).mean(axis=0)
    X, chunks = _draw(wl, np.random.default_rng([ds, 3]), rows)
    y = _teacher_labels(wl, chunks, np.random.default_rng([ds, 1]), centre)
    return X, y


def random_params(dims: Sequence[int], seed: int, scale: float = 1.0) -> np.ndarray:
    """A seeded float32 parameter vector in the packed layout (W_0 row-major
    [d_1][d_0], b_0, W_1, b_1, ...): weights N(0, scale^2 / d_in), biases
    N(0, 0.1^2).  For tests that set a model on both sides."""
    rng = np.random.default_rng([seed, 4])
    parts = []
    for l in range(len(dims) - 1):
        parts.append(rng.standard_normal(dims[l] * dims[l + 1]) * (scale / np.sqrt(dims[l])))
        parts.append(rng.standard_normal(dims[l + 1]) * 0.1)
    return np.concatenate(parts).astype(np.float32)


def commit_orders(wl: Workload, rounds: int | None = None) -> List[np.ndarray]:
    """Per-round commit orders (int32 permutations of 0..n-1)."""
    R = wl.rounds if rounds is None else rounds
    if wl.order == "sequential":
        return [np.arange(wl.n, dtype=np.int32) for _ in range(R)]
    rng = np.random.default_rng([wl.seed, 2])
    return [rng.permutation(wl.n).astype(np.int32) for _ in range(R)]


def data_digest(X: np.ndarray, y: np.ndarray) -> str:
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(X).tobytes())
    h.update(np.ascontiguousarray(y).tobytes())
    return h.hexdigest()
