"""Seeded synthetic inputs for the gradient sparsifier.

This module only draws numbers: it holds none of the sparsifier's arithmetic, and both the GPU
path and the oracle consume the same bytes from it. Every generator is a pure function of its
arguments (numpy ``default_rng`` with a fixed seed), returning C-contiguous float32 arrays.

The five workloads stand in for the gradients the paper sparsifies (its convex experiments use
synthetic logistic-regression data, Section 5.1; its deep-learning experiment sparsifies CNN
layer gradients, Section 5.2), at the sizes of a one-GPU share:

* ``c1`` -- one N(0,1) row, d = 65,536 (data and Philox seed 0), rho = 0.1.
* ``c2`` -- 16 rows (one per simulated worker) of d = 2^20, Laplace(0,1) times a per-row scale
  10^U(-3,0); Philox seeds 1000 + r; rho in {0.01, 0.1}.
* ``c3`` -- the minibatch gradient of the l2-regularised logistic loss of eq. (14) on a sparse
  256 x 2^22 design (0.1 % density): many exact zeros and a heavy tail.
* ``c4`` -- a ResNet-50-shaped gradient, d = 25,557,032, from 54 contiguous segments each
  N(0, sigma_k^2) with sigma_k = 10^U(-5,-1).
* ``c5`` -- d = 2^28 Student-t(2) with 1 % of coordinates multiplied by 100.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# ResNet-50 weight tensors (53 convolutions with their folded batch-norm scale and shift, and
# the 2048 x 1000 classifier with its bias), in network order.
RESNET50_SEGMENTS = [
    9536, 4224, 36992, 16896, 16896, 16512, 36992, 16896, 16512, 36992, 16896, 33024, 147712,
    66560, 132096, 65792, 147712, 66560, 65792, 147712, 66560, 65792, 147712, 66560, 131584,
    590336, 264192, 526336, 262656, 590336, 264192, 262656, 590336, 264192, 262656, 590336,
    264192, 262656, 590336, 264192, 262656, 590336, 264192, 525312, 2360320, 1052672, 2101248,
    1049600, 2360320, 1052672, 1049600, 2360320, 1052672, 2049000,
]
assert len(RESNET50_SEGMENTS) == 54 and sum(RESNET50_SEGMENTS) == 25_557_032


@dataclass
class Workload:
    name: str
    g: np.ndarray                 # float32 [rows, d]
    rhos: list                    # densities the workload is run at
    solvers: list                 # "greedy" and/or "exact"
    seeds: list                   # Philox seed per row
    iters: int = 2                # greedy rescale steps (the paper's experiments use two)
    meta: dict = field(default_factory=dict)

    @property
    def rows(self) -> int:
        return self.g.shape[0]

    @property
    def d(self) -> int:
        return self.g.shape[1]


def c1() -> Workload:
    rng = np.random.default_rng(0)
    g = rng.standard_normal(65536).astype(np.float32).reshape(1, -1)
    return Workload("c1_normal_d65536", np.ascontiguousarray(g), CONFIG_RHOS["c1"], CONFIG_SOLVERS["c1"], [0])


def c2(rows: int = 16, d: int = 1 << 20) -> Workload:
    rng = np.random.default_rng(2)
    scale = 10.0 ** rng.uniform(-3.0, 0.0, rows)
    g = np.empty((rows, d), np.float32)
    for r in range(rows):
        g[r] = (rng.laplace(0.0, 1.0, d) * scale[r]).astype(np.float32)
    return Workload(f"c2_laplace_{rows}x{d}", g, CONFIG_RHOS["c2"], CONFIG_SOLVERS["c2"],
                    [1000 + r for r in range(rows)], meta={"row_scale": scale})


def c3(n: int = 256, d: int = 1 << 22, density: float = 1e-3, lam_reg: float = 1e-4,
       dense_reg: bool = False) -> Workload:
    """Gradient of f(w) = (1/n) sum_n log2(1 + exp(-y_n x_n.w)) + lam_reg ||w||^2 (eq. 14) at a
    random w, on a sparse random design. The regulariser's gradient 2*lam_reg*w is applied only
    on the columns the minibatch touches (lazy regularisation), unless ``dense_reg``."""
    rng = np.random.default_rng(3)
    w = rng.normal(0.0, 0.01, d)
    y = rng.choice(np.array([-1.0, 1.0]), size=n)
    grad = np.zeros(d, np.float64)
    support = np.zeros(d, bool)
    for r in range(n):
        m = rng.binomial(d, density)
        cols = rng.choice(d, size=m, replace=False)
        vals = rng.standard_normal(m)
        margin = y[r] * float(vals @ w[cols])
        # d/dz log2(1 + e^{-z}) = -1 / ((1 + e^{z}) ln 2), z = y x.w
        coef = -y[r] / ((1.0 + np.exp(margin)) * np.log(2.0))
        np.add.at(grad, cols, coef * vals)
        support[cols] = True
    grad /= n
    if dense_reg:
        grad += 2.0 * lam_reg * w
    else:
        grad[support] += 2.0 * lam_reg * w[support]
    g = grad.astype(np.float32).reshape(1, -1)
    return Workload("c3_logreg_256x4194304", np.ascontiguousarray(g), CONFIG_RHOS["c3"], CONFIG_SOLVERS["c3"],
                    [3], meta={"support_fraction": float(support.mean())})


def c4() -> Workload:
    rng = np.random.default_rng(4)
    d = sum(RESNET50_SEGMENTS)
    g = np.empty(d, np.float32)
    sig = 10.0 ** rng.uniform(-5.0, -1.0, len(RESNET50_SEGMENTS))
    off = 0
    for s, sz in zip(sig, RESNET50_SEGMENTS):
        g[off:off + sz] = (rng.standard_normal(sz) * s).astype(np.float32)
        off += sz
    return Workload("c4_resnet50_d25557032", g.reshape(1, -1), CONFIG_RHOS["c4"], CONFIG_SOLVERS["c4"], [4],
                    meta={"segments": list(RESNET50_SEGMENTS), "sigma": sig})


def c5(d: int = 1 << 28, chunk: int = 1 << 24) -> Workload:
    rng = np.random.default_rng(5)
    g = np.empty(d, np.float32)
    for off in range(0, d, chunk):
        m = min(chunk, d - off)
        t = rng.standard_t(2.0, m)
        out = rng.random(m) < 0.01
        t[out] *= 100.0
        g[off:off + m] = t.astype(np.float32)
    return Workload(f"c5_student_t2_outliers_d{d}", g.reshape(1, -1), CONFIG_RHOS["c5"], CONFIG_SOLVERS["c5"], [5])


CONFIGS = {"c1": c1, "c2": c2, "c3": c3, "c4": c4, "c5": c5}
# the solvers and densities each workload is run at (what the generators above attach)
CONFIG_SOLVERS = {"c1": ["greedy", "exact"], "c2": ["greedy"], "c3": ["greedy", "exact"], "c4": ["exact", "greedy"],
                  "c5": ["exact", "greedy"]}
CONFIG_RHOS = {"c1": [0.1], "c2": [0.01, 0.1], "c3": [0.01], "c4": [0.001, 0.01], "c5": [0.001, 0.01, 0.1]}


# ------------------------------------------------------------------------------------------
# Small generators for unit and parity tests (heavy capping, ties, edge cases).
# ------------------------------------------------------------------------------------------

def normal(d: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).standard_normal(d).astype(np.float32)


def two_level(d: int, s: int, hi: float, lo: float, seed: int) -> np.ndarray:
    """s coordinates of magnitude hi and d - s of magnitude lo, random signs and positions."""
    rng = np.random.default_rng(seed)
    a = np.full(d, lo, np.float64)
    a[rng.choice(d, size=s, replace=False)] = hi
    return (a * rng.choice([-1.0, 1.0], size=d)).astype(np.float32)


def approx_sparse(d: int, s: int, rho_def: float, seed: int) -> np.ndarray:
    """A (rho_def, s)-approximately sparse vector in the sense of Definition 2: the off-support
    l1 mass is rho_def times the support's."""
    rng = np.random.default_rng(seed)
    g = np.zeros(d, np.float64)
    sup = rng.choice(d, size=s, replace=False)
    g[sup] = rng.standard_normal(s) * 10.0
    rest = np.setdiff1d(np.arange(d), sup)
    tail = np.abs(rng.standard_normal(rest.size)) + 1e-3
    tail *= rho_def * np.abs(g[sup]).sum() / tail.sum()
    g[rest] = tail * rng.choice([-1.0, 1.0], size=rest.size)
    return g.astype(np.float32)


def t_mixture(d: int, seed: int, nu: float = 2.0, frac: float = 0.01, mult: float = 100.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    t = rng.standard_t(nu, d)
    t[rng.random(d) < frac] *= mult
    return t.astype(np.float32)


def integer_ties(d: int, seed: int, levels: int = 6) -> np.ndarray:
    """Integer magnitudes 0..levels-1 (many exact ties, some zeros), random signs."""
    rng = np.random.default_rng(seed)
    return (rng.integers(0, levels, d) * rng.choice([-1.0, 1.0], size=d)).astype(np.float32)


def strided_large(d: int, seed: int) -> np.ndarray:
    """1e-3 N(0, 1) with 76 large magnitudes (about 100, random signs) in two strided patterns of
    the first 16,384 coordinates: 4-coordinate runs at 256 j for j < 16, and at 4096 + 256 j + 20
    for j < 3. (Runs 256 apart fall to one lane of the sampling pass's decide phase, so at most
    densities that lane keeps more capped survivors than its LDS row holds.) d >= 16384."""
    rng = np.random.default_rng(seed)
    g = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    pos = [256 * j + c for j in range(16) for c in range(4)] + [4096 + 256 * j + 20 + c for j in range(3) for c in range(4)]
    g[pos] = ((100.0 + rng.uniform(0.0, 8.0, len(pos))) * rng.choice([-1.0, 1.0], size=len(pos))).astype(np.float32)
    return g


def lowest_binade(d: int, seed: int) -> np.ndarray:
    """Four fifths of the magnitudes uniform in [0.5, 4), one fifth uniform in [1.0e-3, 1.9e-3)
    (one binade, the row's lowest), random signs and order. At densities near 1 the capped set
    reaches into the small magnitudes, so 1/lambda lies inside the row's lowest binade."""
    rng = np.random.default_rng(seed)
    nt = d // 5
    g = np.empty(d, np.float32)
    g[: d - nt] = rng.uniform(0.5, 4.0, d - nt)
    g[d - nt:] = rng.uniform(1.0e-3, 1.9e-3, nt)
    g *= rng.choice([-1.0, 1.0], size=d).astype(np.float32)
    return g[rng.permutation(d)].astype(np.float32)


def wide_range(d: int, seed: int) -> np.ndarray:
    """Magnitudes spread over many binades, including subnormals."""
    rng = np.random.default_rng(seed)
    e = rng.uniform(-140, 30, d)
    return (rng.choice([-1.0, 1.0], size=d) * np.exp2(e)).astype(np.float32)


def full_range(d: int, seed: int) -> np.ndarray:
    """Magnitudes log-uniform over all of fp32's binades, subnormals to just below the largest
    finite value, with random signs."""
    rng = np.random.default_rng(seed)
    e = rng.uniform(-149.0, 127.99, d)
    return np.minimum(np.exp2(e), 3.4e38).astype(np.float32) * rng.choice([-1.0, 1.0], size=d).astype(np.float32)


def sparse_lists(workers: int, d: int, cap: int, seed: int, empty=(), over=()):
    """Per-worker strictly ascending index lists with fp32 values, as [workers, cap] arrays and an
    int64 length per worker: mixed lengths, every third list clustered into a short index range,
    values spread over sixty binades. Workers in `empty` get length 0 (odd ones -1), those in
    `over` a full list and a length beyond cap (an overflowed list of which cap entries are kept)."""
    rng = np.random.default_rng(seed)
    idx = np.zeros((workers, cap), np.int32)
    val = np.zeros((workers, cap), np.float32)
    nnz = np.zeros(workers, np.int64)
    for m in range(workers):
        n = int(rng.integers(0, cap + 1))
        if m % 3 == 0:
            lo = int(rng.integers(0, d))
            pool = np.arange(lo, min(d, lo + 3 * n + 1))
        else:
            pool = np.arange(d)
        n = min(n, pool.size)
        idx[m, :n] = np.sort(rng.choice(pool, size=n, replace=False))
        val[m, :n] = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
        nnz[m] = n
    for m in empty:
        nnz[m] = -1 if m % 2 else 0
    for m in over:
        nnz[m] = cap + 17
        idx[m] = np.sort(rng.choice(d, size=cap, replace=False))
        val[m] = rng.standard_normal(cap).astype(np.float32)
    return idx, val, nnz
