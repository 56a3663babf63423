"""Oracle for the gradient sparsifier (Wangni et al., arXiv 1710.09854).

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg
of ``bench.py`` may import this package. It is a plain, slow, double-precision CPU statement of
what the sparsifier computes, written from the paper; it shares no code with the GPU library
(``paper_1710_09854_amd``) and imports nothing from it.

The arithmetic lives in ``oracle.cpp`` (built to ``liboracle.so`` by ``oracle/build.py``); this
module only marshals numpy arrays. Every function is pinned by a test in ``tests/test_oracle_*.py``.

Functions and the passage each follows:

* ``exact_sum``           -- exactly rounded sum of non-negative doubles (helper for every sum).
* ``philox4x32_10``/``words`` -- Philox4x32-10 (Salmon et al., SC'11), the random source that
  replaces the paper's precomputed random array (Section 5.3, engineering tricks).
* ``solve_exact``         -- Proposition 1 + eq. (5) + Algorithm 2's criterion, density budget.
* ``solve_variance``      -- Algorithm 2 verbatim (variance budget eps, eqs. 6-7).
* ``solve_greedy``        -- Algorithm 3 as printed (vector form).
* ``solve_greedy_scale``  -- Algorithm 3 rewritten through lambda (cross-check).
* ``sample_compact``      -- Section 3's protocol: Z_i ~ Bernoulli(p_i), Q(g)_i = Z_i g_i / p_i,
  survivors in ascending index order.
* ``sample_hybrid``       -- Section 3.3, eqs. (9)-(10): the survivors split into Q_A (the capped set
  S_k, stored as index and value) and Q_B (index and sign; value sign(g_i)/lambda), plus the dense
  ternary vector of the same section.
* ``coding_bits``         -- coding lengths of one hybrid message: the sparse lists, the entropy-coded
  ternary vector (Section 3.3), and the experiments' per-message formula (Section 5).
* ``aggregate``           -- Algorithm 1, step 6: the average of the workers' sparsified gradients.
* ``sparsify_segments``   -- per-layer sparsification (Section 5.2): every segment of a flat
  gradient solved and sampled on its own.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

FLAG_NONFINITE = 1
FLAG_OVERFLOW = 2
FLAG_ALLZERO = 4

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
    f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
    u32p = np.ctypeslib.ndpointer(np.uint32, flags="C_CONTIGUOUS")
    i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
    i64 = ctypes.c_int64
    pd = ctypes.POINTER(ctypes.c_double)
    pi64 = ctypes.POINTER(ctypes.c_int64)
    pu32 = ctypes.POINTER(ctypes.c_uint32)
    pint = ctypes.POINTER(ctypes.c_int)
    lib.orc_philox4x32_10.argtypes = [u32p, u32p, u32p]
    lib.orc_philox4x32_10.restype = None
    lib.orc_words.argtypes = [ctypes.c_uint64, i64, u32p]
    lib.orc_words.restype = None
    lib.orc_words_at.argtypes = [ctypes.c_uint64, i64, np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS"), u32p]
    lib.orc_words_at.restype = None
    lib.orc_exact_sum.argtypes = [f64p, i64]
    lib.orc_exact_sum.restype = ctypes.c_double
    lib.orc_exact_density.argtypes = [f32p, i64, ctypes.c_double, f64p, pd, pi64, pu32]
    lib.orc_exact_density.restype = ctypes.c_int
    lib.orc_exact_variance.argtypes = [f32p, i64, ctypes.c_double, f64p, pd, pi64, pu32]
    lib.orc_exact_variance.restype = ctypes.c_int
    for name in ("orc_greedy_alg3", "orc_greedy_scale"):
        fn = getattr(lib, name)
        fn.argtypes = [f32p, i64, ctypes.c_double, ctypes.c_int, f64p, pd, pi64, pint, pu32]
        fn.restype = ctypes.c_int
    lib.orc_sample.argtypes = [f32p, f64p, i64, ctypes.c_uint64, i32p, f32p, i64, pi64]
    lib.orc_sample.restype = ctypes.c_int
    _lib = lib
    return lib


@dataclass
class Solution:
    p: np.ndarray        # float64 [d], keep probabilities
    lam: float           # lambda of Proposition 1 (inf when every nonzero is kept surely)
    k: int               # size of the capped set {p_i = 1}
    iters: int           # greedy rescale steps taken (0 for the exact solvers)
    flags: int           # FLAG_* bits


def _f32(g) -> np.ndarray:
    g = np.ascontiguousarray(g, dtype=np.float32)
    if g.ndim != 1:
        raise ValueError("oracle works on one row at a time")
    return g


def exact_sum(x) -> float:
    x = np.ascontiguousarray(x, dtype=np.float64)
    if np.any(x < 0) or not np.all(np.isfinite(x)):
        raise ValueError("exact_sum takes finite non-negative values")
    return float(_load().orc_exact_sum(x, x.size))


def philox4x32_10(counter, key):
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, np.uint32)
    _load().orc_philox4x32_10(c, k, out)
    return out


def words(seed: int, d: int) -> np.ndarray:
    """x_i for i < d: word (i mod 4) of Philox4x32-10(key=seed, counter=(i//4, 0, 0))."""
    x = np.zeros(d, np.uint32)
    _load().orc_words(ctypes.c_uint64(seed), d, x)
    return x


def words_at(seed: int, idx) -> np.ndarray:
    """x_i for the given coordinates i (same layout as ``words``)."""
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    x = np.zeros(idx.size, np.uint32)
    _load().orc_words_at(ctypes.c_uint64(seed), idx.size, idx, x)
    return x


def _solve(fn, g, param, iters=None) -> Solution:
    g = _f32(g)
    p = np.zeros(g.size, np.float64)
    lam = ctypes.c_double()
    k = ctypes.c_int64()
    fl = ctypes.c_uint32()
    if iters is None:
        rc = fn(g, g.size, float(param), p, ctypes.byref(lam), ctypes.byref(k), ctypes.byref(fl))
        used = 0
    else:
        u = ctypes.c_int()
        rc = fn(g, g.size, float(param), int(iters), p, ctypes.byref(lam), ctypes.byref(k),
                ctypes.byref(u), ctypes.byref(fl))
        used = u.value
    if rc != 0:
        raise RuntimeError(f"oracle solver failed ({rc})")
    return Solution(p, lam.value, k.value, used, fl.value)


def solve_exact(g, rho: float) -> Solution:
    return _solve(_load().orc_exact_density, g, rho)


def solve_variance(g, eps: float) -> Solution:
    return _solve(_load().orc_exact_variance, g, eps)


def solve_greedy(g, rho: float, iters: int = 2) -> Solution:
    return _solve(_load().orc_greedy_alg3, g, rho, iters)


def solve_greedy_scale(g, rho: float, iters: int = 2) -> Solution:
    return _solve(_load().orc_greedy_scale, g, rho, iters)


def solve(g, rho: float, solver: str = "greedy", iters: int = 2) -> Solution:
    """rho is the density for "greedy" and "exact", the variance budget eps for "variance"."""
    if solver == "greedy":
        return solve_greedy(g, rho, iters)
    if solver == "exact":
        return solve_exact(g, rho)
    if solver == "variance":
        return solve_variance(g, rho)
    raise ValueError(solver)


def sample_compact(g, p, seed: int, cap: int | None = None):
    """Returns (idx int32, val float32, nnz) with survivors in ascending index order."""
    g = _f32(g)
    p = np.ascontiguousarray(p, dtype=np.float64)
    if p.shape != g.shape:
        raise ValueError("p and g differ in shape")
    cap = g.size if cap is None else int(cap)
    idx = np.zeros(max(cap, 1), np.int32)
    val = np.zeros(max(cap, 1), np.float32)
    n = ctypes.c_int64()
    _load().orc_sample(g, p, g.size, ctypes.c_uint64(seed), idx, val, cap, ctypes.byref(n))
    m = min(n.value, cap)
    return idx[:m].copy(), val[:m].copy(), n.value


def sparsify(g, rho: float, solver: str = "greedy", iters: int = 2, seed: int = 0):
    """Solve, then sample, amplify and compact one row. Returns (Solution, idx, val, nnz)."""
    sol = solve(g, rho, solver, iters)
    if sol.flags & FLAG_NONFINITE:
        return sol, np.zeros(0, np.int32), np.zeros(0, np.float32), 0
    idx, val, n = sample_compact(g, sol.p, seed)
    return sol, idx, val, n


@dataclass
class HybridMessage:
    qa_idx: np.ndarray   # int32, ascending: the capped survivors (every i with p_i = 1 survives)
    qa_val: np.ndarray   # float32 g_i (= g_i / p_i since p_i = 1)
    qb_idx: np.ndarray   # int32, ascending: the other survivors
    qb_neg: np.ndarray   # bool, g_i < 0 for each entry of qb_idx (Q_B's value is sign(g_i) / lambda)
    q: np.ndarray        # int8 [d]: 2 on S_k, sign(g_i) on the other survivors, 0 elsewhere


def sample_hybrid(g, p, seed: int) -> HybridMessage:
    """Section 3.3, eqs. (9)-(10). The survivors are those of ``sample_compact`` (same generator, same
    test Z_i = [x_i < p_i 2^32]); a survivor belongs to Q_A when p_i = 1 (the capped set S_k), to Q_B
    otherwise. The dense vector q takes 2 on S_k and lambda Q(g_i) = sign(g_i) on Q_B's entries."""
    g = _f32(g)
    p = np.ascontiguousarray(p, dtype=np.float64)
    idx, _, n = sample_compact(g, p, seed)
    assert idx.size == n
    capped = p[idx] == 1.0
    qa_idx = idx[capped]
    qb_idx = idx[~capped]
    q = np.zeros(g.size, np.int8)
    q[qa_idx] = 2
    q[qb_idx] = np.where(g[qb_idx] < 0, -1, 1).astype(np.int8)
    return HybridMessage(qa_idx, g[qa_idx].copy(), qb_idx, g[qb_idx] < 0, q)


def coding_bits(d: int, n_a: int, n_b: int, n_b_neg: int, float_bits: int = 32):
    """Bits of one hybrid message of a d-coordinate gradient (Section 3.3; Theorem 4's accounting):
    (1) the sparse lists: each Q_A entry an index (log2 d bits) and a float, each Q_B entry an index
        and a sign bit, plus the single float 1/lambda;
    (2) the ternary vector with entropy coding, sum over its symbols l of d_l log2(d / d_l), plus a
        float per Q_A entry and the float 1/lambda;
    (3) the experiments' per-message cost, n_a (b + log2 d) + min(2d, n_b log2 d) + b, with the
        realised |Q_B| standing in for the expected sum of p over the uncapped set."""
    b = float(float_bits)
    L = np.log2(float(d))
    sparse = n_a * (b + L) + n_b * (L + 1.0) + b
    counts = [n_a, n_b_neg, n_b - n_b_neg, d - n_a - n_b]
    ent = sum(c * np.log2(d / c) for c in counts if c > 0)
    ternary = ent + n_a * b + b
    paper = n_a * (b + L) + min(2.0 * d, n_b * L) + b
    return float(sparse), float(ternary), float(paper)


def aggregate(lists, d: int) -> np.ndarray:
    """Algorithm 1, step 6: v = (1/M) sum_m Q(g^m) for the M workers' sparse messages, given as
    (idx, val) pairs of arrays with distinct indices. Each coordinate's sum is taken in fp64 in
    worker order, divided by M and rounded to fp32."""
    acc = np.zeros(int(d), np.float64)
    for idx, val in lists:
        idx = np.asarray(idx, np.int64)
        assert np.unique(idx).size == idx.size, "indices must be distinct within a message"
        acc[idx] += np.asarray(val, np.float32).astype(np.float64)
    return (acc / len(lists)).astype(np.float32)


def sparsify_segments(g, offsets, rhos, seeds, solver: str = "greedy", iters: int = 2):
    """Section 5.2 sparsifies each layer independently: segment s = g[off[s]:off[s+1]] gets its own
    budget rho[s] * length, its own solution and its own random words (key seeds[s], counters
    counted within the segment). Returns one (Solution, idx, val, nnz) per segment, idx within the
    segment."""
    g = _f32(g)
    out = []
    for s_, (b, e) in enumerate(zip(offsets[:-1], offsets[1:])):
        seg = g[int(b):int(e)]
        if seg.size == 0:
            out.append((None, np.zeros(0, np.int32), np.zeros(0, np.float32), 0))
            continue
        out.append(sparsify(seg, float(rhos[s_]), solver, iters, int(seeds[s_])))
    return out
