"""Parity rule between a GPU result and the oracle (test infrastructure only).

For one row sparsified at the same (g, rho, solver, iters, seed):

* the GPU's survivor indices are strictly ascending and inside [0, d);
* its index set equals the oracle's except at coordinates where the uniform u_i = x_i * 2^-32 lies
  within ``band`` (1e-6) of the oracle's p_i, where either decision is acceptable;
* |nnz_gpu - nnz_oracle| is at most the number of excused coordinates;
* values on common indices agree to relative ``val_rtol`` (1e-5);
* lambda agrees to relative ``lam_rtol`` (1e-9), or both are the same non-finite value;
* keep probabilities (when compared) agree to absolute ``p_atol`` (1e-6).

Inputs are numpy arrays; nothing here touches a GPU or imports the GPU package.
"""
from __future__ import annotations

import math

import numpy as np

from . import sample_compact, words_at


def lam_close(a: float, b: float, rtol: float = 1e-9) -> bool:
    if math.isnan(a) or math.isnan(b):
        return math.isnan(a) and math.isnan(b)
    if math.isinf(a) or math.isinf(b):
        return a == b
    if a == 0.0 or b == 0.0:
        return a == b
    return abs(a - b) <= rtol * abs(b)


def compare_sample(g, p, seed, idx, val, nnz, lam_gpu, lam_oracle, band=1e-6, val_rtol=1e-5,
                   lam_rtol=1e-9, cap=None, oracle_out=None):
    """Returns a report dict; raises AssertionError on any violation of the rule."""
    g = np.ascontiguousarray(g, np.float32)
    d = g.size
    idx = np.asarray(idx, np.int64)
    val = np.asarray(val, np.float32)
    rep = {"d": d, "nnz_gpu": int(nnz)}
    assert lam_close(float(lam_gpu), float(lam_oracle), lam_rtol), (lam_gpu, lam_oracle)
    if idx.size:
        assert idx.min() >= 0 and idx.max() < d, "index out of range"
        assert np.all(np.diff(idx) > 0), "indices not strictly ascending"
    if oracle_out is None:
        oi, ov, on = sample_compact(g, p, seed)
    else:
        oi, ov, on = oracle_out
    oi = np.asarray(oi, np.int64)
    rep["nnz_oracle"] = int(on)
    if cap is not None and on > cap:
        # the GPU wrote the first `cap` survivors only
        oi, ov = oi[:cap], np.asarray(ov)[:cap]
        limit = oi[-1] if oi.size else -1
        idx_cmp, val_cmp = idx[idx <= limit], val[idx <= limit]
    else:
        idx_cmp, val_cmp = idx, val
    diff = np.setxor1d(idx_cmp, oi, assume_unique=True)
    if diff.size:
        u = words_at(seed, diff).astype(np.float64) * 2.0 ** -32
        gap = np.abs(u - p[diff])
        bad = diff[gap > band]
        assert bad.size == 0, f"{bad.size} unexcused index differences, first {bad[:5]} gap {gap[gap > band][:5]}"
    rep["excused"] = int(diff.size)
    assert abs(int(nnz) - int(on)) <= diff.size, (int(nnz), int(on), diff.size)
    common, ig, io = np.intersect1d(idx_cmp, oi, assume_unique=True, return_indices=True)
    vg = val_cmp[ig].astype(np.float64)
    vo = np.asarray(ov, np.float64)[io]
    if common.size:
        # an amplified value sign(g_i)/lambda beyond fp32's range rounds to an infinity of that sign
        # on both sides (lambda below about 2.9e-39): equal infinities agree, any other infinity
        # does not
        inf = np.isinf(vo) | np.isinf(vg)
        assert np.array_equal(vg[inf], vo[inf]), f"infinite value mismatch at {common[inf][vg[inf] != vo[inf]][:5]}"
        fin = ~inf
        rel = np.abs(vg[fin] - vo[fin]) / np.maximum(np.abs(vo[fin]), 1e-300)
        rep["max_val_rel"] = float(rel.max(initial=0.0))
        assert rel.max(initial=0.0) <= val_rtol, f"value mismatch {rel.max()} at {common[fin][np.argmax(rel)]}"
    return rep


def compare_probs(p_gpu, p_oracle, atol=1e-6):
    p_gpu = np.asarray(p_gpu, np.float64)
    err = np.abs(p_gpu - p_oracle)
    assert err.max(initial=0.0) <= atol, f"p mismatch {err.max()} at {np.argmax(err)}"
    return float(err.max(initial=0.0))
