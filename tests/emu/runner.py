"""Runs the emulated library on host buffers and checks it against the oracle (test
infrastructure). Usable in-process or as a script (so it can run under AddressSanitizer)."""
import ctypes
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as W  # noqa: E402
from oracle.compare import compare_probs, compare_sample  # noqa: E402


def load(path):
    L = ctypes.CDLL(path)
    vp, i64, u64, f64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_int
    L.gspar_workspace_bytes.argtypes = [i64, i64, i32]
    L.gspar_workspace_bytes.restype = ctypes.c_size_t
    L.sparsify_sample_compact.argtypes = [vp, i64, f64, i32, i32, u64, vp, vp, i64, vp, vp, vp, vp, vp,
                                          ctypes.c_size_t, vp]
    L.sparsify_probs.argtypes = [vp, i64, f64, i32, i32, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_sample_compact_batched.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, vp, vp, i64, vp, vp,
                                                  vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_sample_hybrid_batched.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, vp, vp, i64, vp, vp, i64,
                                                 vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.gspar_aggregate.argtypes = [vp, vp, i64, vp, i64, i64, vp, vp]
    L.sparsify_sample_compact_segmented.argtypes = [vp, i64, vp, vp, vp, i32, i32, vp, vp, vp, i64, vp, vp, vp,
                                                    vp, vp, ctypes.c_size_t, vp]
    L.sparsify_probs_segmented.argtypes = [vp, i64, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_sample_hybrid_segmented.argtypes = [vp, i64, vp, vp, vp, i32, i32, vp, vp, vp, i64, vp, vp, i64,
                                                   vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    return L


def _aligned(nbytes):
    raw = np.zeros(nbytes + 512, np.uint8)
    off = (-raw.ctypes.data) % 256
    return raw, raw[off:off + nbytes]


def sample_row(L, g, rho, solver, seed, iters=2, cap=None):
    d = g.size
    cap = d if cap is None else cap
    idx = np.zeros(max(cap, 1), np.int32)
    val = np.zeros(max(cap, 1), np.float32)
    nnz = np.zeros(1, np.int64)
    lam = np.zeros(1)
    k = np.zeros(1, np.int64)
    fl = np.zeros(1, np.uint32)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(1, d, sid)
    keep, ws = _aligned(wsb)
    rc = L.sparsify_sample_compact(g.ctypes.data, d, rho, sid, iters, seed, idx.ctypes.data, val.ctypes.data, cap,
                                   nnz.ctypes.data, lam.ctypes.data, k.ctypes.data, fl.ctypes.data, ws.ctypes.data,
                                   wsb, None)
    assert rc == 0, rc
    n = int(nnz[0])
    m = min(n, cap)
    return idx[:m], val[:m], n, float(lam[0]), int(k[0]), int(fl[0])


def probs_row(L, g, rho, solver, iters=2):
    d = g.size
    p = np.zeros(d, np.float32)
    lam = np.zeros(1)
    k = np.zeros(1, np.int64)
    fl = np.zeros(1, np.uint32)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(1, d, sid)
    keep, ws = _aligned(wsb)
    rc = L.sparsify_probs(g.ctypes.data, d, rho, sid, iters, p.ctypes.data, lam.ctypes.data, k.ctypes.data,
                          fl.ctypes.data, ws.ctypes.data, wsb, None)
    assert rc == 0, rc
    return p, float(lam[0]), int(k[0]), int(fl[0])


CASES = [
    ("normal_65536", lambda: W.normal(65536, 0)),
    ("normal_spiked_65536", lambda: np.concatenate([W.normal(37, 9) * np.float32(40), W.normal(65536 - 37, 0)])),
    ("tmix_50001", lambda: W.t_mixture(50001, 2)),
    ("ties_20001", lambda: W.integer_ties(20001, 3)),
    ("wide_range_30000", lambda: W.wide_range(30000, 4)),
    ("two_level_20001", lambda: W.two_level(20001, 100, 50.0, 1.0, 5)),
    ("approx_sparse_20000", lambda: W.approx_sparse(20000, 100, 0.05, 6)),
    ("tiny_7", lambda: W.normal(7, 7)),
]


def run_all(path, rhos=(0.001, 0.01, 0.1, 0.5), verbose=True):
    L = load(path)
    n_checked = 0
    for name, mk in CASES:
        g = np.ascontiguousarray(mk(), np.float32)
        for solver in ("greedy", "exact"):
            for rho in rhos:
                seed = 99 + len(name)
                sol = oracle.solve(g, rho, solver, 2)
                idx, val, n, lam, k, fl = sample_row(L, g, rho, solver, seed)
                assert fl == 0, (name, solver, rho, fl)
                rep = compare_sample(g, sol.p, seed, idx, val, n, lam, sol.lam)
                if solver == "exact":
                    assert lam == sol.lam and k == sol.k, (name, rho, lam, sol.lam, k, sol.k)
                n_checked += 1
                if verbose:
                    print(f"{name} {solver} rho={rho}: nnz={n} excused={rep['excused']} lam={lam:.12g}", flush=True)
        p, lam, k, fl = probs_row(L, g, 0.1, "exact")
        compare_probs(p, oracle.solve_exact(g, 0.1).p)
    return n_checked




def batched(L, g2, rhos, seeds, solver, iters=2, cap=None, ld=None):
    rows, d = g2.shape
    ld = d if ld is None else ld
    buf = np.zeros((rows, ld), np.float32)
    buf[:, :d] = g2
    cap = d if cap is None else cap
    idx = np.zeros((rows, max(cap, 1)), np.int32)
    val = np.zeros((rows, max(cap, 1)), np.float32)
    nnz = np.zeros(rows, np.int64)
    lam = np.zeros(rows)
    k = np.zeros(rows, np.int64)
    fl = np.zeros(rows, np.uint32)
    r = np.ascontiguousarray(rhos, np.float64)
    s = np.array([int(x) & 0xFFFFFFFFFFFFFFFF for x in seeds], np.uint64)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(rows, d, sid)
    keep, ws = _aligned(wsb)
    rc = L.sparsify_sample_compact_batched(buf.ctypes.data, rows, d, ld, r.ctypes.data, sid, iters, s.ctypes.data,
                                           idx.ctypes.data, val.ctypes.data, cap, nnz.ctypes.data, lam.ctypes.data,
                                           k.ctypes.data, fl.ctypes.data, ws.ctypes.data, wsb, None)
    assert rc == 0, rc
    return idx, val, nnz, lam, k, fl


def hybrid_batched(L, g2, rhos, seeds, solver, iters=2, cap=None, ld=None):
    """The hybrid-coding entry point on host buffers: (idx_a, val_a, n_a, code_b, n_b, inv, q, lam, flags)."""
    rows, d = g2.shape
    ld = d if ld is None else ld
    buf = np.zeros((rows, ld), np.float32)
    buf[:, :d] = g2
    cap = d if cap is None else cap
    idx_a = np.zeros((rows, max(cap, 1)), np.int32)
    val_a = np.zeros((rows, max(cap, 1)), np.float32)
    code_b = np.zeros((rows, max(cap, 1)), np.int32)
    n_a = np.zeros(rows, np.int64)
    n_b = np.zeros(rows, np.int64)
    inv = np.zeros(rows, np.float32)
    q = np.full((rows, ld), 77, np.int8)
    lam = np.zeros(rows)
    fl = np.zeros(rows, np.uint32)
    r = np.ascontiguousarray(rhos, np.float64)
    s = np.array([int(x) & 0xFFFFFFFFFFFFFFFF for x in seeds], np.uint64)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(rows, d, sid)
    keep, ws = _aligned(wsb)
    rc = L.sparsify_sample_hybrid_batched(buf.ctypes.data, rows, d, ld, r.ctypes.data, sid, iters, s.ctypes.data,
                                          idx_a.ctypes.data, val_a.ctypes.data, cap, n_a.ctypes.data,
                                          code_b.ctypes.data, cap, n_b.ctypes.data, inv.ctypes.data, q.ctypes.data,
                                          lam.ctypes.data, fl.ctypes.data, ws.ctypes.data, wsb, None)
    assert rc == 0, rc
    return idx_a, val_a, n_a, code_b, n_b, inv, q[:, :d], lam, fl


def check_hybrid(L, verbose=True):
    """The hybrid coding against the compaction of the same call (identical survivors and values)
    and against the oracle's split (Section 3.3)."""
    rows, d = 3, 40003
    rng = np.random.default_rng(81)
    g2 = np.stack([W.t_mixture(d, 200 + r) * np.float32(10.0 ** rng.uniform(-3, 0)) for r in range(rows)])
    g2[:, ::13] = 0
    rhos, seeds = [0.02, 0.1, 0.4], [7, 8, 9]
    for solver in ("greedy", "exact"):
        idx, val, nnz, lam, k, fl = batched(L, g2, rhos, seeds, solver, ld=d + 5)
        ia, va, na, cb, nb, inv, q, lam2, fl2 = hybrid_batched(L, g2, rhos, seeds, solver, ld=d + 5)
        assert np.array_equal(lam, lam2) and not fl2.any()
        for r in range(rows):
            n = int(nnz[r])
            A, B = int(na[r]), int(nb[r])
            assert A + B == n and A == k[r]
            bi = cb[r, :B] & 0x7FFFFFFF
            neg = cb[r, :B] < 0
            merged = np.concatenate([ia[r, :A], bi])
            vals = np.concatenate([va[r, :A], np.where(neg, -inv[r], inv[r]).astype(np.float32)])
            o = np.argsort(merged, kind="stable")
            assert np.array_equal(merged[o], idx[r, :n]) and np.array_equal(vals[o], val[r, :n])
            assert np.array_equal(neg, g2[r][bi] < 0)
            assert np.all(q[r][ia[r, :A]] == 2) and np.array_equal(q[r][bi], np.where(neg, -1, 1).astype(np.int8))
            assert np.count_nonzero(q[r]) == n
            sol = oracle.solve(g2[r], rhos[r], solver, 2)
            h = oracle.sample_hybrid(g2[r], sol.p, seeds[r])
            if solver == "exact":  # identical lambda: identical capped set and survivors
                assert np.array_equal(ia[r, :A], h.qa_idx) and np.array_equal(bi, h.qb_idx)
                assert np.array_equal(q[r], h.q)
    if verbose:
        print("hybrid cases ok", flush=True)
    return True


def tied_boundary(d=40000, n_hi=3000, n_zero=3000, seed=5):
    """A vector whose exact solution at rho = 0.5 meets Algorithm 2's criterion with equality:
    n_hi entries of +-2, n_zero zeros and the rest +-1 at seeded positions (so ties fall in full
    and partial sample tiles), giving lambda = 0.5 and lambda * 2 = 1: the whole tied run of 2s has
    p_i = 1 and forms the capped set."""
    rng = np.random.default_rng(seed)
    g = np.where(rng.random(d) < 0.5, -1.0, 1.0).astype(np.float32)
    pos = rng.permutation(d)
    g[pos[:n_hi]] *= 2
    g[pos[n_hi:n_hi + n_zero]] = 0
    return g


def check_ties(L, verbose=True):
    """One capped test everywhere: the compaction (fast and scalar paths), the probabilities, the
    hybrid coding and the look-back's own recount all treat a coordinate with p_i = 1 as capped."""
    g = tied_boundary()
    hi = np.flatnonzero(np.abs(g) == 2)
    A = 3000.0 * 4 + 34000.0
    for solver, rho in (("exact", 0.5), ("variance", (3000.0 * 4 + 34000.0 / 0.5) / A - 1.0)):
        sol = oracle.solve(g, rho, solver)
        assert sol.k == hi.size
        idx, val, n, lam, k, fl = sample_row(L, g, rho, solver, 13)
        assert fl == 0 and lam == sol.lam and k == sol.k, (solver, lam, sol.lam, k, sol.k)
        compare_sample(g, sol.p, 13, idx, val, n, lam, sol.lam)
        assert np.all(np.isin(hi, idx))  # every capped coordinate survives
        # the same row at an unaligned start (scalar decisions everywhere)
        buf = np.zeros(g.size + 16, np.float32)
        base = (-buf.ctypes.data // 4) % 4 + 1
        view = buf[base:base + g.size]
        view[:] = g
        a = sample_row(L, view, rho, solver, 13)
        assert a[2] == n and a[4] == k and np.array_equal(a[0], idx) and np.array_equal(a[1], val)
        p, lam2, k2, fl2 = probs_row(L, g, rho, solver)
        assert k2 == sol.k and lam2 == sol.lam
        compare_probs(p, sol.p)
        ia, va, na, cb, nb, inv, q, lam3, fl3 = hybrid_batched(L, g[None, :], [rho], [13], solver)
        A_, B_ = int(na[0]), int(nb[0])
        assert not fl3.any() and A_ == hi.size and A_ + B_ == n
        assert np.array_equal(ia[0, :A_], hi) and np.array_equal(va[0, :A_], g[hi])
        bi = cb[0, :B_] & 0x7FFFFFFF
        assert np.all(np.diff(bi) > 0)
        merged = np.sort(np.concatenate([ia[0, :A_], bi]))
        assert np.array_equal(merged, idx)
        h = oracle.sample_hybrid(g, sol.p, 13)
        assert np.array_equal(ia[0, :A_], h.qa_idx) and np.array_equal(bi, h.qb_idx)
        assert np.array_equal(q[0], h.q)
    if verbose:
        print("tie cases ok", flush=True)
    return True


def row_state(ws, row=0):
    """Fields of a row's control block in a workspace after a call (offsets fixed by static
    asserts in the library source): the source of the last refinement request, the candidate
    band and the number of collected keys."""
    b = np.asarray(ws, np.uint8)[256 + 256 * row: 256 + 256 * (row + 1)]
    u32 = lambda o: int(b[o:o + 4].view(np.uint32)[0])
    return {"src": u32(192), "band_lo": u32(220), "band_hi": u32(224),
            "cand_n": int(b[232:240].view(np.uint64)[0]), "stage": u32(208)}


def sample_row_ws(L, g, rho, solver, seed, iters=2, ws_bytes=None):
    """sample_row that also returns the workspace, for row_state (a workspace of ws_bytes bytes
    when given, else the size the library asks for)."""
    d = g.size
    idx = np.zeros(d, np.int32)
    val = np.zeros(d, np.float32)
    nnz = np.zeros(1, np.int64)
    lam = np.zeros(1)
    k = np.zeros(1, np.int64)
    fl = np.zeros(1, np.uint32)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(1, d, sid) if ws_bytes is None else ws_bytes
    keep, ws = _aligned(wsb)
    rc = L.sparsify_sample_compact(g.ctypes.data, d, rho, sid, iters, seed, idx.ctypes.data, val.ctypes.data, d,
                                   nnz.ctypes.data, lam.ctypes.data, k.ctypes.data, fl.ctypes.data, ws.ctypes.data,
                                   wsb, None)
    assert rc == 0, rc
    n = int(nnz[0])
    return idx[:n], val[:n], n, float(lam[0]), int(k[0]), int(fl[0]), ws.copy()


def check_candidates(L, verbose=True):
    """Rows long enough for a candidate band (in the emulation build): the band is predicted, the keys in it
    are collected, refinement windows inside it read them, and every result still equals the
    oracle's (bit for bit in lambda for the exact solver). A row whose sample misleads the
    prediction (large magnitudes only on lines the sample skips) refines over the row instead."""
    used = 0
    for name, g in (("tmix", W.t_mixture(65536, 12)), ("tmix_ragged", W.t_mixture(50003, 13)),
                    ("ties", W.integer_ties(40000, 14))):
        g = np.ascontiguousarray(g, np.float32)
        for solver in ("greedy", "exact"):
            for rho in (0.01, 0.1, 0.4):
                sol = oracle.solve(g, rho, solver, 2)
                idx, val, n, lam, k, fl, ws = sample_row_ws(L, g, rho, solver, 21)
                st = row_state(ws)
                assert fl == 0, (name, solver, rho, fl)
                compare_sample(g, sol.p, 21, idx, val, n, lam, sol.lam)
                if solver == "exact":
                    assert lam == sol.lam and k == sol.k, (name, rho, lam, sol.lam, k, sol.k)
                if g.size % 4:
                    # a row length that is not a multiple of 4 takes the scalar-load path: no band
                    assert st["band_hi"] == st["band_lo"] and st["src"] == 0, (name, st)
                    continue
                if st["band_hi"] == st["band_lo"]:
                    # no band: the sample showed nothing capped (B times its largest magnitude well
                    # below its sum), so the solvers need no window
                    assert st["src"] == 0 and k == 0 or solver == "greedy", (name, st, k)
                    continue
                keys = np.abs(g).view(np.uint32)
                inband = int(np.count_nonzero((keys >= st["band_lo"]) & (keys < st["band_hi"])))
                # reserved slots: every key of the band, plus zeroed ends of the waves' reservations
                assert st["cand_n"] == inband, (name, st, inband)
                used += st["src"]
                if verbose:
                    print(f"{name} {solver} rho={rho}: band [{st['band_lo'] >> 23}, {st['band_hi'] >> 23}) "
                          f"cand={st['cand_n']} src={st['src']} stage={st['stage']}", flush=True)
    assert used > 0, "no refinement window was read from the candidates"
    # a misleading sample: the sample reads every 4th 64-byte line of this row (64 workgroups x 64
    # lines in the emulation build, of its 16384 lines); put all the large magnitudes on the other lines
    d = 1 << 18
    g = (W.normal(d, 15) * np.float32(1e-3)).astype(np.float32)
    lines = np.arange(d) // 16
    big = (lines % 4 != 0) & (np.arange(d) % 7 == 0)
    g[big] = W.t_mixture(int(big.sum()), 16) * np.float32(50)
    for solver in ("greedy", "exact"):
        sol = oracle.solve(g, 0.05, solver, 2)
        idx, val, n, lam, k, fl, ws = sample_row_ws(L, g, 0.05, solver, 22)
        st = row_state(ws)
        compare_sample(g, sol.p, 22, idx, val, n, lam, sol.lam)
        if solver == "exact":
            assert lam == sol.lam and k == sol.k
        if verbose:
            print(f"misleading sample {solver}: band [{st['band_lo'] >> 23}, {st['band_hi'] >> 23}) "
                  f"cand={st['cand_n']} src={st['src']}", flush=True)
    if verbose:
        print("candidate cases ok", flush=True)
    return True


def check_lowest_binade(L, verbose=True):
    """Exact solver with 1/lambda inside the row's lowest occupied binade (workloads.lowest_binade):
    no binade's maximum passes the criterion, and the solver refines that binade instead of giving
    up; lambda and k bit for bit, the sample under the parity rule, the probabilities too."""
    for d, rho in ((500, 0.96), (5003, 0.97)):
        g = W.lowest_binade(d, 3)
        sol = oracle.solve_exact(g, rho)
        assert 1.0e-3 <= 1.0 / sol.lam < 1.9e-3
        idx, val, n, lam, k, fl = sample_row(L, g, rho, "exact", 29)
        assert fl == 0 and lam == sol.lam and k == sol.k, (d, fl, lam, sol.lam, k, sol.k)
        compare_sample(g, sol.p, 29, idx, val, n, lam, sol.lam)
        p, lam2, k2, fl2 = probs_row(L, g, rho, "exact")
        assert fl2 == 0 and lam2 == sol.lam and k2 == sol.k
        compare_probs(p, sol.p)
        if verbose:
            print(f"lowest binade d={d} rho={rho}: k={k} lambda={lam!r}", flush=True)
    return True


def check_full_range(L, verbose=True):
    """Rows whose magnitudes span all of fp32's binades (workloads.full_range), both solvers, and a
    row of magnitudes in [2^120, 2^127.9) at rho = 0.01, whose 1/lambda lies beyond fp32's range: its
    amplified values are +-inf on both sides, as is the hybrid coding's shared 1/lambda."""
    rng = np.random.default_rng(12)
    for case in range(12):
        d = int(np.exp(rng.uniform(0.0, np.log(20000.0))))
        g = W.full_range(d, 100 + case)
        rho = float(10.0 ** rng.uniform(-3.0, 0.0))
        for solver in ("exact", "greedy"):
            sol = oracle.solve(g, rho, solver, 2)
            idx, val, n, lam, k, fl = sample_row(L, g, rho, solver, 31 + case)
            assert fl == 0, (case, solver, fl)
            compare_sample(g, sol.p, 31 + case, idx, val, n, lam, sol.lam)
            if solver == "exact":
                assert lam == sol.lam and k == sol.k, (case, lam, sol.lam, k, sol.k)
    r2 = np.random.default_rng(9)
    g = (r2.choice([-1.0, 1.0], 3001) * np.exp2(r2.uniform(120.0, 127.9, 3001))).astype(np.float32)
    for solver in ("exact", "greedy"):
        sol = oracle.solve(g, 0.01, solver, 2)
        assert sol.lam < 2.0 ** -128
        idx, val, n, lam, k, fl = sample_row(L, g, 0.01, solver, 5)
        assert fl == 0 and np.isinf(val[:n]).any()
        compare_sample(g, sol.p, 5, idx, val, n, lam, sol.lam)
        ia, va, na, cb, nb, inv, q, lam2, fl2 = hybrid_batched(L, g[None, :], [0.01], [5], solver)
        assert fl2[0] == 0 and lam2[0] == lam and inv[0] == np.inf and int(na[0] + nb[0]) == n
    if verbose:
        print("full-range rows ok", flush=True)
    return True


def _draw(rng, d):
    """A seeded random vector of length d: one of seven distributions, scaled over ten decades
    (the full-range one spans all of fp32's binades as it is)."""
    seed = int(rng.integers(1 << 30))
    kind = int(rng.integers(7))
    if kind == 0:
        g = W.normal(d, seed)
    elif kind == 1:
        g = W.t_mixture(d, seed)
    elif kind == 2:
        g = W.integer_ties(d, seed)
    elif kind == 3:
        g = W.wide_range(d, seed)
    elif kind == 4:
        g = W.two_level(d, max(1, d // 50), 30.0, 1.0, seed)
    elif kind == 5:
        return W.full_range(d, seed)
    else:
        g = W.approx_sparse(d, max(1, d // 20), 0.05, seed) if d >= 20 else W.normal(d, seed)
    return (g * np.float32(10.0 ** rng.uniform(-6, 4))).astype(np.float32)


def _random_row(rng, dmax):
    """A seeded random row: log-uniform length up to dmax, random distribution, density and solver."""
    d = int(np.exp(rng.uniform(0.0, np.log(dmax))))
    g = _draw(rng, d)
    return g, float(10.0 ** rng.uniform(-3.5, 0.0)), ("greedy", "exact")[int(rng.integers(2))], int(rng.integers(100000))


def check_random(L, verbose=True, cases=40, seed=4242):
    """Seeded random rows (up to 60 K coordinates) for the density solvers and the variance budget,
    padded batches of one random length and segmented layouts with random lengths (empty segments
    among them), each against the oracle; lambda and k bit for bit for the exact solvers."""
    rng = np.random.default_rng(seed)
    for case in range(cases):
        g, rho, solver, seed = _random_row(rng, 60000.0)
        sol = oracle.solve(g, rho, solver, 2)
        idx, val, n, lam, k, fl = sample_row(L, g, rho, solver, seed)
        assert fl == (0 if g.any() else 4), (case, fl)
        compare_sample(g, sol.p, seed, idx, val, n, lam, sol.lam)
        if solver == "exact":
            assert lam == sol.lam and k == sol.k, (case, lam, sol.lam, k, sol.k)
    for case in range(cases // 4):
        g = _draw(rng, int(np.exp(rng.uniform(0.0, np.log(60000.0)))))
        eps = float(10.0 ** rng.uniform(-3.0, 1.0))
        sol = oracle.solve_variance(g, eps)
        idx, val, n, lam, k, fl = sample_row(L, g, eps, "variance", 50 + case)
        assert fl == (0 if g.any() else 4), (case, fl)
        compare_sample(g, sol.p, 50 + case, idx, val, n, lam, sol.lam)
        assert lam == sol.lam and k == sol.k, (case, eps, lam, sol.lam, k, sol.k)
    for case in range(cases // 4):
        rows = int(rng.integers(1, 6))
        d = int(np.exp(rng.uniform(0.0, np.log(30000.0))))
        solver = ("greedy", "exact")[case % 2]
        g2 = np.stack([_draw(rng, d) for _ in range(rows)])
        rhos = [float(10.0 ** rng.uniform(-3.0, 0.0)) for _ in range(rows)]
        seeds = [int(rng.integers(1 << 40)) for _ in range(rows)]
        idx, val, nnz, lam, k, fl = batched(L, g2, rhos, seeds, solver, ld=d + int(rng.integers(0, 9)))
        for r in range(rows):
            sol = oracle.solve(g2[r], rhos[r], solver, 2)
            n = int(nnz[r])
            assert fl[r] == (0 if g2[r].any() else 4), (case, r, fl[r])
            compare_sample(g2[r], sol.p, seeds[r], idx[r, :n], val[r, :n], n, lam[r], sol.lam)
            if solver == "exact":
                assert lam[r] == sol.lam and k[r] == sol.k
    for case in range(cases // 4):
        segs = int(rng.integers(1, 9))
        lengths = [int(np.exp(rng.uniform(0.0, np.log(20000.0)))) if rng.random() > 0.15 else 0 for _ in range(segs)]
        g, off = layered(lengths, 1300 + case)
        rhos = [float(10.0 ** rng.uniform(-3.0, 0.0)) for _ in range(segs)]
        seeds = [int(rng.integers(1 << 30)) for _ in range(segs)]
        solver = ("exact", "greedy")[case % 2]
        idx, val, nnz, lam, k, fl = segmented(L, g, off, rhos, seeds, solver, g_shift=int(rng.integers(0, 4)))
        ref = oracle.sparsify_segments(g, off, rhos, seeds, solver)
        for s_ in range(segs):
            seg = g[off[s_]:off[s_ + 1]]
            n = int(nnz[s_])
            if seg.size == 0 or not np.any(seg):
                assert n == 0 and fl[s_] & 4
                continue
            sol = ref[s_][0]
            assert fl[s_] == 0
            compare_sample(seg, sol.p, seeds[s_], idx[s_, :n], val[s_, :n], n, lam[s_], sol.lam)
            if solver == "exact":
                assert lam[s_] == sol.lam and k[s_] == sol.k
    if verbose:
        print("random cases ok", flush=True)
    return True


def check_lane_rows(L, verbose=True):
    """Capped coordinates that one decide-phase lane takes beyond its LDS row (workloads.strided_large):
    those waves read their capped values from g while emitting, lane by lane (rho 0.01, 0.05) or
    group by group (rho 0.5), in the compaction and the hybrid coding; every capped coordinate
    survives with value g_i and the rest follows the oracle. (One tile and a ragged tail: the
    patterns lie in the first tile.)"""
    g = W.strided_large(16384 + 123, 7)
    big = np.flatnonzero(np.abs(g) >= 100.0)
    for rho in (0.01, 0.05, 0.5):
        for solver in ("exact", "greedy"):
            sol = oracle.solve(g, rho, solver, 2)
            idx, val, n, lam, k, fl = sample_row(L, g, rho, solver, 17)
            assert fl == 0, fl
            compare_sample(g, sol.p, 17, idx, val, n, lam, sol.lam)
            assert np.all(np.isin(big, idx)) and np.array_equal(val[np.isin(idx, big)], g[big])
            ia, va, na, cb, nb, inv, q, lam3, fl3 = hybrid_batched(L, g[None, :], [rho], [17], solver)
            A_, B_ = int(na[0]), int(nb[0])
            assert not fl3.any() and A_ + B_ == n
            bi = cb[0, :B_] & 0x7FFFFFFF
            assert np.all(np.isin(big, ia[0, :A_])) and np.array_equal(va[0, :A_], g[ia[0, :A_]])
            assert np.array_equal(np.sort(np.concatenate([ia[0, :A_], bi])), idx)
            if verbose:
                print(f"lane rows {solver} rho={rho}: nnz={n} capped={k}", flush=True)
    return True


def check_band_region_overflow(L, verbose=True):
    """A band row whose first statistics workgroup holds more band keys than its staging region:
    2^17 coordinates, a workspace with room for 2^16 candidates (16 regions of 4096 for chunks of
    8192), the first chunk's magnitudes uniform in [8, 16) and the rest 1e-3 N(0, 1), rho putting
    1/lambda near 12. The band is predicted and collected, the overflowing region makes the first
    solve drop it, the solver refines over the row, and the result equals the oracle's (lambda bit
    for bit for the exact solver)."""
    d = 1 << 17
    rng = np.random.default_rng(92)
    g = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    big = rng.uniform(8.0, 16.0, 8192) * np.where(rng.random(8192) < 0.5, -1.0, 1.0)
    g[:8192] = big.astype(np.float32)
    rho = 0.0574
    fixed = L.gspar_workspace_bytes(1, d, 2)  # the layout without candidate buffers
    for solver in ("greedy", "exact"):
        sol = oracle.solve(g, rho, solver, 2)
        assert sol.k > 0 and 8.0 <= 1.0 / sol.lam < 16.0, (sol.k, sol.lam)
        idx, val, n, lam, k, fl, ws = sample_row_ws(L, g, rho, solver, 23, ws_bytes=fixed + 8 * (1 << 16) + 4096)
        st = row_state(ws)
        if verbose:
            print(f"region overflow {solver}: band [{st['band_lo'] >> 23}, {st['band_hi'] >> 23}) "
                  f"cand={st['cand_n']} src={st['src']}", flush=True)
        assert fl == 0, fl
        # collected (the count exceeds the list's capacity: the overflowing region reserved past
        # it), then dropped by the first solve, and no window read the candidates
        assert st["cand_n"] > (1 << 16) and st["band_lo"] == st["band_hi"] == 0 and st["src"] == 0, st
        compare_sample(g, sol.p, 23, idx, val, n, lam, sol.lam)
        if solver == "exact":
            assert lam == sol.lam and k == sol.k, (lam, sol.lam, k, sol.k)
    return True


def segmented(L, g, off, rhos, seeds, solver, iters=2, cap=None, off_dev=None, g_shift=0):
    """sparsify_sample_compact_segmented on a flat host vector (placed g_shift floats past a
    16-byte boundary); off_dev defaults to the host offsets."""
    off = np.ascontiguousarray(off, np.int64)
    od = off.copy() if off_dev is None else np.ascontiguousarray(off_dev, np.int64)
    segs = off.size - 1
    lens = np.diff(off)
    maxlen = max(1, int(lens.max()))
    raw = np.zeros(g.size + 8, np.float32)
    base = (-raw.ctypes.data // 4) % 4 + g_shift
    buf = raw[base:base + g.size]
    buf[:] = g
    cap = maxlen if cap is None else cap
    idx = np.zeros((segs, max(cap, 1)), np.int32)
    val = np.zeros((segs, max(cap, 1)), np.float32)
    nnz = np.zeros(segs, np.int64)
    lam = np.zeros(segs)
    k = np.zeros(segs, np.int64)
    fl = np.zeros(segs, np.uint32)
    r = np.ascontiguousarray(rhos, np.float64)
    s = np.array([int(x) & 0xFFFFFFFFFFFFFFFF for x in seeds], np.uint64)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(segs, maxlen, sid)
    keep, ws = _aligned(wsb)
    rc = L.sparsify_sample_compact_segmented(buf.ctypes.data, segs, off.ctypes.data, od.ctypes.data, r.ctypes.data,
                                             sid, iters, s.ctypes.data, idx.ctypes.data, val.ctypes.data, cap,
                                             nnz.ctypes.data, lam.ctypes.data, k.ctypes.data, fl.ctypes.data,
                                             ws.ctypes.data, wsb, None)
    assert rc == 0, rc
    return idx, val, nnz, lam, k, fl


def hybrid_segmented(L, g, off, rhos, seeds, solver, iters=2):
    off = np.ascontiguousarray(off, np.int64)
    segs = off.size - 1
    maxlen = max(1, int(np.diff(off).max()))
    gg = np.ascontiguousarray(g, np.float32)
    cap = maxlen
    ia = np.zeros((segs, cap), np.int32)
    va = np.zeros((segs, cap), np.float32)
    cb = np.zeros((segs, cap), np.int32)
    na = np.zeros(segs, np.int64)
    nb = np.zeros(segs, np.int64)
    inv = np.zeros(segs, np.float32)
    q = np.full(g.size, 7, np.int8)
    lam = np.zeros(segs)
    fl = np.zeros(segs, np.uint32)
    r = np.ascontiguousarray(rhos, np.float64)
    sd = np.array([int(x) & 0xFFFFFFFFFFFFFFFF for x in seeds], np.uint64)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(segs, maxlen, sid)
    keep, ws = _aligned(wsb)
    rc = L.sparsify_sample_hybrid_segmented(gg.ctypes.data, segs, off.ctypes.data, off.ctypes.data, r.ctypes.data,
                                            sid, iters, sd.ctypes.data, ia.ctypes.data, va.ctypes.data, cap,
                                            na.ctypes.data, cb.ctypes.data, cap, nb.ctypes.data, inv.ctypes.data,
                                            q.ctypes.data, lam.ctypes.data, fl.ctypes.data, ws.ctypes.data, wsb, None)
    assert rc == 0, rc
    return ia, va, na, cb, nb, inv, q, lam, fl


def probs_segmented(L, g, off, rhos, solver, iters=2):
    off = np.ascontiguousarray(off, np.int64)
    segs = off.size - 1
    maxlen = max(1, int(np.diff(off).max()))
    p = np.full(g.size, -1.0, np.float32)
    lam = np.zeros(segs)
    k = np.zeros(segs, np.int64)
    fl = np.zeros(segs, np.uint32)
    r = np.ascontiguousarray(rhos, np.float64)
    sid = {"greedy": 0, "exact": 1, "variance": 2}[solver]
    wsb = L.gspar_workspace_bytes(segs, maxlen, sid)
    keep, ws = _aligned(wsb)
    gg = np.ascontiguousarray(g, np.float32)
    rc = L.sparsify_probs_segmented(gg.ctypes.data, segs, off.ctypes.data, off.ctypes.data, r.ctypes.data, sid,
                                    iters, p.ctypes.data, lam.ctypes.data, k.ctypes.data, fl.ctypes.data,
                                    ws.ctypes.data, wsb, None)
    assert rc == 0, rc
    return p, lam, k, fl


def layered(lengths, seed):
    """A flat gradient of layers with per-layer scales 10^U(-4, 0) and mixed shapes."""
    rng = np.random.default_rng(seed)
    parts = []
    for i, n in enumerate(lengths):
        mk = (W.t_mixture, W.normal, W.integer_ties)[i % 3]
        parts.append(mk(n, seed + i) * np.float32(10.0 ** rng.uniform(-4, 0)) if n else np.zeros(0, np.float32))
    return np.concatenate(parts).astype(np.float32), np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)


def check_segmented(L, verbose=True):
    """Per-layer sparsification (Section 5.2) against the oracle segment by segment, aligned and
    unaligned offsets, empty and tiny layers, layers spanning several tiles, and device offsets
    that disagree with the host's."""
    # offsets that are not all multiples of 4 (scalar path), then aligned ones (vector path); an
    # unaligned g takes the scalar path too
    for lengths, shift in (([3000, 0, 3, 16384 + 8, 1, 5000, 4], 0), ([4096, 16388, 12, 12000, 0, 8], 0)):
        g, off = layered(lengths, 600 + len(lengths))
        segs = len(lengths)
        rhos = [(0.01, 0.1, 0.5, 0.3, 1.0, 0.05, 0.2)[i % 7] for i in range(segs)]
        seeds = [7000 + i for i in range(segs)]
        for solver in ("greedy", "exact"):
            idx, val, nnz, lam, k, fl = segmented(L, g, off, rhos, seeds, solver, g_shift=shift)
            ref = oracle.sparsify_segments(g, off, rhos, seeds, solver)
            for s_ in range(segs):
                seg = g[off[s_]:off[s_ + 1]]
                n = int(nnz[s_])
                if seg.size == 0 or not np.any(seg):
                    assert n == 0 and fl[s_] & 4, (s_, n, fl[s_])
                    continue
                assert fl[s_] == 0, (s_, fl[s_])
                sol = ref[s_][0]
                compare_sample(seg, sol.p, seeds[s_], idx[s_, :n], val[s_, :n], n, lam[s_], sol.lam)
                if solver == "exact":
                    assert lam[s_] == sol.lam and k[s_] == sol.k
                if solver == "exact" and shift == 0:  # a segment equals a single-row call on it
                    one = sample_row(L, np.ascontiguousarray(seg), rhos[s_], solver, seeds[s_])
                    assert one[2] == n and np.array_equal(one[0], idx[s_, :n])
                    assert np.array_equal(one[1], val[s_, :n])
            # the hybrid coding of the same call: the same survivors split by the capped set
            ia, va, na, cb, nb, inv, q, lam3, fl3 = hybrid_segmented(L, g, off, rhos, seeds, solver)
            assert np.array_equal(lam3, lam, equal_nan=True) and np.array_equal(fl3, fl)
            for s_ in range(segs):
                n, A, B = int(nnz[s_]), int(na[s_]), int(nb[s_])
                assert A + B == n and A == k[s_]
                bi = cb[s_, :B] & 0x7FFFFFFF
                merged = np.concatenate([ia[s_, :A], bi])
                vals = np.concatenate([va[s_, :A], np.where(cb[s_, :B] < 0, -inv[s_], inv[s_]).astype(np.float32)])
                o = np.argsort(merged, kind="stable")
                assert np.array_equal(merged[o], idx[s_, :n]) and np.array_equal(vals[o], val[s_, :n])
                qs = q[off[s_]:off[s_ + 1]]
                assert np.count_nonzero(qs) == n and np.all(qs[ia[s_, :A]] == 2)
            if solver == "greedy":
                continue
            p, lam2, k2, fl2 = probs_segmented(L, g, off, rhos, "exact")
            for s_ in range(segs):
                seg = g[off[s_]:off[s_ + 1]]
                if seg.size and np.any(seg):
                    compare_probs(p[off[s_]:off[s_ + 1]], oracle.solve_exact(seg, rhos[s_]).p)
    # device offsets that break the host's bounds (a start that is not a multiple of 4 on the vector
    # path, an end past the host's last offset) change the launch shape: every segment is flagged
    # and skipped, and a later call with the right offsets on the same workspace runs normally
    g, off = layered([4000, 8000, 4000], 650)
    bad = off.copy()
    bad[1] = 4001
    bad[3] = off[3] + 400
    idx, val, nnz, lam, k, fl = segmented(L, g, off, [0.1] * 3, [1, 2, 3], "greedy", off_dev=bad)
    assert np.all(fl & 32) and not nnz.any() and np.isnan(lam).all()
    idx, val, nnz, lam, k, fl = segmented(L, g, off, [0.1] * 3, [1, 2, 3], "greedy")
    assert not fl.any() and np.all(nnz > 0)
    if verbose:
        print("segmented cases ok", flush=True)
    return True


def check_variance(L, verbose=True):
    """Algorithm 2 with the variance budget: lambda and k bit for bit, the sample under the parity
    rule, p within 1e-6."""
    cases = [("normal", W.normal(9001, 1)), ("tmix", W.t_mixture(17001, 2)), ("ties", W.integer_ties(8001, 3)),
             ("two_level", W.two_level(6001, 40, 50.0, 1.0, 5)), ("wide", W.wide_range(6000, 4)),
             ("approx_sparse", W.approx_sparse(5000, 60, 0.05, 6)), ("tiny", W.normal(7, 7))]
    for name, g in cases:
        g = np.ascontiguousarray(g, np.float32)
        for eps in (0.0, 0.05, 5.0):
            sol = oracle.solve_variance(g, eps)
            idx, val, n, lam, k, fl = sample_row(L, g, eps, "variance", 31)
            assert fl == 0, (name, eps, fl)
            assert lam == sol.lam and k == sol.k, (name, eps, lam, sol.lam, k, sol.k)
            compare_sample(g, sol.p, 31, idx, val, n, lam, sol.lam)
            if eps == 0.05:
                p, lam2, k2, fl2 = probs_row(L, g, eps, "variance")
                assert lam2 == sol.lam
                compare_probs(p, sol.p)
    if verbose:
        print("variance cases ok", flush=True)
    return True


def aggregate(L, idx, val, nnz, d):
    """gspar_aggregate on [workers, cap] lists; returns v [d]."""
    workers, cap = idx.shape
    v = np.full(d, np.nan, np.float32)
    nn = np.ascontiguousarray(nnz, np.int64)
    rc = L.gspar_aggregate(idx.ctypes.data, val.ctypes.data, cap, nn.ctypes.data, workers, d, v.ctypes.data, None)
    assert rc == 0, rc
    return v


def _lists(idx, val, nnz):
    cap = idx.shape[1]
    return [(idx[m, :max(0, min(int(n), cap))], val[m, :max(0, min(int(n), cap))]) for m, n in enumerate(nnz)]


def check_aggregate(L, verbose=True):
    """Algorithm 1, step 6: bit-exact against the oracle's worker-order fp64 average."""
    # the sampling pass's own lists: a batch of workers of one gradient size
    rows, d = 5, 20011
    rng = np.random.default_rng(91)
    g2 = np.stack([W.t_mixture(d, 300 + r) * np.float32(10.0 ** rng.uniform(-3, 0)) for r in range(rows)])
    for rho in (0.01, 0.3, 1.0):
        idx, val, nnz, lam, k, fl = batched(L, g2, [rho] * rows, [40 + r for r in range(rows)], "greedy")
        v = aggregate(L, idx, val, nnz, d)
        assert np.array_equal(v, oracle.aggregate(_lists(idx, val, nnz), d), equal_nan=True)
    # synthetic lists: more workers than one pass holds, empty and overflowing lists, ragged d,
    # long ranges inside one block, a single worker
    for i, (workers, d, cap) in enumerate(((37, 10007, 3000), (1, 4096 * 3 + 5, 9000), (16, 2048, 2048),
                                           (17, 999, 400))):
        idx, val, nnz = W.sparse_lists(workers, d, cap, 500 + i, empty=(1, 2) if workers > 2 else (), over=(0,))
        v = aggregate(L, idx, val, nnz, d)
        assert np.array_equal(v, oracle.aggregate(_lists(idx, val, nnz), d)), (workers, d, cap)
    # zero capacity: every list empty
    v = aggregate(L, np.zeros((3, 0), np.int32), np.zeros((3, 0), np.float32), np.array([5, 0, 2]), 5000)
    assert np.array_equal(v, np.zeros(5000, np.float32))
    # lists that break the contract: out-of-range indices are skipped, disorder never reads outside
    idx, val, nnz = W.sparse_lists(4, 6000, 1500, 510)
    idx[0, :3] = [-5, -1, 0]
    idx[0, 3:] = np.sort(idx[0, 3:])
    idx[1, :nnz[1]] = np.minimum(idx[1, :nnz[1]] + 5990, 2**31 - 1)
    idx[2, :nnz[2]] = rng.permutation(idx[2, :nnz[2]])
    v = aggregate(L, idx, val, nnz, 6000)
    assert v.shape == (6000,) and not np.isnan(v).any()
    if verbose:
        print("aggregate cases ok", flush=True)
    return True


def check_asan_subset(L, verbose=True):
    """A bounded selection for the AddressSanitizer build: every kernel family once, on shapes that
    reach the ragged ends. A padded batch whose rows end in a partial group on the vector path
    (long enough for a candidate band in the emulation build), the scalar path, the variance budget,
    segments on both paths with the hybrid coding, and aggregation of the batch's lists."""
    rows, d = 2, 12003
    g2 = np.stack([W.t_mixture(d, 310 + r) for r in range(rows)])
    for solver, ld, rhos in (("greedy", d + 1, [0.1, 0.01]), ("exact", d + 1, [0.01, 0.1]), ("exact", d + 2, [0.05, 0.2])):
        seeds = [3 + r for r in range(rows)]
        idx, val, nnz, lam, k, fl = batched(L, g2, rhos, seeds, solver, ld=ld)
        assert not fl.any(), fl
        for r in range(rows):
            sol = oracle.solve(g2[r], rhos[r], solver, 2)
            n = int(nnz[r])
            compare_sample(g2[r], sol.p, seeds[r], idx[r, :n], val[r, :n], n, lam[r], sol.lam)
            if solver == "exact":
                assert lam[r] == sol.lam and k[r] == sol.k
        v = aggregate(L, idx, val, nnz, d)
        assert np.array_equal(v, oracle.aggregate(_lists(idx, val, nnz), d), equal_nan=True)
    g = np.ascontiguousarray(W.t_mixture(9001, 2), np.float32)
    sol = oracle.solve_variance(g, 0.05)
    idx, val, n, lam, k, fl = sample_row(L, g, 0.05, "variance", 31)
    assert fl == 0 and lam == sol.lam and k == sol.k
    compare_sample(g, sol.p, 31, idx, val, n, lam, sol.lam)
    for lengths in ([3000, 0, 3, 16384 + 8, 1], [4096, 16388, 12, 0, 8]):
        g, off = layered(lengths, 620 + len(lengths))
        segs = len(lengths)
        rhos = [(0.01, 0.1, 0.5, 0.3, 1.0)[i % 5] for i in range(segs)]
        seeds = [7100 + i for i in range(segs)]
        idx, val, nnz, lam, k, fl = segmented(L, g, off, rhos, seeds, "exact")
        ref = oracle.sparsify_segments(g, off, rhos, seeds, "exact")
        for s_ in range(segs):
            seg = g[off[s_]:off[s_ + 1]]
            n = int(nnz[s_])
            if seg.size == 0 or not np.any(seg):
                assert n == 0 and fl[s_] & 4
                continue
            sol = ref[s_][0]
            compare_sample(seg, sol.p, seeds[s_], idx[s_, :n], val[s_, :n], n, lam[s_], sol.lam)
            assert lam[s_] == sol.lam and k[s_] == sol.k
        ia, va, na, cb, nb, inv, q, lam3, fl3 = hybrid_segmented(L, g, off, rhos, seeds, "exact")
        assert np.array_equal(lam3, lam, equal_nan=True) and np.all(na + nb == nnz)
    if verbose:
        print("asan subset ok", flush=True)
    return True


def run_extra(path, verbose=True, lite=False):
    """Edge cases, batching, overflow and the unaligned path; `lite` (for reruns of the same cases
    under other launch conditions) keeps one greedy step count and skips the single-row repeats."""
    L = load(path)
    # greedy step counts
    g = W.t_mixture(30001, 11)
    for T in ((2,) if lite else (0, 1, 3, 8)):
        for rho in (0.01, 0.3):
            sol = oracle.solve_greedy(g, rho, T)
            idx, val, n, lam, k, fl = sample_row(L, g, rho, "greedy", 5, iters=T)
            compare_sample(g, sol.p, 5, idx, val, n, lam, sol.lam)
    # special cases
    d = 10000
    idx, val, n, lam, k, fl = sample_row(L, np.zeros(d, np.float32), 0.1, "exact", 0, cap=10)
    assert n == 0 and fl & 4
    h = W.normal(d, 41)
    h[::3] = 0
    nzi = np.flatnonzero(h)
    for solver in ("greedy", "exact"):
        idx, val, n, lam, k, fl = sample_row(L, h, 0.0, solver, 0, cap=10)
        assert n == 0 and lam == 0.0 and fl == 0
        for rho in (1.0, 0.7):
            idx, val, n, lam, k, fl = sample_row(L, h, rho, solver, 0, cap=d)
            assert n == nzi.size and np.array_equal(idx, nzi) and np.array_equal(val, h[nzi]) and np.isinf(lam)
    for bad in (np.inf, np.nan):
        q = W.normal(d, 42)
        q[1234] = bad
        idx, val, n, lam, k, fl = sample_row(L, q, 0.1, "greedy", 0, cap=100)
        assert n == 0 and fl & 1 and np.isnan(lam)
    # capacity overflow
    g = W.t_mixture(40000, 51)
    sol = oracle.solve_exact(g, 0.1)
    idx, val, n, lam, k, fl = sample_row(L, g, 0.1, "exact", 9, cap=333)
    assert fl & 2 and n > 333
    compare_sample(g, sol.p, 9, idx, val, n, lam, sol.lam, cap=333)
    # batched rows with a padded leading dimension, per-row rho and seeds, and a bad rho
    rows, d = 6, 12003
    rng = np.random.default_rng(71)
    g2 = np.stack([W.t_mixture(d, 100 + r) * np.float32(10.0 ** rng.uniform(-3, 0)) for r in range(rows)])
    rhos = [0.01, 0.1, 0.3, 0.001, 0.5, 0.05]
    seeds = [1000, 1001, 0xFFFFFFFFFFFFFFF1, 3, 4, 5]
    for solver in ("greedy", "exact"):
        idx, val, nnz, lam, k, fl = batched(L, g2, rhos, seeds, solver, ld=d + 13)
        for r in range(rows):
            sol = oracle.solve(g2[r], rhos[r], solver, 2)
            n = int(nnz[r])
            compare_sample(g2[r], sol.p, seeds[r], idx[r, :n], val[r, :n], n, lam[r], sol.lam)
            if not lite:
                one = sample_row(L, np.ascontiguousarray(g2[r]), rhos[r], solver, seeds[r])
                assert one[2] == n and np.array_equal(one[0], idx[r, :n]) and np.array_equal(one[1], val[r, :n])
                assert one[3] == lam[r]
    idx, val, nnz, lam, k, fl = batched(L, g2[:2], [0.1, 1.5], [1, 2], "greedy")
    assert fl[1] & 8 and nnz[1] == 0 and fl[0] == 0 and nnz[0] > 0
    # unaligned row start (scalar-load path)
    g = W.t_mixture(20001, 61)
    buf = np.zeros(20002 + 16, np.float32)
    base = (-buf.ctypes.data // 4) % 4 + 1  # a start that is not 16-byte aligned
    view = buf[base:base + 20001]
    view[:] = g
    assert view.ctypes.data % 16 != 0
    a = sample_row(L, view, 0.05, "exact", 3)
    b = sample_row(L, g, 0.05, "exact", 3)
    assert a[2] == b[2] and np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    if verbose:
        print("extra cases ok", flush=True)
    return True


if __name__ == "__main__":
    which = sys.argv[2] if len(sys.argv) > 2 else "all"
    if which in ("all", "extra"):
        run_extra(sys.argv[1])
    if which == "extra_lite":
        run_extra(sys.argv[1], lite=True)
    if which in ("all", "hybrid"):
        check_hybrid(load(sys.argv[1]))
    if which in ("all", "ties"):
        check_ties(load(sys.argv[1]))
    if which in ("all", "candidates"):
        check_candidates(load(sys.argv[1]))
    if which in ("all", "aggregate"):
        check_aggregate(load(sys.argv[1]))
    if which in ("all", "variance"):
        check_variance(load(sys.argv[1]))
    if which in ("all", "segmented"):
        check_segmented(load(sys.argv[1]))
    if which in ("all", "edges"):
        L = load(sys.argv[1])
        check_lowest_binade(L)
        check_full_range(L)
        check_lane_rows(L)
        check_band_region_overflow(L)
    if which in ("all", "random"):
        check_random(load(sys.argv[1]))
    if which == "asan_subset":
        check_asan_subset(load(sys.argv[1]))
    if which in ("all", "main"):
        print("checked", run_all(sys.argv[1]))
