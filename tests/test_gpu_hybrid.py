"""GPU parity of the hybrid coding (Section 3.3, eqs. 9-10) through the C ABI: Q_A holds the capped
survivors as (index, value), Q_B the others as index | sign << 31, sharing the float 1/lambda; the
optional dense ternary vector marks 2 on the capped set and sign(g_i) on Q_B. Checked against the
oracle's split under the parity rule (index sets equal except where |u_i - p_i| <= 1e-6, values to
rel 1e-5, lambda to rel 1e-9; for the exact solver, whose lambda is bit-identical, the capped set,
both lists and the ternary vector are compared exactly), and bit for bit against the compaction
entry point on the same arguments, up to the workloads' full sizes."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from oracle.compare import compare_sample, lam_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def gs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1710_09854_amd as m

    m.lib()
    return m


def _merge(idx_a, val_a, code_b, inv):
    """Q_A and Q_B back into ascending (index, value) pairs, Q_B's value being sign / lambda."""
    bi = code_b & 0x7FFFFFFF
    neg = code_b < 0
    idx = np.concatenate([idx_a, bi])
    val = np.concatenate([val_a, np.where(neg, -inv, inv).astype(np.float32)])
    o = np.argsort(idx, kind="stable")
    return idx[o], val[o], bi, neg


VECTORS = {
    "normal_ragged_100003": lambda: W.normal(100003, 1),
    "tmix_200001": lambda: W.t_mixture(200001, 2),
    "ties_50001": lambda: W.integer_ties(50001, 3),
    "wide_range_120000": lambda: W.wide_range(120000, 4),
    "two_level_70001": lambda: W.two_level(70001, 300, 50.0, 1.0, 5),
    "approx_sparse_40000": lambda: W.approx_sparse(40000, 200, 0.05, 6),
    "tiny_7": lambda: W.normal(7, 7),
}


@pytest.mark.parametrize("name", list(VECTORS))
@pytest.mark.parametrize("solver", ["greedy", "exact"])
@pytest.mark.parametrize("rho", [0.01, 0.1, 0.5])
def test_hybrid_row_parity(gs, name, solver, rho):
    g = VECTORS[name]()
    g[::17] = 0
    d = g.size
    seed = 4321 + len(name)
    _say(f"[hybrid] {name} d={d} solver={solver} rho={rho} seed={seed}")
    gd = torch.from_numpy(g).cuda()
    h = gs.sparsify_sample_hybrid(gd, rho, seed=seed, solver=solver, cap_a=d, cap_b=d, dense_q=True)
    c = gs.sparsify_sample_compact(gd, rho, seed=seed, solver=solver, capacity=d)
    torch.cuda.synchronize()
    assert int(h.flags.item()) == 0 and int(c.flags.item()) == 0
    A, B, n = int(h.n_a.item()), int(h.n_b.item()), int(c.nnz.item())
    lam = float(h.lam.item())
    inv = np.float32(h.inv_lam.item())
    assert A + B == n and A == int(c.k.item()) and lam == float(c.lam.item())
    ia, va, cb = h.idx_a[:A].cpu().numpy(), h.val_a[:A].cpu().numpy(), h.code_b[:B].cpu().numpy()
    idx, val, bi, neg = _merge(ia, va, cb, inv)
    # the same survivors and values as the compaction of the same call
    assert np.array_equal(idx, c.idx[:n].cpu().numpy()) and np.array_equal(val, c.val[:n].cpu().numpy())
    assert np.array_equal(neg, g[bi] < 0) and np.array_equal(va, g[ia])
    if np.isfinite(lam) and lam > 0:
        assert inv == np.float32(1.0 / lam)
    # the capped set by the returned lambda, and the dense ternary vector
    capped = lam * np.abs(g.astype(np.float64)) >= 1.0 if np.isfinite(lam) else g != 0
    assert np.array_equal(ia, np.flatnonzero(capped))
    q = h.q.cpu().numpy()
    assert np.all(q[ia] == 2) and np.array_equal(q[bi], np.where(neg, -1, 1).astype(np.int8))
    assert np.count_nonzero(q) == n
    # against the oracle
    sol = oracle.solve(g, rho, solver, 2)
    rep = compare_sample(g, sol.p, seed, idx, val, n, lam, sol.lam)
    if solver == "exact":
        o = oracle.sample_hybrid(g, sol.p, seed)
        assert lam == sol.lam
        assert np.array_equal(ia, o.qa_idx) and np.array_equal(bi, o.qb_idx) and np.array_equal(q, o.q)
        assert gs.coding_bits(d, A, B, int(neg.sum())) == pytest.approx(
            oracle.coding_bits(d, o.qa_idx.size, o.qb_idx.size, int(o.qb_neg.sum())), rel=1e-12)
    _say(f"   ok n_a={A} n_b={B} excused={rep['excused']} lam={lam:.12g}")


@pytest.mark.parametrize("name", ["c2", "c4", "c5"])
def test_hybrid_equals_compaction_full_size(gs, name):
    """At the workloads' full sizes, in the batched launch configuration: the hybrid lists merge
    into exactly the compaction's output, for every solver the workload lists, at its largest rho."""
    wl = W.CONFIGS[name]()
    rows, d = wl.rows, wl.d
    rho = max(wl.rhos)
    g = torch.from_numpy(wl.g).cuda()
    for solver in W.CONFIG_SOLVERS[name]:
        _say(f"[hybrid-full] {name} rows={rows} d={d} solver={solver} rho={rho}")
        cap = gs.capacity_hint(d, rho)
        h = gs.sparsify_sample_hybrid_batched(g, [rho] * rows, wl.seeds, solver=solver, iters=wl.iters, cap_a=cap,
                                              cap_b=cap)
        c = gs.sparsify_sample_compact_batched(g, [rho] * rows, wl.seeds, solver=solver, iters=wl.iters,
                                               cap_per_row=cap)
        torch.cuda.synchronize()
        assert not h.flags.any().item() and not c.flags.any().item()
        for r in range(rows):
            A, B, n = int(h.n_a[r].item()), int(h.n_b[r].item()), int(c.nnz[r].item())
            assert A + B == n
            idx, val, bi, neg = _merge(h.idx_a[r, :A].cpu().numpy(), h.val_a[r, :A].cpu().numpy(),
                                       h.code_b[r, :B].cpu().numpy(), np.float32(h.inv_lam[r].item()))
            assert np.array_equal(idx, c.idx[r, :n].cpu().numpy()) and np.array_equal(val, c.val[r, :n].cpu().numpy())
            assert np.array_equal(neg, wl.g[r][bi] < 0)
        _say(f"   ok row0 n_a={int(h.n_a[0].item())} n_b={int(h.n_b[0].item())}")
    del g


def test_hybrid_overflow_and_special_cases(gs):
    g = W.t_mixture(50000, 91)
    gd = torch.from_numpy(g).cuda()
    full = gs.sparsify_sample_hybrid(gd, 0.1, seed=3, solver="exact", cap_a=50000, cap_b=50000)
    small = gs.sparsify_sample_hybrid(gd, 0.1, seed=3, solver="exact", cap_a=5, cap_b=40)
    torch.cuda.synchronize()
    assert int(small.flags.item()) & gs.FLAG_OVERFLOW
    assert int(small.n_a.item()) == int(full.n_a.item()) and int(small.n_b.item()) == int(full.n_b.item())
    assert torch.equal(small.idx_a[:5], full.idx_a[:5]) and torch.equal(small.code_b[:40], full.code_b[:40])
    z = torch.zeros(10000, device="cuda")
    o = gs.sparsify_sample_hybrid(z, 0.1, seed=1, solver="greedy", dense_q=True)
    torch.cuda.synchronize()
    assert int(o.n_a.item()) == 0 and int(o.n_b.item()) == 0 and int(o.flags.item()) & gs.FLAG_ALLZERO
    assert not o.q.any().item()
    h = W.normal(9999, 92)
    h[::3] = 0
    hd = torch.from_numpy(h).cuda()
    for solver in ("greedy", "exact"):
        allk = gs.sparsify_sample_hybrid(hd, 1.0, seed=1, solver=solver, cap_a=9999, cap_b=9999, dense_q=True)
        none = gs.sparsify_sample_hybrid(hd, 0.0, seed=1, solver=solver, cap_a=9999, cap_b=9999, dense_q=True)
        torch.cuda.synchronize()
        nz = np.flatnonzero(h)
        A = int(allk.n_a.item())
        assert A == nz.size and int(allk.n_b.item()) == 0
        assert np.array_equal(allk.idx_a[:A].cpu().numpy(), nz) and np.array_equal(allk.val_a[:A].cpu().numpy(), h[nz])
        assert np.array_equal(allk.q.cpu().numpy() != 0, h != 0) and float(allk.inv_lam.item()) == 0.0
        assert int(none.n_a.item()) == 0 and int(none.n_b.item()) == 0 and not none.q.any().item()
