"""GPU parity of per-layer sparsification (Section 5.2: each layer sparsified on its own) through the
C ABI: segment s of a flat gradient gets its own lambda, budget rho_s * length and Philox key, and
must match the oracle run on that segment alone under the parity rule (index sets equal except
where |u_i - p_i| <= 1e-6, values to rel 1e-5, lambda to rel 1e-9; the exact solver's lambda and
capped count bit for bit). Covers the ResNet-50 layer layout of the 25,557,032-coordinate gradient
(54 segments, 4,224 to 2,360,320 long), layers that are empty, shorter than one float4 group or
span many tiles, offsets that are not multiples of 4, the probabilities entry point, and device
offsets that disagree with the host's."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from oracle.compare import compare_probs, compare_sample

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


def _check(g, off, rhos, seeds, solver, out, exact_bits):
    ref = oracle.sparsify_segments(g, off, rhos, seeds, solver)
    idx, val = out.idx.cpu().numpy(), out.val.cpu().numpy()
    nnz, lam, k, fl = (out.nnz.cpu().numpy(), out.lam.cpu().numpy(), out.k.cpu().numpy(), out.flags.cpu().numpy())
    for s in range(len(off) - 1):
        seg = g[off[s]:off[s + 1]]
        n = int(nnz[s])
        if seg.size == 0 or not np.any(seg):
            assert n == 0 and fl[s] & 4, (s, n, fl[s])
            continue
        assert fl[s] == 0, (s, fl[s])
        sol = ref[s][0]
        compare_sample(seg, sol.p, seeds[s], idx[s, :n], val[s, :n], n, lam[s], sol.lam)
        if exact_bits:
            assert lam[s] == sol.lam and k[s] == sol.k, (s, lam[s], sol.lam)


@pytest.fixture(scope="module")
def c4():
    w = W.c4()
    return w.g[0], np.concatenate([[0], np.cumsum(w.meta["segments"])]).astype(np.int64)


@pytest.mark.parametrize("rho", [0.001, 0.01])
@pytest.mark.parametrize("solver", ["exact", "greedy"])
def test_resnet50_layers(gs, c4, solver, rho):
    g, off = c4
    segs = off.size - 1
    seeds = [4000 + s for s in range(segs)]
    _say("segmented resnet50 54 layers", solver, rho)
    seg = gs.Segments(off)
    out = gs.sparsify_sample_compact_segmented(torch.from_numpy(g).cuda(), seg, rho, seeds, solver)
    torch.cuda.synchronize()
    _check(g, off, [rho] * segs, seeds, solver, out, solver == "exact")


def _layered(lengths, seed):
    rng = np.random.default_rng(seed)
    parts = []
    for i, n in enumerate(lengths):
        mk = (W.t_mixture, W.normal, W.integer_ties, W.wide_range)[i % 4]
        parts.append(mk(n, seed + i) * np.float32(10.0 ** rng.uniform(-4, 0)) if n else np.zeros(0, np.float32))
    return np.concatenate(parts).astype(np.float32), np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)


LAYOUTS = {
    "aligned_mixed": [4096, 16388, 12, 200000, 0, 8, 65536 * 3, 44],
    "unaligned_tiny": [3000, 0, 3, 16384 + 8, 1, 70001, 4, 2],
    "many_small": [int(x) for x in np.random.default_rng(5).integers(0, 3000, 300)],
    "one_long_many_short": [1 << 21] + [40] * 200,
    # more tiles than are resident at once: two tiles per sample workgroup
    "two_tiles_per_workgroup": [1 << 22] * 7 + [16384 * 3 + 5, 4],
}


@pytest.mark.parametrize("layout", list(LAYOUTS))
@pytest.mark.parametrize("solver", ["greedy", "exact"])
def test_layouts(gs, layout, solver):
    lengths = LAYOUTS[layout]
    g, off = _layered(lengths, 900 + len(lengths))
    segs = len(lengths)
    rhos = [(0.01, 0.1, 0.5, 0.3, 1.0, 0.05, 0.2)[i % 7] for i in range(segs)]
    seeds = [123456789 * (i + 1) for i in range(segs)]
    _say("segmented layout", layout, solver, "segments", segs)
    out = gs.sparsify_sample_compact_segmented(torch.from_numpy(g).cuda(), gs.Segments(off), rhos, seeds, solver)
    torch.cuda.synchronize()
    _check(g, off, rhos, seeds, solver, out, solver == "exact")


def test_random_layouts(gs):
    """Twenty seeded random layer layouts: 1 to 40 segments with lengths from 0 to ~200 K
    (log-uniform, some empty, offsets of any alignment), a random density per segment and one
    solver per call; every segment against the oracle run on it alone."""
    rng = np.random.default_rng(515)
    for case in range(20):
        segs = int(rng.integers(1, 41))
        lengths = [0 if rng.random() < 0.08 else int(np.exp(rng.uniform(0.0, np.log(200000.0)))) for _ in range(segs)]
        g, off = _layered(lengths, 7000 + case)
        rhos = [float(10.0 ** rng.uniform(-3.0, 0.0)) for _ in range(segs)]
        seeds = [int(rng.integers(1 << 62)) for _ in range(segs)]
        solver = ("greedy", "exact")[int(rng.integers(2))]
        _say(f"[random-layout] case={case} segments={segs} total={int(off[-1])} solver={solver}")
        out = gs.sparsify_sample_compact_segmented(torch.from_numpy(g).cuda(), gs.Segments(off), rhos, seeds, solver)
        torch.cuda.synchronize()
        _check(g, off, rhos, seeds, solver, out, solver == "exact")


@pytest.mark.parametrize("layout", ["aligned_mixed", "unaligned_tiny", "two_tiles_per_workgroup"])
def test_hybrid_segmented(gs, layout):
    """Per-layer hybrid coding: the compaction's survivors split by the capped set, row by row,
    the dense ternary vector in g's layout; for the exact solver Q_A, Q_B and q equal the oracle's
    split of each segment."""
    lengths = LAYOUTS[layout]
    g, off = _layered(lengths, 1200 + len(lengths))
    segs = len(lengths)
    rhos = [(0.01, 0.1, 0.5, 0.3, 1.0, 0.05, 0.2)[i % 7] for i in range(segs)]
    seeds = [77 + 5 * i for i in range(segs)]
    gd = torch.from_numpy(g).cuda()
    seg = gs.Segments(off)
    for solver in ("greedy", "exact"):
        _say("hybrid segmented", layout, solver)
        c = gs.sparsify_sample_compact_segmented(gd, seg, rhos, seeds, solver)
        h = gs.sparsify_sample_hybrid_segmented(gd, seg, rhos, seeds, solver, dense_q=True)
        idx, val, nnz, k = c.idx.cpu().numpy(), c.val.cpu().numpy(), c.nnz.cpu().numpy(), c.k.cpu().numpy()
        ia, va, na = h.idx_a.cpu().numpy(), h.val_a.cpu().numpy(), h.n_a.cpu().numpy()
        cb, nb, inv, q = h.code_b.cpu().numpy(), h.n_b.cpu().numpy(), h.inv_lam.cpu().numpy(), h.q.cpu().numpy()
        assert torch.equal(c.flags.cpu(), h.flags.cpu()) and np.array_equal(c.lam.cpu().numpy(), h.lam.cpu().numpy(),
                                                                            equal_nan=True)
        for s in range(segs):
            n, A, B = int(nnz[s]), int(na[s]), int(nb[s])
            assert A + B == n and A == k[s]
            bi = cb[s, :B] & 0x7FFFFFFF
            merged = np.concatenate([ia[s, :A], bi])
            vals = np.concatenate([va[s, :A], np.where(cb[s, :B] < 0, -inv[s], inv[s]).astype(np.float32)])
            o = np.argsort(merged, kind="stable")
            assert np.array_equal(merged[o], idx[s, :n]) and np.array_equal(vals[o], val[s, :n])
            qs = q[off[s]:off[s + 1]]
            assert np.count_nonzero(qs) == n and np.all(qs[ia[s, :A]] == 2)
            seg_g = g[off[s]:off[s + 1]]
            if solver == "exact" and seg_g.size and np.any(seg_g):
                ref = oracle.sample_hybrid(seg_g, oracle.solve_exact(seg_g, rhos[s]).p, seeds[s])
                assert np.array_equal(ia[s, :A], ref.qa_idx) and np.array_equal(bi, ref.qb_idx)
                assert np.array_equal(qs, ref.q)


def test_segment_equals_single_row_call(gs):
    g, off = _layered(LAYOUTS["aligned_mixed"], 77)
    segs = off.size - 1
    rhos, seeds = [0.05] * segs, [31 + s for s in range(segs)]
    _say("segmented vs single-row calls")
    gd = torch.from_numpy(g).cuda()
    out = gs.sparsify_sample_compact_segmented(gd, gs.Segments(off), rhos, seeds, "greedy")
    for s in range(segs):
        if off[s + 1] == off[s]:
            continue
        one = gs.sparsify_sample_compact(gd[off[s]:off[s + 1]].contiguous(), rhos[s], seeds[s], "greedy")
        n = int(out.nnz[s].item())
        assert int(one.nnz[0].item()) == n
        assert torch.equal(one.idx[:n].cpu(), out.idx[s, :n].cpu())
        assert torch.equal(one.val[:n].cpu(), out.val[s, :n].cpu())
        assert one.lam[0].item() == out.lam[s].item()


@pytest.mark.parametrize("layout", ["aligned_mixed", "unaligned_tiny"])
def test_probs_segmented(gs, layout):
    g, off = _layered(LAYOUTS[layout], 300)
    segs = off.size - 1
    rhos = [0.02 + 0.03 * (s % 5) for s in range(segs)]
    _say("segmented probabilities", layout)
    pr = gs.sparsify_probs_segmented(torch.from_numpy(g).cuda(), gs.Segments(off), rhos, "exact")
    torch.cuda.synchronize()
    p = pr.p.cpu().numpy()
    for s in range(segs):
        seg = g[off[s]:off[s + 1]]
        if seg.size and np.any(seg):
            sol = oracle.solve_exact(seg, rhos[s])
            compare_probs(p[off[s]:off[s + 1]], sol.p)
            assert pr.lam[s].item() == sol.lam and int(pr.k[s].item()) == sol.k


def test_random_layouts_probs(gs):
    """Twenty seeded random layer layouts through the probabilities entry point (exact solver):
    every segment's p against the oracle to 1e-6, lambda and k bit for bit."""
    rng = np.random.default_rng(616)
    for case in range(20):
        segs = int(rng.integers(1, 41))
        lengths = [0 if rng.random() < 0.08 else int(np.exp(rng.uniform(0.0, np.log(200000.0)))) for _ in range(segs)]
        g, off = _layered(lengths, 8000 + case)
        rhos = [float(10.0 ** rng.uniform(-3.0, 0.0)) for _ in range(segs)]
        _say(f"[random-layout-probs] case={case} segments={segs} total={int(off[-1])}")
        pr = gs.sparsify_probs_segmented(torch.from_numpy(g).cuda(), gs.Segments(off), rhos, "exact")
        torch.cuda.synchronize()
        p = pr.p.cpu().numpy()
        for s_ in range(segs):
            seg = g[off[s_]:off[s_ + 1]]
            if seg.size and np.any(seg):
                sol = oracle.solve_exact(seg, rhos[s_])
                compare_probs(p[off[s_]:off[s_ + 1]], sol.p)
                assert pr.lam[s_].item() == sol.lam and int(pr.k[s_].item()) == sol.k, (case, s_)


def test_device_offsets_that_disagree_are_flagged(gs):
    """Device offsets that break the host's bounds (a start that is not a multiple of 4 on the
    vector path, an end past the host's last offset) change the launch shape: every segment is
    flagged and skipped, without reading outside the segments; the same workspace then serves a
    call with the right offsets."""
    g, off = _layered([4000, 8000, 4000], 650)
    seg = gs.Segments(off)
    good = seg.dev
    bad = off.copy()
    bad[1] = 4001
    bad[3] = off[3] + 400
    seg.dev = torch.from_numpy(bad).cuda()
    gd = torch.from_numpy(g).cuda()
    _say("segmented bad device offsets")
    out = gs.sparsify_sample_compact_segmented(gd, seg, 0.1, [1, 2, 3], "greedy")
    fl = out.flags.cpu().numpy()
    assert np.all(fl & gs.FLAG_BADSEG) and not out.nnz.cpu().numpy().any()
    assert np.isnan(out.lam.cpu().numpy()).all()
    pr = gs.sparsify_probs_segmented(gd, seg, 0.1, "exact")
    assert np.all(pr.flags.cpu().numpy() & gs.FLAG_BADSEG)
    seg.dev = good
    out = gs.sparsify_sample_compact_segmented(gd, seg, 0.1, [1, 2, 3], "greedy")
    assert not out.flags.cpu().numpy().any() and np.all(out.nnz.cpu().numpy() > 0)
