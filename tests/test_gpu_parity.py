"""GPU parity: the HIP path (through the C ABI) against the oracle, element by element, at sizes
the oracle finishes in seconds that still span many tiles and ragged tails, plus edge cases,
batching, determinism, capacity overflow, the unaligned (scalar-load) path and sampling
statistics. Rule: index sets equal except where |u_i - p_i| <= 1e-6, values to rel 1e-5, lambda
to rel 1e-9, probabilities to 1e-6 absolute."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from oracle.compare import compare_probs, compare_sample, lam_close

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


def _run_row(gs, g, rho, solver, seed, iters=2, cap=None):
    gd = torch.from_numpy(g).cuda()
    out = gs.sparsify_sample_compact(gd, rho, seed=seed, solver=solver, iters=iters, capacity=cap)
    torch.cuda.synchronize()
    n = int(out.nnz.item())
    m = min(n, out.idx.numel())
    return (out.idx[:m].cpu().numpy(), out.val[:m].cpu().numpy(), n, float(out.lam.item()),
            int(out.k.item()), int(out.flags.item()) & 0xFFFFFFFF)


VECTORS = {
    "normal_65536": lambda: W.normal(65536, 0),
    "normal_ragged_100003": lambda: W.normal(100003, 1),
    "tmix_200001": lambda: W.t_mixture(200001, 2),
    "ties_50001": lambda: W.integer_ties(50001, 3),
    "wide_range_120000": lambda: W.wide_range(120000, 4),
    "two_level_70001": lambda: W.two_level(70001, 300, 50.0, 1.0, 5),
    "approx_sparse_40000": lambda: W.approx_sparse(40000, 200, 0.05, 6),
    "tiny_7": lambda: W.normal(7, 7),
    "one_1": lambda: np.array([-2.5], np.float32),
    "laplace_row": lambda: W.c2(rows=1, d=1 << 18).g[0].copy(),
}


@pytest.mark.parametrize("name", list(VECTORS))
@pytest.mark.parametrize("solver", ["greedy", "exact"])
@pytest.mark.parametrize("rho", [0.001, 0.01, 0.1, 0.5])
def test_row_parity(gs, name, solver, rho):
    g = VECTORS[name]()
    seed = 1234 + len(name)
    _say(f"[parity] {name} d={g.size} solver={solver} rho={rho} seed={seed}")
    sol = oracle.solve(g, rho, solver, 2)
    idx, val, n, lam, k, fl = _run_row(gs, g, rho, solver, seed, cap=g.size)
    assert fl == 0, fl
    rep = compare_sample(g, sol.p, seed, idx, val, n, lam, sol.lam)
    assert k == sol.k or solver == "greedy", (k, sol.k)
    if solver == "greedy":
        # the capped count reported is that of the returned lambda
        assert k == int(np.count_nonzero(lam * np.abs(g.astype(np.float64)) >= 1.0)) or np.isinf(lam)
    _say(f"   ok nnz={n} oracle={rep['nnz_oracle']} excused={rep['excused']} lam={lam:.12g}")


def test_emission_paths(gs):
    """Rows whose waves emit through each of the sampling pass's paths: staged in LDS (up to 512
    survivors in a wave's 4096 coordinates), written directly lane by lane (up to 1024), written
    group by group (more), and a row that mixes them (a loud half and a quiet half, with a tile and
    a wave's quarter across the boundary)."""
    loud = W.normal(100000, 41)
    quiet = W.normal(100003, 42) * np.float32(0.01)
    cases = [("staged", W.t_mixture(200003, 40), 0.1), ("direct", W.normal(200003, 43), 0.2),
             ("groups", W.normal(200003, 44), 0.4), ("mixed", np.concatenate([loud, quiet]), 0.1)]
    for label, g, rho in cases:
        for solver in ("exact", "greedy"):
            seed = 77
            _say(f"[emission] {label} d={g.size} solver={solver} rho={rho} seed={seed}")
            sol = oracle.solve(g, rho, solver, 2)
            idx, val, n, lam, k, fl = _run_row(gs, g, rho, solver, seed, cap=g.size)
            assert fl == 0, fl
            rep = compare_sample(g, sol.p, seed, idx, val, n, lam, sol.lam)
            _say(f"   ok nnz={n} oracle={rep['nnz_oracle']} excused={rep['excused']}")


def _random_case(rng):
    """A seeded draw of a row: length (1 to ~300 K, log-uniform, often ragged), distribution,
    scale, density and solver."""
    d = int(np.exp(rng.uniform(0.0, np.log(300000.0))))
    g, seed = _random_vector(rng, d)
    rho = float(10.0 ** rng.uniform(-3.5, 0.0))
    solver = ("greedy", "exact")[int(rng.integers(2))]
    return g, rho, solver, seed % 100000


def _random_vector(rng, d):
    """A seeded vector of length d: one of six distributions, scaled over ten decades; and the seed
    it was drawn with."""
    seed = int(rng.integers(1 << 30))
    kind = int(rng.integers(6))
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
    else:
        g = W.approx_sparse(d, max(1, d // 20), 0.05, seed) if d >= 20 else W.normal(d, seed)
    return (g * np.float32(10.0 ** rng.uniform(-6, 4))).astype(np.float32), seed


def test_random_rows(gs):
    """Two hundred seeded random rows (length, distribution, scale over ten decades, density,
    solver) against the oracle under the parity rule, lambda bit for bit for the exact solver."""
    rng = np.random.default_rng(2024)
    for case in range(200):
        g, rho, solver, seed = _random_case(rng)
        _say(f"[random] case={case} d={g.size} rho={rho:.5g} solver={solver} seed={seed}")
        sol = oracle.solve(g, rho, solver, 2)
        idx, val, n, lam, k, fl = _run_row(gs, g, rho, solver, seed, cap=g.size)
        assert fl == (0 if g.any() else gs.FLAG_ALLZERO), (case, fl)  # an all-zero row is reported
        compare_sample(g, sol.p, seed, idx, val, n, lam, sol.lam)
        if solver == "exact":
            assert lam == sol.lam and k == sol.k, (case, lam, sol.lam, k, sol.k)


def test_random_long_rows(gs):
    """Eight seeded rows of 2^22 to 2^26 coordinates (log-uniform, ragged; from 2^25 on the
    statistics pass collects a candidate band) with random distribution, scale and density, both
    solvers, against the oracle; lambda and k bit for bit for the exact solver."""
    rng = np.random.default_rng(9090)
    for case in range(8):
        d = int(2.0 ** rng.uniform(22.0, 26.0))
        g, seed = _random_vector(rng, d)
        rho = float(10.0 ** rng.uniform(-3.5, -0.5))
        solver = ("greedy", "exact")[case % 2]
        _say(f"[random-long] case={case} d={d} rho={rho:.5g} solver={solver} seed={seed}")
        sol = oracle.solve(g, rho, solver, 2)
        idx, val, n, lam, k, fl = _run_row(gs, g, rho, solver, seed % 100000)
        assert fl == 0, (case, fl)
        compare_sample(g, sol.p, seed % 100000, idx, val, n, lam, sol.lam)
        if solver == "exact":
            assert lam == sol.lam and k == sol.k, (case, lam, sol.lam, k, sol.k)


def test_full_range_rows(gs):
    """Forty seeded rows whose magnitudes span all of fp32's binades (subnormals to near the
    largest finite value), random length, density and solver, against the oracle; then a row of
    magnitudes in [2^120, 2^127.9) at rho = 0.01, whose 1/lambda lies beyond fp32's range, so the
    amplified values are +-inf on both sides and the hybrid coding's shared 1/lambda is +inf."""
    rng = np.random.default_rng(77)
    for case in range(40):
        d = int(np.exp(rng.uniform(0.0, np.log(300000.0))))
        g = W.full_range(d, 500 + case)
        rho = float(10.0 ** rng.uniform(-3.5, 0.0))
        solver = ("greedy", "exact")[case % 2]
        _say(f"[full-range] case={case} d={d} rho={rho:.5g} solver={solver}")
        sol = oracle.solve(g, rho, solver, 2)
        idx, val, n, lam, k, fl = _run_row(gs, g, rho, solver, case, cap=d)
        assert fl == 0, (case, fl)
        compare_sample(g, sol.p, case, idx, val, n, lam, sol.lam)
        if solver == "exact":
            assert lam == sol.lam and k == sol.k, (case, lam, sol.lam, k, sol.k)
    r2 = np.random.default_rng(9)
    d = 100003
    g = (r2.choice([-1.0, 1.0], d) * np.exp2(r2.uniform(120.0, 127.9, d))).astype(np.float32)
    for solver in ("exact", "greedy"):
        _say(f"[full-range] overflow row solver={solver}")
        sol = oracle.solve(g, 0.01, solver, 2)
        assert sol.lam < 2.0 ** -128
        idx, val, n, lam, k, fl = _run_row(gs, g, 0.01, solver, 5, cap=d)
        assert fl == 0 and np.isinf(val[:n]).any()
        compare_sample(g, sol.p, 5, idx, val, n, lam, sol.lam)
        h = gs.sparsify_sample_hybrid(torch.from_numpy(g).cuda(), 0.01, seed=5, solver=solver, cap_a=d, cap_b=d)
        torch.cuda.synchronize()
        assert int(h.flags.item()) == 0 and float(h.inv_lam.item()) == float("inf")
        assert int(h.n_a.item()) + int(h.n_b.item()) == n


@pytest.mark.parametrize("iters", [0, 1, 3, 8])
def test_greedy_iterations(gs, iters):
    g = W.t_mixture(150000, 11)
    _say(f"[greedy-iters] T={iters}")
    for rho in (0.01, 0.1, 0.3):
        sol = oracle.solve_greedy(g, rho, iters)
        idx, val, n, lam, k, fl = _run_row(gs, g, rho, "greedy", 5, iters=iters, cap=g.size)
        compare_sample(g, sol.p, 5, idx, val, n, lam, sol.lam)


def test_exact_is_bit_identical_lambda(gs):
    """Exact sums on both sides: the exact solver's lambda must match the oracle's to the bit."""
    for maker, rho in [(lambda: W.t_mixture(300000, 21), 0.05), (lambda: W.normal(100000, 22), 0.2),
                       (lambda: W.integer_ties(80000, 23), 0.3), (lambda: W.wide_range(90000, 24), 0.02)]:
        g = maker()
        sol = oracle.solve_exact(g, rho)
        _, _, _, lam, k, fl = _run_row(gs, g, rho, "exact", 1, cap=1)
        _say(f"[bit-lambda] d={g.size} rho={rho} gpu={lam!r} oracle={sol.lam!r} k={k}/{sol.k}")
        assert lam == sol.lam and k == sol.k


@pytest.mark.parametrize("solver", ["greedy", "exact"])
def test_probs_parity(gs, solver):
    for maker, rho in [(lambda: W.t_mixture(100001, 31), 0.1), (lambda: W.normal(65536, 32), 0.01),
                       (lambda: W.integer_ties(30000, 33), 0.4)]:
        g = maker()
        _say(f"[probs] {solver} d={g.size} rho={rho}")
        sol = oracle.solve(g, rho, solver, 2)
        out = gs.sparsify_probs(torch.from_numpy(g).cuda(), rho, solver=solver, iters=2)
        torch.cuda.synchronize()
        compare_probs(out.p.cpu().numpy(), sol.p)
        assert lam_close(float(out.lam.item()), sol.lam)
        assert int(out.k.item()) == int(np.count_nonzero(out.p.cpu().numpy() == 1.0))
        assert int(out.flags.item()) == 0


def _tied_boundary(d, n_hi, seed):
    """+-1 entries with n_hi entries of +-2 and n_hi zeros at seeded positions: at rho = 0.5 the
    total is 2 B, so Algorithm 2's criterion holds at k = 0 with equality, lambda = 0.5 and the
    tied run of 2s has p_i = 1 (the capped set)."""
    rng = np.random.default_rng(seed)
    g = np.where(rng.random(d) < 0.5, -1.0, 1.0).astype(np.float32)
    pos = rng.permutation(d)
    g[pos[:n_hi]] *= 2
    g[pos[n_hi:2 * n_hi]] = 0
    return g


def test_capped_values_past_the_lane_rows(gs):
    """A row whose 76 capped coordinates sit in two strided patterns that one lane of the sampling
    pass's decide phase takes (64 and 12 coordinates, against LDS rows of 8): those waves read their
    capped values from g while emitting, at densities whose waves emit lane by lane (rho 0.002 and
    0.01) or group by group (rho 0.5), in the compaction and in the hybrid coding. Every capped
    coordinate survives with value g_i, and the rest follows the oracle under the parity rule."""
    g = W.strided_large(65536 + 123, 7)
    d = g.size
    big = np.flatnonzero(np.abs(g) >= 100.0)
    gd = torch.from_numpy(g).cuda()
    for rho in (0.002, 0.01, 0.5):
        for solver in ("exact", "greedy"):
            _say(f"[lane-rows] d={d} solver={solver} rho={rho}")
            sol = oracle.solve(g, rho, solver, 2)
            assert np.all(sol.p[big] == 1.0)
            idx, val, n, lam, k, fl = _run_row(gs, g, rho, solver, 17, cap=d)
            assert fl == 0, fl
            compare_sample(g, sol.p, 17, idx, val, n, lam, sol.lam)
            assert np.all(np.isin(big, idx)) and np.array_equal(val[np.isin(idx, big)], g[big])
            h = gs.sparsify_sample_hybrid(gd, rho, seed=17, solver=solver, cap_a=d, cap_b=d)
            torch.cuda.synchronize()
            A, B = int(h.n_a.item()), int(h.n_b.item())
            assert int(h.flags.item()) == 0 and A + B == n
            ia = h.idx_a[:A].cpu().numpy()
            bi = h.code_b[:B].cpu().numpy() & 0x7FFFFFFF
            assert np.all(np.isin(big, ia)) and np.array_equal(h.val_a[:A].cpu().numpy(), g[ia])
            assert np.all(np.diff(ia) > 0) and np.all(np.diff(bi) > 0)
            assert np.array_equal(np.sort(np.concatenate([ia, bi])), idx)


@pytest.mark.parametrize("d,n_hi", [(40000, 3000), (1000003, 77777), ((1 << 25) + 5, 1 << 20)])
def test_capped_ties_one_rule(gs, d, n_hi):
    """Every pass takes the same capped set {p_i = 1}: compaction (whole tiles and the partial last
    tile; one and two tiles per workgroup), probabilities and the hybrid coding. Closed form:
    lambda = 0.5, k = n_hi, every 2 kept with value g_i."""
    g = _tied_boundary(d, n_hi, 17)
    hi = np.flatnonzero(np.abs(g) == 2)
    gd = torch.from_numpy(g).cuda()
    _say(f"[ties] d={d} n_hi={n_hi}")
    out = gs.sparsify_sample_compact(gd, 0.5, seed=3, solver="exact", capacity=d)
    h = gs.sparsify_sample_hybrid(gd, 0.5, seed=3, solver="exact", cap_a=d, cap_b=d, dense_q=True)
    pr = gs.sparsify_probs(gd, 0.5, solver="exact")
    torch.cuda.synchronize()
    n = int(out.nnz.item())
    idx, val = out.idx[:n].cpu().numpy(), out.val[:n].cpu().numpy()
    assert float(out.lam.item()) == 0.5 and int(out.k.item()) == n_hi and int(out.flags.item()) == 0
    assert np.all(np.isin(hi, idx)) and np.array_equal(val[np.isin(idx, hi)], g[hi])
    A, B = int(h.n_a.item()), int(h.n_b.item())
    assert A == n_hi and A + B == n and int(h.flags.item()) == 0
    ia = h.idx_a[:A].cpu().numpy()
    bi = h.code_b[:B].cpu().numpy() & 0x7FFFFFFF
    assert np.array_equal(ia, hi) and np.all(np.diff(bi) > 0)
    assert np.array_equal(np.sort(np.concatenate([ia, bi])), idx)
    q = h.q.cpu().numpy()
    assert np.array_equal(np.flatnonzero(q == 2), hi)
    p = pr.p.cpu().numpy()
    assert int(pr.k.item()) == n_hi and float(pr.lam.item()) == 0.5
    assert np.all(p[hi] == 1.0) and np.count_nonzero(p == 1.0) == n_hi
    if d <= 1000003:  # the oracle's sample under the parity rule
        sol = oracle.solve_exact(g, 0.5)
        assert sol.lam == 0.5 and sol.k == n_hi
        compare_sample(g, sol.p, 3, idx, val, n, 0.5, sol.lam)
        compare_probs(p, sol.p)
    _say(f"   ok nnz={n}")


def _row_state(ws, row=0):
    """src / band / collected count of a row's control block in a workspace (offsets fixed by
    static asserts in the library source)."""
    b = ws.cpu().numpy()[256 + 256 * row: 256 + 256 * (row + 1)]
    u32 = lambda o: int(b[o:o + 4].view(np.uint32)[0])
    return {"src": u32(192), "band_lo": u32(220), "band_hi": u32(224), "cand_n": int(b[232:240].view(np.uint64)[0])}


@pytest.mark.parametrize("solver", ["greedy", "exact"])
def test_candidate_band_on_a_long_row(gs, solver):
    """A row of 2^25 + 12 coordinates (long enough for a candidate band): the statistics pass
    collects exactly the keys of the predicted binades, the refinement windows read them, and the
    result equals the oracle's under the parity rule (lambda bit for bit for the exact solver)."""
    d = (1 << 25) + 12
    g = W.t_mixture(d, 71)
    keys = np.abs(g).view(np.uint32)
    gd = torch.from_numpy(g).cuda().reshape(1, -1)
    seeds = torch.tensor([5], dtype=torch.int64, device="cuda")
    used = 0
    for rho in (0.001, 0.01, 0.1):
        plan = gs.Plan(1, d, solver=solver, cap_per_row=gs.capacity_hint(d, rho))
        plan.run(gd, torch.tensor([rho], dtype=torch.float64, device="cuda"), seeds)
        torch.cuda.synchronize()
        st = _row_state(plan.ws)
        n = int(plan.nnz[0].item())
        _say(f"[band] {solver} rho={rho} band=[{st['band_lo'] >> 23},{st['band_hi'] >> 23}) cand={st['cand_n']} "
             f"src={st['src']} nnz={n}")
        assert int(plan.flags[0].item()) == 0
        assert st["band_hi"] > st["band_lo"]  # this row has capped coordinates at every density
        assert st["cand_n"] == int(np.count_nonzero((keys >= st["band_lo"]) & (keys < st["band_hi"])))
        used += st["src"]
        sol = oracle.solve(g, rho, solver, 2)
        compare_sample(g, sol.p, 5, plan.idx[0, :n].cpu().numpy(), plan.val[0, :n].cpu().numpy(), n,
                       float(plan.lam[0].item()), sol.lam)
        if solver == "exact":
            assert float(plan.lam[0].item()) == sol.lam and int(plan.k[0].item()) == sol.k
    assert used > 0


def test_candidate_band_on_ragged_rows(gs):
    """Two rows of 2^25 + 3 coordinates stored with a leading dimension of 2^25 + 4 (vector loads;
    each row ends in a partial group of 3): the band is collected over the whole row, its last
    partial group included, and both rows match the oracle (exact solver, lambda bit for bit)."""
    rows, d, ld = 2, (1 << 25) + 3, (1 << 25) + 4
    g = np.stack([W.t_mixture(d, 81 + r) for r in range(rows)])
    # the partial group holds a key of each density's band and the row's largest magnitude
    g[:, -3:] = np.float32([12.0, -3000.0, 1.0e4])
    buf = np.zeros((rows, ld), np.float32)
    buf[:, :d] = g
    gd = torch.from_numpy(buf).cuda()
    seeds = torch.tensor([11, 12], dtype=torch.int64, device="cuda")
    for rho in (0.001, 0.1):
        plan = gs.Plan(rows, d, ld=ld, solver="exact", cap_per_row=gs.capacity_hint(d, rho))
        plan.run(gd, torch.full((rows,), rho, dtype=torch.float64, device="cuda"), seeds)
        torch.cuda.synchronize()
        for r in range(rows):
            st = _row_state(plan.ws, r)
            keys = np.abs(g[r]).view(np.uint32)
            n = int(plan.nnz[r].item())
            _say(f"[band-ragged] row {r} rho={rho} band=[{st['band_lo'] >> 23},{st['band_hi'] >> 23}) "
                 f"cand={st['cand_n']} src={st['src']} nnz={n}")
            assert int(plan.flags[r].item()) == 0
            assert st["band_hi"] > st["band_lo"]
            assert st["cand_n"] == int(np.count_nonzero((keys >= st["band_lo"]) & (keys < st["band_hi"])))
            sol = oracle.solve(g[r], rho, "exact", 2)
            compare_sample(g[r], sol.p, 11 + r, plan.idx[r, :n].cpu().numpy(), plan.val[r, :n].cpu().numpy(), n,
                           float(plan.lam[r].item()), sol.lam)
            assert float(plan.lam[r].item()) == sol.lam and int(plan.k[r].item()) == sol.k


@pytest.mark.parametrize("solver", ["greedy", "exact"])
def test_candidate_band_region_overflow(gs, solver):
    """A row of 2^25 coordinates whose first statistics workgroup's chunk (65,536 coordinates) lies
    wholly in the predicted band (magnitudes uniform in [8, 16), the rest of the row 1e-3 N(0, 1),
    rho putting 1/lambda near 12): that workgroup has more band keys than its staging region holds,
    so the band is dropped and the solver refines over the row; the result still equals the
    oracle's (lambda bit for bit for the exact solver)."""
    d = 1 << 25
    rng = np.random.default_rng(91)
    g = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    big = rng.uniform(8.0, 16.0, 1 << 16) * np.where(rng.random(1 << 16) < 0.5, -1.0, 1.0)
    g[: 1 << 16] = big.astype(np.float32)
    rho = 0.00186
    gd = torch.from_numpy(g).cuda().reshape(1, -1)
    seeds = torch.tensor([13], dtype=torch.int64, device="cuda")
    plan = gs.Plan(1, d, solver=solver, cap_per_row=gs.capacity_hint(d, rho))
    plan.run(gd, torch.tensor([rho], dtype=torch.float64, device="cuda"), seeds)
    torch.cuda.synchronize()
    st = _row_state(plan.ws)
    n = int(plan.nnz[0].item())
    _say(f"[band-region] {solver} band=[{st['band_lo'] >> 23},{st['band_hi'] >> 23}) cand={st['cand_n']} "
         f"src={st['src']} nnz={n} k={int(plan.k[0].item())}")
    assert int(plan.flags[0].item()) == 0
    # collected (the count exceeds the list's capacity, d / 16 keys: the overflowing region
    # reserved past it), then dropped by the first solve, and no window read the candidates
    assert st["cand_n"] > d // 16 and st["band_lo"] == st["band_hi"] == 0 and st["src"] == 0
    sol = oracle.solve(g, rho, solver, 2)
    assert sol.k > 0
    compare_sample(g, sol.p, 13, plan.idx[0, :n].cpu().numpy(), plan.val[0, :n].cpu().numpy(), n,
                   float(plan.lam[0].item()), sol.lam)
    if solver == "exact":
        assert float(plan.lam[0].item()) == sol.lam and int(plan.k[0].item()) == sol.k


def test_candidate_band_with_smaller_workspaces(gs):
    """The same long row with the full workspace (band used), a workspace with room for 2^16
    candidates only (the band overflows and is dropped) and the fixed part alone (no band): the
    three calls return identical results, equal to the oracle's."""
    d = (1 << 25) + 12
    g = W.t_mixture(d, 73)
    gd = torch.from_numpy(g).cuda().reshape(1, -1)
    seeds = torch.tensor([9], dtype=torch.int64, device="cuda")
    rho = 0.1
    fixed = gs.workspace_bytes(1, d, "variance")  # the layout without candidate buffers
    full = gs.workspace_bytes(1, d, "exact")
    outs = []
    for name, size in (("full", full), ("2^16 candidates", fixed + 8 * (1 << 16) + 4096), ("fixed part", fixed)):
        plan = gs.Plan(1, d, solver="exact", cap_per_row=gs.capacity_hint(d, rho))
        assert size <= plan.ws.numel()
        plan.ws = plan.ws[:size]
        plan.run(gd, torch.tensor([rho], dtype=torch.float64, device="cuda"), seeds)
        torch.cuda.synchronize()
        st = _row_state(plan.ws)
        n = int(plan.nnz[0].item())
        _say(f"[band-ws] {name}: {size} bytes band=[{st['band_lo'] >> 23},{st['band_hi'] >> 23}) cand={st['cand_n']} "
             f"src={st['src']} nnz={n}")
        assert int(plan.flags[0].item()) == 0
        outs.append((plan.idx[0, :n].cpu().numpy(), plan.val[0, :n].cpu().numpy(), float(plan.lam[0].item()),
                     int(plan.k[0].item()), st["src"]))
    assert outs[0][4] == 1 and outs[1][4] == 0 and outs[2][4] == 0
    for o in outs[1:]:
        assert np.array_equal(o[0], outs[0][0]) and np.array_equal(o[1], outs[0][1]) and o[2:4] == outs[0][2:4]
    sol = oracle.solve(g, rho, "exact", 2)
    idx, val, lam, k, _ = outs[0]
    compare_sample(g, sol.p, 9, idx, val, idx.size, lam, sol.lam)
    assert lam == sol.lam and k == sol.k


def test_special_cases(gs):
    d = 50000
    z = np.zeros(d, np.float32)
    _say("[special] all-zero")
    idx, val, n, lam, k, fl = _run_row(gs, z, 0.1, "exact", 0, cap=10)
    assert n == 0 and fl & gs.FLAG_ALLZERO
    g = W.normal(d, 41)
    g[::3] = 0
    for solver in ("greedy", "exact"):
        _say(f"[special] rho=0 and rho=1 {solver}")
        idx, val, n, lam, k, fl = _run_row(gs, g, 0.0, solver, 0, cap=10)
        assert n == 0 and lam == 0.0 and fl == 0
        idx, val, n, lam, k, fl = _run_row(gs, g, 1.0, solver, 0, cap=d)
        nzi = np.flatnonzero(g)
        assert n == nzi.size and np.array_equal(idx, nzi) and np.array_equal(val, g[nzi])
        assert np.isinf(lam) and k == nzi.size
        idx, val, n, lam, k, fl = _run_row(gs, g, 0.7, solver, 0, cap=d)  # B >= nnz
        assert n == nzi.size and np.array_equal(val, g[nzi])
    for bad in (np.inf, -np.inf, np.nan):
        h = W.normal(d, 42)
        h[12345] = bad
        _say(f"[special] non-finite {bad}")
        idx, val, n, lam, k, fl = _run_row(gs, h, 0.1, "greedy", 0, cap=100)
        assert n == 0 and fl & gs.FLAG_NONFINITE and np.isnan(lam)


def test_capacity_overflow(gs):
    g = W.t_mixture(200000, 51)
    sol = oracle.solve_exact(g, 0.1)
    cap = 777
    _say("[overflow]")
    idx, val, n, lam, k, fl = _run_row(gs, g, 0.1, "exact", 9, cap=cap)
    assert fl & gs.FLAG_OVERFLOW and n > cap and idx.size == cap
    compare_sample(g, sol.p, 9, idx, val, n, lam, sol.lam, cap=cap)


def test_capacity_boundaries(gs):
    """Output capacities at and around the survivor count n: exactly n (no overflow, the same
    output as with room to spare), n - 1 and a cut inside a wave's run of survivors (overflow
    flagged, n still reported, the first cap entries identical)."""
    g = W.t_mixture(300007, 52)
    gd = torch.from_numpy(g).cuda()
    for rho, solver in ((0.1, "exact"), (0.01, "greedy")):
        ref = gs.sparsify_sample_compact(gd, rho, seed=19, solver=solver, capacity=g.size)
        torch.cuda.synchronize()
        n = int(ref.nnz.item())
        for cap in (n, n - 1, n // 2 + 37):
            _say(f"[capacity] {solver} rho={rho} n={n} cap={cap}")
            out = gs.sparsify_sample_compact(gd, rho, seed=19, solver=solver, capacity=cap)
            torch.cuda.synchronize()
            fl = int(out.flags.item())
            assert int(out.nnz.item()) == n and float(out.lam.item()) == float(ref.lam.item())
            assert bool(fl & gs.FLAG_OVERFLOW) == (cap < n)
            assert torch.equal(out.idx[:cap], ref.idx[:cap]) and torch.equal(out.val[:cap], ref.val[:cap])


def test_unaligned_scalar_path(gs):
    g = W.t_mixture(100001, 61)
    big = torch.from_numpy(np.concatenate([np.zeros(1, np.float32), g])).cuda()
    view = big[1:]
    assert view.data_ptr() % 16 != 0
    _say("[unaligned]")
    for solver in ("greedy", "exact"):
        a = gs.sparsify_sample_compact(view, 0.05, seed=3, solver=solver, capacity=g.size)
        b = gs.sparsify_sample_compact(torch.from_numpy(g).cuda(), 0.05, seed=3, solver=solver, capacity=g.size)
        torch.cuda.synchronize()
        na, nb = int(a.nnz.item()), int(b.nnz.item())
        assert na == nb and float(a.lam.item()) == float(b.lam.item())
        assert torch.equal(a.idx[:na], b.idx[:nb]) and torch.equal(a.val[:na], b.val[:nb])


def test_batched_equals_rows_and_oracle(gs):
    rows, d = 12, 50003
    rng = np.random.default_rng(71)
    g = np.stack([W.t_mixture(d, 100 + r) * np.float32(10.0 ** rng.uniform(-3, 0)) for r in range(rows)])
    rhos = [0.01, 0.1, 0.3, 0.001] * 3
    seeds = [1000 + r for r in range(rows)] + []
    seeds[5] = 0xFFFFFFFFFFFFFFF1  # a seed using the high key word
    ld = d + 13  # padded rows: leading dimension > d
    buf = np.zeros((rows, ld), np.float32)
    buf[:, :d] = g
    gd = torch.from_numpy(buf).cuda()[:, :d]
    for solver in ("greedy", "exact"):
        _say(f"[batched] {solver} rows={rows} d={d} ld={ld}")
        out = gs.sparsify_sample_compact_batched(gd, rhos, seeds, solver=solver, iters=2, cap_per_row=d)
        torch.cuda.synchronize()
        for r in range(rows):
            n = int(out.nnz[r].item())
            sol = oracle.solve(g[r], rhos[r], solver, 2)
            compare_sample(g[r], sol.p, seeds[r], out.idx[r, :n].cpu().numpy(), out.val[r, :n].cpu().numpy(), n,
                           float(out.lam[r].item()), sol.lam)
            one = gs.sparsify_sample_compact(torch.from_numpy(g[r].copy()).cuda(), rhos[r], seed=seeds[r],
                                             solver=solver, capacity=d)
            torch.cuda.synchronize()
            assert int(one.nnz.item()) == n
            assert torch.equal(one.idx[:n], out.idx[r, :n]) and torch.equal(one.val[:n], out.val[r, :n])
            assert float(one.lam.item()) == float(out.lam[r].item())


@pytest.mark.parametrize("d,rho", [(500, 0.96), (5003, 0.97), ((1 << 25) + 7, 0.97)])
def test_answer_inside_the_lowest_binade(gs, d, rho):
    """Exact solver, 1/lambda inside the row's lowest occupied binade: no binade's maximum passes
    Algorithm 2's criterion, so the solver refines that binade (and its lowest sub-bin) instead of
    giving up; lambda and k equal the oracle's bit for bit, and the probabilities entry point and
    the hybrid coding agree."""
    g = W.lowest_binade(d, 3)
    _say(f"[lowest-binade] d={d} rho={rho}")
    sol = oracle.solve_exact(g, rho)
    assert 1.0e-3 <= 1.0 / sol.lam < 1.9e-3
    idx, val, n, lam, k, fl = _run_row(gs, g, rho, "exact", 29, cap=d)
    assert fl == 0, fl
    assert lam == sol.lam and k == sol.k, (lam, sol.lam, k, sol.k)
    compare_sample(g, sol.p, 29, idx, val, n, lam, sol.lam)
    gd = torch.from_numpy(g).cuda()
    pr = gs.sparsify_probs(gd, rho, solver="exact")
    torch.cuda.synchronize()
    assert int(pr.flags.item()) == 0 and float(pr.lam.item()) == sol.lam and int(pr.k.item()) == sol.k
    if d <= 1 << 20:
        compare_probs(pr.p.cpu().numpy(), sol.p)


def test_random_rows_hybrid_and_probs(gs):
    """Sixty seeded random rows through the hybrid coding and the probabilities entry point: Q_A
    holds the capped survivors with their values, Q_B the others in ascending order, together the
    compaction's indices; p equals the oracle's to 1e-6 with the same lambda and capped count."""
    rng = np.random.default_rng(7070)
    for case in range(60):
        g, rho, solver, seed = _random_case(rng)
        if not g.any():
            continue
        d = g.size
        _say(f"[random-hyb] case={case} d={d} rho={rho:.5g} solver={solver} seed={seed}")
        gd = torch.from_numpy(g).cuda()
        out = gs.sparsify_sample_compact(gd, rho, seed=seed, solver=solver, capacity=d)
        h = gs.sparsify_sample_hybrid(gd, rho, seed=seed, solver=solver, cap_a=d, cap_b=d)
        pr = gs.sparsify_probs(gd, rho, solver=solver)
        torch.cuda.synchronize()
        n = int(out.nnz.item())
        idx = out.idx[:n].cpu().numpy()
        A, B = int(h.n_a.item()), int(h.n_b.item())
        assert int(h.flags.item()) == 0 and A + B == n and A == int(out.k.item())  # every capped one survives
        ia = h.idx_a[:A].cpu().numpy()
        bi = h.code_b[:B].cpu().numpy() & 0x7FFFFFFF
        assert np.array_equal(h.val_a[:A].cpu().numpy(), g[ia])
        assert np.all(np.diff(ia) > 0) and np.all(np.diff(bi) > 0)
        assert np.array_equal(np.sort(np.concatenate([ia, bi])), idx)
        sol = oracle.solve(g, rho, solver, 2)
        compare_probs(pr.p.cpu().numpy(), sol.p)
        if solver == "exact":
            assert float(pr.lam.item()) == sol.lam and int(pr.k.item()) == sol.k


def test_random_batches(gs):
    """Thirty seeded random batches: 1 to 24 rows of one random length (1 to ~100 K), stored with a
    random padding of the leading dimension (so both the vector and the scalar load paths occur),
    a random density per row and one solver per batch; every row against the oracle under the
    parity rule (lambda bit for bit for the exact solver)."""
    rng = np.random.default_rng(4048)
    for case in range(30):
        rows = int(rng.integers(1, 25))
        d = int(np.exp(rng.uniform(0.0, np.log(100000.0))))
        ld = d + int(rng.integers(0, 9))
        solver = ("greedy", "exact")[int(rng.integers(2))]
        g = np.stack([W.t_mixture(d, 5000 + 31 * case + r) * np.float32(10.0 ** rng.uniform(-4, 2))
                      for r in range(rows)]).astype(np.float32)
        rhos = [float(10.0 ** rng.uniform(-3.0, 0.0)) for _ in range(rows)]
        seeds = [int(rng.integers(1 << 62)) for _ in range(rows)]
        buf = np.zeros((rows, ld), np.float32)
        buf[:, :d] = g
        gd = torch.from_numpy(buf).cuda()[:, :d]
        _say(f"[random-batch] case={case} rows={rows} d={d} ld={ld} solver={solver}")
        out = gs.sparsify_sample_compact_batched(gd, rhos, seeds, solver=solver, iters=2, cap_per_row=d)
        torch.cuda.synchronize()
        assert not out.flags.cpu().numpy().any(), out.flags
        for r in range(rows):
            n = int(out.nnz[r].item())
            sol = oracle.solve(g[r], rhos[r], solver, 2)
            compare_sample(g[r], sol.p, seeds[r], out.idx[r, :n].cpu().numpy(), out.val[r, :n].cpu().numpy(), n,
                           float(out.lam[r].item()), sol.lam)
            if solver == "exact":
                assert float(out.lam[r].item()) == sol.lam and int(out.k[r].item()) == sol.k


def test_deterministic_reruns(gs):
    g = torch.from_numpy(W.t_mixture(500000, 81)).cuda()
    _say("[determinism]")
    ref = gs.sparsify_sample_compact(g, 0.05, seed=4, solver="exact", capacity=500000)
    torch.cuda.synchronize()
    n = int(ref.nnz.item())
    for _ in range(5):
        o = gs.sparsify_sample_compact(g, 0.05, seed=4, solver="exact", capacity=500000)
        torch.cuda.synchronize()
        assert int(o.nnz.item()) == n and torch.equal(o.idx[:n], ref.idx[:n]) and torch.equal(o.val[:n], ref.val[:n])


def test_bad_rho_row_flagged(gs):
    g = torch.from_numpy(np.stack([W.normal(10000, 91), W.normal(10000, 92)])).cuda()
    _say("[bad-rho]")
    out = gs.sparsify_sample_compact_batched(g, [0.1, 1.5], [1, 2], cap_per_row=10000)
    torch.cuda.synchronize()
    assert int(out.flags[1].item()) & gs.FLAG_BADRHO and int(out.nnz[1].item()) == 0
    assert int(out.flags[0].item()) == 0 and int(out.nnz[0].item()) > 0


def test_unbiased_over_seeds(gs):
    """E[Q(g)_i] = g_i: one batched call with the same row under S different seeds."""
    d, S = 256, 8192
    rng = np.random.default_rng(7)
    g = (rng.standard_t(2, d) * 2).astype(np.float32)
    g[:8] = 0
    sol = oracle.solve_exact(g, 0.2)
    p = sol.p
    gd = torch.from_numpy(np.tile(g, (S, 1))).cuda()
    _say("[unbiased]")
    out = gs.sparsify_sample_compact_batched(gd, [0.2] * S, list(range(50_000, 50_000 + S)), solver="exact",
                                             cap_per_row=d)
    torch.cuda.synchronize()
    nnz = out.nnz.cpu().numpy()
    idx = out.idx.cpu().numpy()
    val = out.val.cpu().numpy().astype(np.float64)
    counts = np.zeros(d)
    qsum = np.zeros(d)
    for s in range(S):
        n = nnz[s]
        counts[idx[s, :n]] += 1
        qsum[idx[s, :n]] += val[s, :n]
    live = (p > 0) & (p < 1)
    z = (counts[live] - S * p[live]) / np.sqrt(S * p[live] * (1 - p[live]))
    m = z.size
    assert np.count_nonzero(np.abs(z) > 3) <= m * 0.0027 + 4 * np.sqrt(m * 0.0027) + 1
    assert abs((z ** 2).mean() - 1) < 4 * np.sqrt(2 / m) + 0.1
    assert np.all(counts[p == 1] == S) and np.all(counts[p == 0] == 0)
    sd = np.sqrt(np.where(p > 0, g.astype(np.float64) ** 2 * (1 - p) / np.where(p > 0, p, 1), 0) / S)
    assert np.all(np.abs(qsum / S - g) <= 4 * sd + 1e-6 * np.abs(g))
    assert abs(nnz.mean() - p.sum()) < 4 * np.sqrt((p * (1 - p)).sum() / S)
