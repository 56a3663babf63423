"""GPU parity of the variance-budget exact solver (Algorithm 2 as printed: the budget (1 + eps) on
the variance, eqs. 6-7) through the C ABI, solver id GSPAR_VARIANCE with eps in place of rho. Both
sides evaluate the criterion of eq. 6 on exactly rounded sums, sums of squares and totals with
the same roundings, so lambda and the capped count are compared bit for bit; the sample under the
parity rule (index sets equal except where |u_i - p_i| <= 1e-6, values to rel 1e-5) and the
probabilities to 1e-6."""
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
@pytest.mark.parametrize("eps", [0.01, 0.1, 1.0, 10.0])
def test_variance_vectors(gs, name, eps):
    g = np.ascontiguousarray(VECTORS[name](), np.float32)
    _say("variance", name, eps)
    sol = oracle.solve_variance(g, eps)
    gd = torch.from_numpy(g).cuda()
    out = gs.sparsify_sample_compact(gd, eps, 99, "variance", capacity=g.size)
    n = int(out.nnz[0].item())
    assert int(out.flags[0].item()) == 0
    assert out.lam[0].item() == sol.lam and int(out.k[0].item()) == sol.k
    compare_sample(g, sol.p, 99, out.idx[:n].cpu().numpy(), out.val[:n].cpu().numpy(), n, out.lam[0].item(), sol.lam)
    pr = gs.sparsify_probs(gd, eps, "variance")
    assert pr.lam[0].item() == sol.lam
    compare_probs(pr.p.cpu().numpy(), sol.p)


def test_variance_random_rows(gs):
    """One hundred seeded random rows for the variance budget (length 1 to ~300 K log-uniform,
    distribution, scale over ten decades, eps from 1e-3 to 1e2): lambda and k bit for bit, the
    sample under the parity rule, the probabilities to 1e-6."""
    rng = np.random.default_rng(9191)
    makers = (W.normal, W.t_mixture, W.integer_ties, W.wide_range, W.lowest_binade)
    for case in range(100):
        d = int(np.exp(rng.uniform(0.0, np.log(300000.0))))
        seed = int(rng.integers(1 << 30))
        g = makers[int(rng.integers(len(makers)))](d, seed)
        g = (g * np.float32(10.0 ** rng.uniform(-6, 4))).astype(np.float32)
        if not g.any():
            continue
        eps = float(10.0 ** rng.uniform(-3.0, 2.0))
        _say(f"[variance-random] case={case} d={d} eps={eps:.5g}")
        sol = oracle.solve_variance(g, eps)
        gd = torch.from_numpy(g).cuda()
        out = gs.sparsify_sample_compact(gd, eps, seed % 100000, "variance", capacity=d)
        n = int(out.nnz[0].item())
        assert int(out.flags[0].item()) == 0, (case, int(out.flags[0].item()))
        assert out.lam[0].item() == sol.lam and int(out.k[0].item()) == sol.k, (case, out.lam[0].item(), sol.lam)
        compare_sample(g, sol.p, seed % 100000, out.idx[:n].cpu().numpy(), out.val[:n].cpu().numpy(), n,
                       out.lam[0].item(), sol.lam)
        pr = gs.sparsify_probs(gd, eps, "variance")
        assert pr.lam[0].item() == sol.lam
        compare_probs(pr.p.cpu().numpy(), sol.p)


def test_variance_batched_laplace_rows(gs):
    """The 16 x 2^20 Laplace batch, one eps per row, through the batched entry point."""
    w = W.c2()
    eps = [0.01 * (1 + r) for r in range(w.rows)]
    _say("variance batched 16 x 2^20")
    out = gs.sparsify_sample_compact_batched(torch.from_numpy(w.g).cuda(), eps, w.seeds, "variance",
                                             cap_per_row=w.d)
    lam, k, nnz = out.lam.cpu().numpy(), out.k.cpu().numpy(), out.nnz.cpu().numpy()
    idx, val = out.idx.cpu().numpy(), out.val.cpu().numpy()
    assert not out.flags.cpu().numpy().any()
    for r in range(w.rows):
        sol = oracle.solve_variance(w.g[r], eps[r])
        assert lam[r] == sol.lam and k[r] == sol.k, (r, lam[r], sol.lam)
        n = int(nnz[r])
        compare_sample(w.g[r], sol.p, w.seeds[r], idx[r, :n], val[r, :n], n, lam[r], sol.lam)


@pytest.mark.parametrize("eps", [0.05, 1.0])
def test_variance_resnet50_gradient(gs, eps):
    """The 25,557,032-coordinate ResNet-50-shaped gradient as one row, and per layer."""
    w = W.c4()
    g = w.g[0]
    gd = torch.from_numpy(g).cuda()
    _say("variance resnet50 whole", eps)
    sol = oracle.solve_variance(g, eps)
    pr = gs.sparsify_probs(gd, eps, "variance", want_p=False)
    assert pr.lam[0].item() == sol.lam and int(pr.k[0].item()) == sol.k
    out = gs.sparsify_sample_compact(gd, eps, 4, "variance", capacity=int(sol.p.sum() * 1.1) + 4096)
    n = int(out.nnz[0].item())
    compare_sample(g, sol.p, 4, out.idx[:n].cpu().numpy(), out.val[:n].cpu().numpy(), n, out.lam[0].item(), sol.lam)
    _say("variance resnet50 per layer", eps)
    off = np.concatenate([[0], np.cumsum(w.meta["segments"])]).astype(np.int64)
    seg = gs.Segments(off)
    segs = off.size - 1
    seeds = [4000 + s for s in range(segs)]
    o = gs.sparsify_sample_compact_segmented(gd, seg, eps, seeds, "variance", cap_per_seg=int(max(w.meta["segments"])))
    lam, k, nnz = o.lam.cpu().numpy(), o.k.cpu().numpy(), o.nnz.cpu().numpy()
    idx, val = o.idx.cpu().numpy(), o.val.cpu().numpy()
    for s in range(segs):
        layer = g[off[s]:off[s + 1]]
        sl = oracle.solve_variance(layer, eps)
        assert lam[s] == sl.lam and k[s] == sl.k, (s, lam[s], sl.lam)
        n = int(nnz[s])
        compare_sample(layer, sl.p, seeds[s], idx[s, :n], val[s, :n], n, lam[s], sl.lam)


def test_variance_bad_eps_is_flagged(gs):
    g = torch.from_numpy(np.ascontiguousarray(np.stack([W.normal(5000, 1), W.normal(5000, 2)]))).cuda()
    _say("variance bad eps")
    out = gs.sparsify_sample_compact_batched(g, [0.1, -1.0], [1, 2], "variance", cap_per_row=5000)
    fl = out.flags.cpu().numpy()
    assert fl[0] == 0 and fl[1] & gs.FLAG_BADRHO and int(out.nnz[1].item()) == 0


def test_variance_hybrid_split(gs):
    """The hybrid coding with the variance-budget solver: Q_A is the capped set {a > v*}, Q_A and
    Q_B together are the compaction's survivors, and both match the oracle's split."""
    g = np.ascontiguousarray(W.t_mixture(150001, 8), np.float32)
    gd = torch.from_numpy(g).cuda()
    _say("variance hybrid")
    for eps in (0.1, 2.0):
        sol = oracle.solve_variance(g, eps)
        h = gs.sparsify_sample_hybrid(gd, eps, 17, "variance", cap_a=g.size, cap_b=g.size, dense_q=True)
        A, B = int(h.n_a[0].item()), int(h.n_b[0].item())
        assert h.lam[0].item() == sol.lam and A == sol.k
        ref = oracle.sample_hybrid(g, sol.p, 17)
        assert np.array_equal(h.idx_a[:A].cpu().numpy(), ref.qa_idx)
        assert np.array_equal(h.code_b[:B].cpu().numpy() & 0x7FFFFFFF, ref.qb_idx)
        assert np.array_equal(h.q.cpu().numpy(), ref.q)


def test_variance_full_size_student_t(gs):
    """The 2^28-coordinate Student-t(2) gradient with 1 % outliers at eps = 1, in the launch the
    benchmark times (one call, output capacity d): lambda and k bit for bit, every survivor under
    the parity rule."""
    w = W.c5()
    g = w.g[0]
    _say("variance 2^28 student-t eps 1")
    gd = torch.from_numpy(g).cuda()
    out = gs.sparsify_sample_compact_batched(gd.view(1, -1), [1.0], w.seeds, "variance", cap_per_row=w.d)
    lam, k, n = out.lam[0].item(), int(out.k[0].item()), int(out.nnz[0].item())
    idx, val = out.idx[0, :n].cpu().numpy(), out.val[0, :n].cpu().numpy()
    del out, gd
    torch.cuda.empty_cache()
    sol = oracle.solve_variance(g, 1.0)
    assert lam == sol.lam and k == sol.k, (lam, sol.lam, k, sol.k)
    compare_sample(g, sol.p, w.seeds[0], idx, val, n, lam, sol.lam)
