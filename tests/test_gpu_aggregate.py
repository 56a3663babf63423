"""GPU parity of the aggregation step (Algorithm 1, step 6) through the C ABI: v = (1/M) sum_m Q(g^m)
from M workers' ascending (index, value) lists. Both sides sum each coordinate in fp64 in worker
order, divide by M and round to fp32, so the comparison is bit for bit. The lists come from the
oracle's own sparsifier on the 16 x 2^20 Laplace batch (one worker per row, as the sampling pass
writes them) and from the seeded list generator (empty and overflowed lists, clustered ranges,
more workers than one pass of the kernel holds, ragged lengths)."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W

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


def _lists(idx, val, nnz):
    cap = idx.shape[1]
    return [(idx[m, :max(0, min(int(n), cap))], val[m, :max(0, min(int(n), cap))]) for m, n in enumerate(nnz)]


def _gpu(gs, idx, val, nnz, d):
    dev = torch.device("cuda:0")
    v = gs.aggregate(torch.from_numpy(idx).to(dev), torch.from_numpy(val).to(dev), torch.from_numpy(nnz).to(dev), d)
    torch.cuda.synchronize()
    return v.cpu().numpy()


@pytest.fixture(scope="module")
def c2_lists():
    w = W.c2()
    out = {}
    for rho in (0.01, 0.1):
        lists = []
        for r in range(w.rows):
            sol = oracle.solve_greedy(w.g[r], rho, w.iters)
            idx, val, n = oracle.sample_compact(w.g[r], sol.p, w.seeds[r])
            lists.append((idx, val))
        cap = max(i.size for i, _ in lists) + 5
        I = np.zeros((w.rows, cap), np.int32)
        V = np.zeros((w.rows, cap), np.float32)
        N = np.zeros(w.rows, np.int64)
        for r, (i, v) in enumerate(lists):
            I[r, :i.size], V[r, :i.size], N[r] = i, v, i.size
        out[rho] = (I, V, N, w.d)
    return out


@pytest.mark.parametrize("rho", [0.01, 0.1])
def test_aggregate_c2_batch(gs, c2_lists, rho):
    I, V, N, d = c2_lists[rho]
    _say("aggregate c2 16 x 2^20 rho", rho)
    v = _gpu(gs, I, V, N, d)
    assert np.array_equal(v, oracle.aggregate(_lists(I, V, N), d))


@pytest.mark.parametrize("rho", [0.01, 0.1])
def test_aggregate_c2_first_workers(gs, c2_lists, rho):
    """Fewer workers than rows (M = 1, 3, 7), a capacity that truncates the longest lists."""
    I, V, N, d = c2_lists[rho]
    for M in (1, 3, 7):
        cap = int(np.median(N[:M]))
        Ic, Vc = np.ascontiguousarray(I[:M, :cap]), np.ascontiguousarray(V[:M, :cap])
        _say("aggregate c2 rho", rho, "workers", M, "cap", cap)
        v = _gpu(gs, Ic, Vc, N[:M].copy(), d)
        assert np.array_equal(v, oracle.aggregate(_lists(Ic, Vc, N[:M]), d))


SYNTH = [  # workers, d, cap
    (37, 100003, 30000),
    (1, (1 << 22) + 3, 200000),
    (16, 2048, 2048),
    (17, 999, 400),
    (64, 1 << 20, 20000),
    (2, 1, 1),
    (300, 50001, 500),
]


@pytest.mark.parametrize("case", range(len(SYNTH)))
def test_aggregate_synthetic_lists(gs, case):
    workers, d, cap = SYNTH[case]
    idx, val, nnz = W.sparse_lists(workers, d, cap, 700 + case, empty=(1, 2) if workers > 2 else (),
                                   over=(0,) if workers > 1 else ())
    _say("aggregate synthetic", workers, d, cap)
    v = _gpu(gs, idx, val, nnz, d)
    assert np.array_equal(v, oracle.aggregate(_lists(idx, val, nnz), d))


def test_aggregate_zero_capacity(gs):
    _say("aggregate zero capacity")
    dev = torch.device("cuda:0")
    idx = torch.zeros((3, 0), dtype=torch.int32, device=dev)
    val = torch.zeros((3, 0), dtype=torch.float32, device=dev)
    v = gs.aggregate(idx, val, torch.tensor([5, 0, 2], device=dev), 5000)
    torch.cuda.synchronize()
    assert torch.equal(v.cpu(), torch.zeros(5000))


def test_aggregate_skips_out_of_range_entries(gs):
    """Entries outside [0, d) at either end of an ascending list are skipped."""
    idx, val, nnz = W.sparse_lists(4, 60000, 1500, 800)
    n0 = int(nnz[0])
    idx[0, :n0] = np.sort(idx[0, :n0])
    idx[0, :3] = [-7, -1, 0]
    n1 = int(nnz[1])
    idx[1, n1 - 3:n1] = [60000, 60001, 2**31 - 1]
    idx[1, :n1] = np.sort(idx[1, :n1])
    _say("aggregate out-of-range entries")
    v = _gpu(gs, idx, val, nnz, 60000)
    lists = []
    for i, x in _lists(idx, val, nnz):
        keep = (i >= 0) & (i < 60000)
        lists.append((i[keep], x[keep]))
    assert np.array_equal(v, oracle.aggregate(lists, 60000))


@pytest.mark.parametrize("solver", ["greedy", "exact"])
def test_aggregate_then_sparsify_the_average(gs, c2_lists, solver):
    """Algorithm 1 steps 6-7 on one device: the average of the workers' messages, sparsified again
    before it is broadcast. The average is bit-exact, so the second sparsification is checked under
    the parity rule against the oracle's sparsification of the oracle's average."""
    from oracle.compare import compare_sample

    I, V, N, d = c2_lists[0.1]
    _say("aggregate then sparsify", solver)
    v = gs.aggregate(torch.from_numpy(I).cuda(), torch.from_numpy(V).cuda(), torch.from_numpy(N).cuda(), d)
    out = gs.sparsify_sample_compact(v, 0.01, 4242, solver)
    torch.cuda.synchronize()
    v_ref = oracle.aggregate(_lists(I, V, N), d)
    assert np.array_equal(v.cpu().numpy(), v_ref)
    sol = oracle.solve(v_ref, 0.01, solver, 2)
    n = int(out.nnz[0].item())
    compare_sample(v_ref, sol.p, 4242, out.idx[:n].cpu().numpy(), out.val[:n].cpu().numpy(), n, out.lam[0].item(),
                   sol.lam)
