"""The no-allocation entry point, sparsify_sample_compact_batched_noalloc, through the C ABI: its
scratch is the library's fixed device array instead of a caller workspace. Its outputs must equal
those of sparsify_sample_compact_batched bit for bit (the same kernels), on calls in a row, each
smaller than the one before (the array keeps the earlier calls' contents), and a call that needs
more scratch than the array holds is rejected before anything is enqueued."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from oracle.compare import compare_sample

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


def _batch(rows, d, seed):
    rng = np.random.default_rng(seed)
    return np.stack([W.t_mixture(d, seed + r) * np.float32(10.0 ** rng.uniform(-3, 0)) for r in range(rows)])


def _noalloc(gs, g, rhos, seeds, solver, cap):
    rows = g.shape[0]
    dev = g.device
    rho_dev = torch.tensor(rhos, dtype=torch.float64, device=dev)
    seeds_dev = torch.tensor(seeds, dtype=torch.int64, device=dev)
    idx = torch.full((rows, cap), -7, dtype=torch.int32, device=dev)
    val = torch.full((rows, cap), -7.0, dtype=torch.float32, device=dev)
    nnz = torch.full((rows,), -7, dtype=torch.int64, device=dev)
    lam = torch.full((rows,), -7.0, dtype=torch.float64, device=dev)
    k = torch.full((rows,), -7, dtype=torch.int64, device=dev)
    fl = torch.full((rows,), -7, dtype=torch.int32, device=dev)
    rc = gs.sparsify_sample_compact_batched_noalloc(g, rho_dev, seeds_dev, idx, val, nnz, lam, k, fl, solver=solver)
    return rc, idx, val, nnz, lam, k, fl


@pytest.mark.parametrize("solver", ["greedy", "exact"])
def test_noalloc_matches_the_workspace_entry_point(gs, solver):
    """Three calls in a row, each smaller than the one before, the first a single row of
    2^25 + 8 coordinates (long enough for a candidate band, kept in the array too), each against
    the workspace entry point (bit for bit) and, for its first row, against the oracle under the
    parity rule."""
    for rows, d, seed in ((1, (1 << 25) + 8, 70), (8, 300007, 10), (3, 70001, 40)):
        gh = _batch(rows, d, seed)
        g = torch.from_numpy(gh).cuda()
        rhos = [(0.01, 0.1, 0.3)[r % 3] for r in range(rows)]
        seeds = [900 + r for r in range(rows)]
        cap = gs.capacity_hint(d, 0.3)
        _say(f"[noalloc] {solver} rows={rows} d={d} scratch need={gs.workspace_bytes(rows, d, solver)}")
        rc, idx, val, nnz, lam, k, fl = _noalloc(gs, g, rhos, seeds, solver, cap)
        assert rc == gs.OK, rc
        ref = gs.sparsify_sample_compact_batched(g, rhos, seeds, solver=solver, cap_per_row=cap)
        torch.cuda.synchronize()
        assert torch.equal(nnz, ref.nnz) and torch.equal(lam, ref.lam) and torch.equal(k, ref.k)
        assert torch.equal(fl, ref.flags) and not fl.any()
        for r in range(rows):
            n = int(nnz[r].item())
            assert torch.equal(idx[r, :n], ref.idx[r, :n]) and torch.equal(val[r, :n], ref.val[r, :n])
            assert bool((idx[r, n:] == -7).all())  # nothing written past the survivors
        sol = oracle.solve(gh[0], rhos[0], solver, 2)
        n0 = int(nnz[0].item())
        compare_sample(gh[0], sol.p, seeds[0], idx[0, :n0].cpu().numpy(), val[0, :n0].cpu().numpy(), n0,
                       float(lam[0].item()), sol.lam)


def test_noalloc_rejects_a_call_larger_than_its_array(gs):
    rows, d = 512, 1 << 20
    assert gs.workspace_bytes(rows, d, "greedy") > 32 << 20
    g = torch.empty((rows, d), dtype=torch.float32, device="cuda")  # 2 GiB, never read
    rc, idx, val, nnz, lam, k, fl = _noalloc(gs, g, [0.1] * rows, list(range(rows)), "greedy", 4)
    torch.cuda.synchronize()
    assert rc == gs.ERR_TOO_LARGE
    assert bool((nnz == -7).all()) and bool((fl == -7).all())
