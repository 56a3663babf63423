"""CPU runs of the HIP kernels through the host emulation in tests/emu (no GPU needed).

The unchanged library source is compiled with g++ against a small HIP-runtime emulation in which
the threads of a workgroup are fibers switched at barriers, shuffles, ballots and sleeps. These
tests check kernel indexing, the solver's control flow (every thread of a workgroup must pass the
same barriers; a barrier that can never release is reported) and the whole pipeline against the
oracle, on small inputs: each check once in the default schedule, the whole sweep again under
AddressSanitizer, and again with the fibers scheduled at random."""
import os
import subprocess
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "emu"))

import build as emu_build  # noqa: E402
import runner  # noqa: E402


@pytest.fixture(scope="module")
def emu_lib():
    return emu_build.build(asan=False)


def test_emulated_special_batched_overflow_unaligned(emu_lib):
    assert runner.run_extra(emu_lib, verbose=False)


def test_emulated_hybrid_coding(emu_lib):
    assert runner.check_hybrid(runner.load(emu_lib), verbose=False)


def test_emulated_capped_ties(emu_lib):
    assert runner.check_ties(runner.load(emu_lib), verbose=False)


def test_emulated_candidate_band(emu_lib):
    assert runner.check_candidates(runner.load(emu_lib), verbose=False)


def test_emulated_answer_inside_the_lowest_binade(emu_lib):
    assert runner.check_lowest_binade(runner.load(emu_lib), verbose=False)


def test_emulated_full_range_rows(emu_lib):
    assert runner.check_full_range(runner.load(emu_lib), verbose=False)


def test_emulated_random_rows_batches_segments(emu_lib):
    assert runner.check_random(runner.load(emu_lib), verbose=False)


def test_emulated_capped_values_past_the_lane_rows(emu_lib):
    assert runner.check_lane_rows(runner.load(emu_lib), verbose=False)


def test_emulated_band_region_overflow(emu_lib):
    assert runner.check_band_region_overflow(runner.load(emu_lib), verbose=False)


def test_emulated_variance_solver(emu_lib):
    assert runner.check_variance(runner.load(emu_lib), verbose=False)


def test_emulated_segmented(emu_lib):
    assert runner.check_segmented(runner.load(emu_lib), verbose=False)


def test_emulated_aggregate(emu_lib):
    assert runner.check_aggregate(runner.load(emu_lib), verbose=False)


def test_emulated_parity_subset(emu_lib):
    L = runner.load(emu_lib)
    import oracle
    import workloads as W
    from oracle.compare import compare_sample

    for name, mk in [("spiked", lambda: np.concatenate([W.normal(37, 9) * np.float32(40), W.normal(20000, 0)])),
                     ("tmix", lambda: W.t_mixture(30001, 2)), ("ties", lambda: W.integer_ties(12001, 3))]:
        g = np.ascontiguousarray(mk(), np.float32)
        for solver in ("greedy", "exact"):
            for rho in (0.01, 0.5):
                sol = oracle.solve(g, rho, solver, 2)
                idx, val, n, lam, k, fl = runner.sample_row(L, g, rho, solver, 77)
                assert fl == 0
                compare_sample(g, sol.p, 77, idx, val, n, lam, sol.lam)
                if solver == "exact":
                    assert lam == sol.lam and k == sol.k


def test_emulated_full_sweep(emu_lib):
    assert runner.run_all(emu_lib, verbose=False) == 64


def test_emulated_asan_subset():
    """Kernel indexing under AddressSanitizer: a padded batch ending in partial groups with a
    candidate band, the scalar path, the variance budget, segments on both paths with the hybrid
    coding, and aggregation (the whole sweep under ASan is below)."""
    lib = emu_build.build(asan=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", LD_PRELOAD=emu_build.asan_runtime())
    r = subprocess.run([sys.executable, os.path.join(HERE, "emu", "runner.py"), lib, "asan_subset"], env=env,
                       capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0 and "AddressSanitizer" not in r.stderr, r.stderr[-2000:]
    assert "asan subset ok" in r.stdout, r.stdout[-2000:]


def test_emulated_under_asan():
    """Every emulated check (edge cases, batching, overflow, the unaligned path, hybrid coding,
    ties, the candidate band and its overflows, aggregation, the variance budget, segments and the
    parity sweep) under AddressSanitizer."""
    lib = emu_build.build(asan=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", LD_PRELOAD=emu_build.asan_runtime())
    r = subprocess.run([sys.executable, os.path.join(HERE, "emu", "runner.py"), lib, "all"], env=env,
                       capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0 and "AddressSanitizer" not in r.stderr, r.stderr[-2000:]
    assert "checked 64" in r.stdout, r.stdout[-2000:]


def test_emulated_random_schedule(emu_lib):
    """Every emulated check again with the fibers of each workgroup scheduled at random, so that
    lanes run in another order after each barrier: a read of shared state that no barrier
    separates from another lane's write sees the wrong value in some workgroup."""
    env = dict(os.environ, EMU_SHUFFLE="1")
    r = subprocess.run([sys.executable, os.path.join(HERE, "emu", "runner.py"), emu_lib, "all"], env=env,
                       capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-2000:])
    assert "checked 64" in r.stdout, r.stdout[-2000:]


def test_emulated_lookback_fallback():
    """Hide every published tile status so each look-back counts its predecessors itself."""
    lib = emu_build.build(asan=False)
    env = dict(os.environ, EMU_HIDE_STATUS="1", EMU_STALL_SECONDS="300")
    r = subprocess.run([sys.executable, os.path.join(HERE, "emu", "runner.py"), lib, "extra_lite"], env=env,
                       capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0 and "extra cases ok" in r.stdout, (r.stdout[-2000:], r.stderr[-2000:])
    r = subprocess.run([sys.executable, os.path.join(HERE, "emu", "runner.py"), lib, "ties"], env=env,
                       capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0 and "tie cases ok" in r.stdout, (r.stdout[-2000:], r.stderr[-2000:])


def test_emulated_two_tiles_per_workgroup():
    """The sampling pass's two-tiles-per-workgroup path (taken on the GPU by grids larger than the
    resident set) forced on the small emulated inputs: edge cases, batching, overflow, the
    unaligned path and the hybrid coding, with tile counts odd and even (segmented rows with two
    tiles per workgroup run on the GPU, in tests/test_gpu_segmented.py)."""
    env = dict(os.environ, GSPAR_EMU_RESIDENT="1", GSPAR_EMU_CAND_MIN_ROW=str(1 << 22))
    lib = subprocess.run([sys.executable, "-c", "import sys; sys.path.insert(0, %r); import build; print(build.build())"
                          % os.path.join(HERE, "emu")], env=env, capture_output=True, text=True, check=True).stdout.strip()
    r = subprocess.run([sys.executable, os.path.join(HERE, "emu", "runner.py"), lib, "extra_lite"], env=env,
                       capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0 and "extra cases ok" in r.stdout, (r.stdout[-2000:], r.stderr[-2000:])
    r = subprocess.run([sys.executable, os.path.join(HERE, "emu", "runner.py"), lib, "hybrid"], env=env,
                       capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0 and "hybrid cases ok" in r.stdout, (r.stdout[-2000:], r.stderr[-2000:])
