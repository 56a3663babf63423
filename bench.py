"""Benchmark: sparsified gradient elements per second on one MI355X.

A step sparsifies one batch of synthetic gradients with every (solver, density) the workload lists:
solve (exact threshold or Algorithm 3), Philox Bernoulli sampling, amplification and compaction
into (int32 index, fp32 value) pairs, for all rows. Inputs, outputs and the workspace stay resident
in HBM; the timed region holds exactly K steps between two device synchronisations.

Default workload: 16 rows x 2^20 (one per simulated worker), Laplace(0,1) times a per-row scale
10^U(-3,0), greedy solver with two rescale steps, densities 0.01 and 0.1, Philox seeds 1000 + r.

Prints ONE JSON line with the metric, a roofline object for the dominant kernel (the sampling /
compaction pass: algorithmic bytes = 4 B per input element + 8 B per survivor, timed with HIP
events on its stream over the timed region) and the oracle timed on a bounded sample on one host
core as a CPU baseline.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sparsified gradient elements/sec and achieved HBM GB/s (% of MI355X peak)"
HBM_PEAK_GBS = 8000.0
SRC = os.path.join(ROOT, "paper_1710_09854_amd", "csrc", "gspar.hip")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c2", choices=["c1", "c2", "c3", "c4", "c5"])
    ap.add_argument("--solver", default=None, help="restrict to one solver")
    ap.add_argument("--rho", type=float, default=None, help="restrict to one density")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the oracle sample")
    return ap.parse_args()


def src_hash() -> str:
    with open(SRC, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


def traffic_for(workload: str):
    """HBM bytes per launch of the sampling kernel from committed rocprofv3 counter summaries,
    only if they were taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        data = json.load(open(path))
        ent = data.get("k_sample", {}).get(workload)
        if ent and ent.get("src_sha") == src_hash():
            return ent.get("bytes_per_launch")
    except (ValueError, OSError):
        return None
    return None


def cpu_baseline(wl, combos, target_s):
    """The oracle as it stands (single thread), on whole rows of the same workload until about
    target_s seconds of work; returns elements/s and what the sample was."""
    import oracle

    t0 = time.perf_counter()
    elems = 0
    done = []
    r = 0
    while True:
        row = wl.g[r % wl.rows]
        for solver, rho in combos:
            sol = oracle.solve(row, rho, solver, wl.iters)
            oracle.sample_compact(row, sol.p, wl.seeds[r % wl.rows])
            elems += row.size
        done.append(r % wl.rows)
        r += 1
        if time.perf_counter() - t0 >= target_s or r >= 4 * wl.rows:
            break
    dt = time.perf_counter() - t0
    return {"value": elems / dt, "unit": "elements/s", "cores": 1, "kind": "oracle",
            "sample": f"{r} rows of d={wl.d} x {len(combos)} (solver, rho) combos, {dt:.1f} s, "
                      "fp64 oracle single thread"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); multi-GPU runs are not part of "
              "this build", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_1710_09854_amd as gs
    import workloads

    assert torch.cuda.is_available(), "needs a GPU"
    dev = torch.device("cuda:0")
    wl = workloads.CONFIGS[args.workload]()
    solvers = [args.solver] if args.solver else wl.solvers
    rhos = [args.rho] if args.rho is not None else wl.rhos
    combos = [(s, r) for s in solvers for r in rhos]
    g = torch.from_numpy(wl.g).to(dev)
    rows, d = wl.rows, wl.d
    seeds = torch.tensor([s - (1 << 64) if s >= (1 << 63) else s for s in wl.seeds], dtype=torch.int64, device=dev)
    plans = []
    for solver, rho in combos:
        plan = gs.Plan(rows, d, solver=solver, iters=wl.iters, cap_per_row=gs.capacity_hint(d, rho))
        rho_dev = torch.full((rows,), rho, dtype=torch.float64, device=dev)
        plans.append((plan, rho_dev))

    def step():
        for plan, rho_dev in plans:
            plan.run(g, rho_dev, seeds)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for plan, _ in plans:
        fl = plan.flags.cpu().numpy()
        assert not (fl & ~gs.FLAG_OVERFLOW).any(), f"unexpected flags {fl}"

    timer = gs.KernelTimer(0, args.steps * len(plans))
    nnz_tot = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ksample_ms, launches = timer.read()
    timer.close()
    for plan, _ in plans:
        nnz_tot += int(plan.nnz.sum().item())
    # survivors are identical in every step (same seeds), so per-step bytes are exact
    elements_per_step = rows * d * len(plans)
    ms_per_step = elapsed * 1e3 / args.steps
    value = elements_per_step / (elapsed / args.steps)
    alg_bytes_per_step = 4.0 * elements_per_step + 8.0 * nnz_tot
    avg_launch_ms = ksample_ms / max(launches, 1)
    achieved = alg_bytes_per_step / len(plans) / (avg_launch_ms * 1e-3) / 1e9
    traffic = traffic_for(wl.name)
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "rows": rows, "d": d,
                   "solvers": solvers, "rho": rhos, "greedy_iters": wl.iters,
                   "seeds": "per-row Philox keys " + ("1000+r" if args.workload == "c2" else str(wl.seeds[0])),
                   "parallelism": "single GPU, rows batched in one call"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "k_sample (Philox sampling, amplification, compaction)",
                     "algorithmic_bytes_per_launch": alg_bytes_per_step / len(plans),
                     "avg_launch_ms": avg_launch_ms, "launches": launches},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, combos, args.cpu_seconds)
    line["nnz_per_step"] = nnz_tot
    line["src_sha"] = src_hash()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
