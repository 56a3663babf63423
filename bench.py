"""Benchmark: sparsified gradient elements per second on one MI355X.

A step sparsifies one batch of synthetic gradients with every (solver, density) the workload lists:
solve (exact threshold or Algorithm 3), Philox Bernoulli sampling, amplification and compaction
into (int32 index, fp32 value) pairs, for all rows. Inputs, outputs and the workspace stay resident
in HBM; the timed region holds exactly K steps between two device synchronisations, with no timer
armed (product library).

Default workload: one gradient of 2^28 coordinates (1 GiB), Student-t(2) with 1% of the entries
multiplied by 100, the exact and the greedy (two rescale steps) solvers at densities 0.001, 0.01
and 0.1 (six calls per step), Philox seed 5. --workload c2 selects 16 rows x 2^20 (Laplace times a
per-row scale 10^U(-3,0), greedy, densities 0.01 and 0.1, seeds 1000 + r), and so on.

Prints ONE JSON line with the metric, a roofline object for the sampling / compaction pass
(algorithmic bytes = 4 B per input element + 8 B per survivor over its average kernel time), the
time per step of every kernel class, and the oracle timed on a bounded sample on one host core as
a CPU baseline. Kernel times come from a second loop of the same steps through the measurement
build of the library (libgspar_instr.so, the same kernels), whose launches carry HIP events
stamped by the dispatch itself at the kernel's start and end.

With --cells (and --workload all for every workload) it prints instead one line per (workload,
solver, rho): the median time of one call warm and right after a 512 MiB scratch write that evicts
the last-level cache, elements/s, the algorithmic HBM fraction and the oracle's one-core rate.

Counter runs: with --copy-probe the run first copies a 512 MiB device buffer three times (a plain
copy kernel of known size), so that two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) can be
scaled to bytes; `bench.py --summarize-pmc FETCH_DIR WRITE_DIR` turns those two runs into bytes
per launch per kernel and records them in profiles/traffic.json for the current kernel source.
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
    ap.add_argument("--workload", default="c5", choices=["c1", "c2", "c3", "c4", "c5", "all"])
    ap.add_argument("--solver", default=None, choices=["greedy", "exact", "variance"],
                    help="restrict to one solver ('variance': Algorithm 2 with the variance budget eps)")
    ap.add_argument("--rho", type=float, default=None,
                    help="restrict to one density (with --solver variance: one eps; default eps 0.1 and 1)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the oracle sample")
    ap.add_argument("--copy-probe", action="store_true", help="copy a 512 MiB buffer 3 times first (counter scale)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"), default=None,
                    help="summarise two rocprofv3 --pmc runs of this benchmark into profiles/traffic.json")
    ap.add_argument("--hybrid", action="store_true",
                    help="time the hybrid coding entry point (Q_A / Q_B lists) instead of the compaction")
    ap.add_argument("--dense-q", action="store_true", help="with --hybrid, also write the dense ternary vector")
    ap.add_argument("--probs", action="store_true",
                    help="time the probabilities entry point (p = min(lambda |g|, 1) written in full: 8 B per "
                         "coordinate) instead of the compaction")
    ap.add_argument("--per-layer", action="store_true",
                    help="c4 only: sparsify each of the 54 ResNet-50 layers on its own (one lambda per layer, "
                         "Philox keys 4000 + layer) in one segmented call")
    ap.add_argument("--aggregate", action="store_true",
                    help="with --cells: also time the aggregation (Algorithm 1, step 6) of each cell's lists, "
                         "one worker per row")
    ap.add_argument("--cells", action="store_true",
                    help="one JSON line per (workload, solver, rho) cell instead of the step line: median call "
                         "time warm and after evicting the caches, algorithmic HBM fraction, oracle rate")
    ap.add_argument("--stream-probe", action="store_true",
                    help="one JSON line instead of the step line: the bandwidth a plain read kernel and a plain "
                         "copy kernel reach on 1 GiB (the default workload's gradient size)")
    return ap.parse_args()


def stream_probe():
    """Achievable stream bandwidth on this part: the measurement build's plain read kernel over a
    1 GiB buffer (4 B per element read once) and its copy kernel over 512 MiB (read + written), each
    the median of 20 timings with events on the stream: warm (ten runs back to back per timing) and
    right after a 512 MiB write that evicts the last-level cache (one run)."""
    import numpy as np
    import torch

    import paper_1710_09854_amd as gs

    dev = torch.device("cuda:0")
    n = 1 << 28
    src = torch.rand(n, dtype=torch.float32, device=dev)
    sink = torch.zeros(1, dtype=torch.float64, device=dev)
    half = n // 2
    dst = torch.empty(half, dtype=torch.float32, device=dev)
    scratch = torch.empty(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)

    def timed(fn, evict):
        # warm: ten runs back to back, so the host's launch time is hidden behind the kernels;
        # cold: one run queued right behind the eviction (which keeps the device busy meanwhile)
        reps = 1 if evict else 10
        if evict:
            scratch.fill_(0.5)
        else:
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e-3 / reps

    read = lambda: gs.probe_stream(src, sink=sink)
    copy = lambda: gs.probe_stream(src[:half], dst=dst)
    for _ in range(3):
        read()
        copy()
    torch.cuda.synchronize()
    out = {"probe": "stream", "read_bytes": 4 * n, "copy_bytes": 8 * half}
    for name, fn, nbytes in (("read", read, 4 * n), ("copy", copy, 8 * half)):
        for evict in (False, True):
            t = float(np.median([timed(fn, evict) for _ in range(20)]))
            key = name + ("_cold" if evict else "_warm")
            out[key + "_us"] = t * 1e6
            out[key + "_GBps"] = nbytes / t / 1e9
            out[key + "_frac_of_8TBps"] = nbytes / t / 1e9 / HBM_PEAK_GBS
    print(json.dumps(out), flush=True)


def src_hash() -> str:
    with open(SRC, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


TRAFFIC_JSON = os.path.join(ROOT, "profiles", "traffic.json")
COPY_PROBE_BYTES = 512 << 20


def traffic_for(workload: str, kernel: str = "k_sample"):
    """HBM bytes per launch of one kernel from the committed counter summary, only if it was taken
    on the current kernel source (otherwise None)."""
    if not os.path.exists(TRAFFIC_JSON):
        return None
    try:
        data = json.load(open(TRAFFIC_JSON))
        ent = data.get(workload, {})
        if ent.get("src_sha") == src_hash():
            return ent.get("kernels", {}).get(kernel, {}).get("bytes_per_launch")
    except (ValueError, OSError):
        return None
    return None


def _pmc_rows(path):
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {path}")
    rows = []
    for f in files:
        rows.extend(csv.DictReader(open(f)))
    return rows


def _kernel_class(name: str):
    for k in ("k_probs_out", "k_presample", "k_sample", "k_stats", "k_refine", "k_solve", "k_init", "k_probs",
              "k_aggregate"):
        if "gspar::" + k + "<" in name or "gspar::" + k + "(" in name:
            return k
    if "copyBuffer" in name:  # the runtime's device-to-device copy kernel (the probe)
        return "copy"
    return None


def summarize_pmc(fetch_dir, write_dir, workload):
    """Average FETCH_SIZE / WRITE_SIZE (KiB per dispatch) per kernel class; the copy probe's
    readings divided by its known bytes give the scale from counter units to bytes."""
    avg = {}
    for counter, path in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        acc = {}
        for r in _pmc_rows(path):
            if r.get("Counter_Name") != counter:
                continue
            k = _kernel_class(r.get("Kernel_Name", ""))
            if k is None:
                continue
            v = float(r["Counter_Value"])
            if k == "copy" and v * 1024.0 < 0.5 * COPY_PROBE_BYTES:
                continue  # small runtime copies (inputs, scalars), not the probe
            acc.setdefault(k, []).append(v)
        avg[counter] = {k: sum(v) / len(v) for k, v in acc.items()}
    if "copy" not in avg["FETCH_SIZE"] or "copy" not in avg["WRITE_SIZE"]:
        raise SystemExit("the copy probe is missing from the counter runs (run them with --copy-probe)")
    fscale = avg["FETCH_SIZE"]["copy"] * 1024.0 / COPY_PROBE_BYTES
    wscale = avg["WRITE_SIZE"]["copy"] * 1024.0 / COPY_PROBE_BYTES
    kernels = {}
    for k in sorted(set(avg["FETCH_SIZE"]) & set(avg["WRITE_SIZE"]) - {"copy"}):
        fb = avg["FETCH_SIZE"][k] * 1024.0 / fscale
        wb = avg["WRITE_SIZE"][k] * 1024.0 / wscale
        kernels[k] = {"fetch_kib_raw": avg["FETCH_SIZE"][k], "write_kib_raw": avg["WRITE_SIZE"][k],
                      "fetch_bytes": fb, "write_bytes": wb, "bytes_per_launch": fb + wb}
    data = json.load(open(TRAFFIC_JSON)) if os.path.exists(TRAFFIC_JSON) else {}
    data[workload] = {"src_sha": src_hash(), "copy_probe_bytes": COPY_PROBE_BYTES,
                      "fetch_scale": fscale, "write_scale": wscale, "kernels": kernels}
    with open(TRAFFIC_JSON, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
    print(json.dumps(data[workload], indent=1, sort_keys=True))


VARIANCE_EPS = [0.1, 1.0]


def capacity(gs, d, solver, rho):
    """Output capacity per row: from the density, or every coordinate for the variance budget
    (whose expected survivor count is not known before the solve)."""
    return d if solver == "variance" else gs.capacity_hint(d, rho)


def layer_setup(args, wl, dev):
    """Inputs of a per-layer run: the flat gradient, its segments and one Philox key per layer."""
    import torch

    import paper_1710_09854_amd as gs

    if "segments" not in wl.meta:
        raise SystemExit("--per-layer needs a workload with layer segments (c4)")
    seg = gs.Segments.from_lengths(wl.meta["segments"], device=dev)
    g = torch.from_numpy(wl.g[0]).to(dev)
    seeds = torch.arange(4000, 4000 + seg.segs, dtype=torch.int64, device=dev)
    return g, seg, seeds


def cpu_baseline(wl, combos, target_s, per_layer=False, probs=False):
    """The oracle as it stands (single thread), on whole rows of the same workload until about
    target_s seconds of work; returns elements/s and what the sample was."""
    import oracle

    host_cores = len(os.sched_getaffinity(0))
    keep = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {min(keep)})  # the oracle is single-threaded: time it on one core
    try:
        t0 = time.perf_counter()
        elems = 0
        r = 0
        prefix = min(wl.d, 1 << 24)  # rows longer than 2^24 are sampled by their leading 2^24 entries
        if per_layer:
            # layer after layer of the flat gradient, each solved and sampled on its own
            lens = wl.meta["segments"]
            off = [0]
            for n in lens:
                off.append(off[-1] + n)
            while True:
                s = r % len(lens)
                layer = wl.g[0][off[s]:off[s + 1]]
                for solver, rho in combos:
                    oracle.sparsify(layer, rho, solver, wl.iters, 4000 + s)
                    elems += layer.size
                r += 1
                if time.perf_counter() - t0 >= target_s or r >= len(lens):
                    break
            dt = time.perf_counter() - t0
            return {"value": elems / dt, "unit": "elements/s", "cores": 1, "kind": "oracle",
                    "sample": f"the first {r} of the {len(lens)} layers, each solved and sampled on its own, x "
                              f"{len(combos)} (solver, rho) combos; {dt:.1f} s of fp64 oracle work on 1 of the "
                              f"host's {host_cores} cores"}
        while True:
            row = wl.g[r % wl.rows][:prefix]
            for solver, rho in combos:
                sol = oracle.solve(row, rho, solver, wl.iters)
                if not probs:
                    oracle.sample_compact(row, sol.p, wl.seeds[r % wl.rows])
                elems += row.size
            r += 1
            if time.perf_counter() - t0 >= target_s or r >= 4 * wl.rows:
                break
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, keep)
    return {"value": elems / dt, "unit": "elements/s", "cores": 1, "kind": "oracle",
            "sample": f"{r} row passes over {min(r, wl.rows)} distinct rows, each the leading {prefix} of the "
                      f"row's {wl.d} entries, x {len(combos)} (solver, rho) combos"
                      f"{' (solve and p only)' if probs else ''}; {dt:.1f} s of fp64 oracle "
                      f"work on 1 of the host's {host_cores} cores"}


def _class_order():
    import paper_1710_09854_amd as gs

    return gs.PROF_CLASSES


def cells(args):
    """One JSON line per (workload, solver, rho): the median time of one call over 20 (inputs resident,
    warm caches) and over 5 calls each made right after writing a 512 MiB scratch buffer (which evicts
    the 256 MB last-level cache), elements/s for both, the algorithmic HBM fraction
    (4 B per element + 8 B per survivor over the call time, against 8 TB/s), and the oracle's rate
    on one host core on a bounded sample of the same rows."""
    import numpy as np
    import torch

    import paper_1710_09854_amd as gs
    import workloads

    assert torch.cuda.is_available(), "needs a GPU"
    dev = torch.device("cuda:0")
    names = ["c1", "c2", "c3", "c4", "c5"] if args.workload == "all" else [args.workload]
    scratch = torch.empty(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
    for name in names:
        wl = workloads.CONFIGS[name]()
        seg = None
        if args.per_layer:
            if "segments" not in wl.meta:
                continue
            g, seg, seeds = layer_setup(args, wl, dev)
            rows, d = seg.segs, seg.max_len
            n_elems = seg.total
        else:
            g = torch.from_numpy(wl.g).to(dev)
            rows, d = wl.rows, wl.d
            n_elems = rows * d
            seeds = torch.tensor([s - (1 << 64) if s >= (1 << 63) else s for s in wl.seeds], dtype=torch.int64,
                                 device=dev)
        for solver in ([args.solver] if args.solver else wl.solvers):
            for rho in ([args.rho] if args.rho is not None else (VARIANCE_EPS if solver == "variance" else wl.rhos)):
                plan = gs.Plan(rows, d, solver=solver, iters=wl.iters, cap_per_row=capacity(gs, d, solver, rho),
                               hybrid=args.hybrid, dense_q=args.dense_q, segments=seg, probs=args.probs)
                rho_dev = torch.full((rows,), rho, dtype=torch.float64, device=dev)
                for _ in range(3):
                    plan.run(g, rho_dev, seeds)
                torch.cuda.synchronize()
                fl = plan.flags.cpu().numpy()
                assert not fl.any(), f"unexpected flags {fl}"

                def timed(evict):
                    if evict:
                        scratch.fill_(0.5)
                    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    s.record()
                    plan.run(g, rho_dev, seeds)
                    e.record()
                    torch.cuda.synchronize()
                    return s.elapsed_time(e) * 1e-3

                warm = float(np.median([timed(False) for _ in range(20)]))
                cold = float(np.median([timed(True) for _ in range(5)]))
                nnz, out_bytes = plan.survivors_and_bytes()
                alg = 4.0 * n_elems + out_bytes
                entry = ("probs" if args.probs else
                         "hybrid" + ("+q" if args.dense_q else "") if args.hybrid else "compact")
                # kernel times of the same call through the measurement build
                iplan = gs.Plan(rows, d, solver=solver, iters=wl.iters, cap_per_row=capacity(gs, d, solver, rho),
                                hybrid=args.hybrid, dense_q=args.dense_q, segments=seg, probs=args.probs,
                                library=gs.instr_lib())
                iplan.run(g, rho_dev, seeds)
                torch.cuda.synchronize()
                prof = gs.KernelProfiler(10 * 16)
                for _ in range(10):
                    iplan.run(g, rho_dev, seeds)
                kt = prof.read()
                prof.close()
                del iplan
                kernels = {k: {"us_per_call": 100.0 * ms, "launches_per_call": n / 10}
                           for k, (ms, n) in kt.items() if n}
                cell = {"workload": wl.name, "solver": solver, "rho": rho, "rows": rows, "d": d, "nnz": nnz,
                        "entry": entry + ("_per_layer" if args.per_layer else ""),
                        "lambda_row0": float(plan.lam[0].item()),
                        "warm_us": warm * 1e6, "warm_elements_per_s": n_elems / warm,
                        "cold_us": cold * 1e6, "cold_elements_per_s": n_elems / cold,
                        "algorithmic_bytes": alg, "algorithmic_frac_warm": alg / warm / 1e9 / HBM_PEAK_GBS,
                        "algorithmic_frac_cold": alg / cold / 1e9 / HBM_PEAK_GBS, "kernels": kernels}
                if not args.no_cpu_baseline:
                    cell["cpu_baseline"] = cpu_baseline(wl, [(solver, rho)], args.cpu_seconds,
                                                        per_layer=args.per_layer and not args.probs,
                                                        probs=args.probs)
                print(json.dumps(cell), flush=True)
                if args.aggregate and not args.hybrid and not args.per_layer:
                    print(json.dumps(aggregate_cell(args, wl, plan, scratch, solver, rho)), flush=True)
                del plan
        del g
        torch.cuda.empty_cache()


def aggregate_cell(args, wl, plan, scratch, solver, rho):
    """The aggregation v = (1/M) sum_m Q(g^m) of the plan's lists (M = rows): median call time warm
    and after a cache-evicting write, the kernel time from HIP events on its stream, algorithmic bytes
    (8 B per kept list entry and per length read, 4 B per output coordinate), and the oracle's
    one-core time on the same lists."""
    import numpy as np
    import torch

    import paper_1710_09854_amd as gs

    rows, d = wl.rows, wl.d
    idx, val, nnz = plan.idx[:, :plan.cap], plan.val[:, :plan.cap], plan.nnz
    v = torch.empty(d, dtype=torch.float32, device=idx.device)
    for _ in range(3):
        gs.aggregate(idx, val, nnz, d, out=v)
    torch.cuda.synchronize()

    def timed(evict):
        if evict:
            scratch.fill_(0.5)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        gs.aggregate(idx, val, nnz, d, out=v)
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e) * 1e-3

    warm = float(np.median([timed(False) for _ in range(20)]))
    cold = float(np.median([timed(True) for _ in range(5)]))
    L = gs.instr_lib()
    gs.aggregate(idx, val, nnz, d, out=v, library=L)
    torch.cuda.synchronize()
    t = gs.KernelProfiler(20)
    for _ in range(20):
        gs.aggregate(idx, val, nnz, d, out=v, library=L)
    ms, n = t.read()["k_aggregate"]
    t.close()
    kept = int(torch.clamp(nnz, 0, plan.cap).sum().item())
    alg = 8.0 * kept + 8.0 * rows + 4.0 * d
    kernel_s = ms * 1e-3 / max(n, 1)
    cell = {"workload": wl.name, "entry": "aggregate", "solver": solver, "rho": rho, "workers": rows, "d": d,
            "kept_entries": kept, "warm_us": warm * 1e6, "cold_us": cold * 1e6, "kernel_us": kernel_s * 1e6,
            "algorithmic_bytes": alg, "algorithmic_frac_kernel": alg / kernel_s / 1e9 / HBM_PEAK_GBS,
            "algorithmic_frac_cold": alg / cold / 1e9 / HBM_PEAK_GBS}
    if not args.no_cpu_baseline:
        import oracle

        I, V, N = idx.cpu().numpy(), val.cpu().numpy(), nnz.cpu().numpy()
        lists = [(I[m, :min(int(N[m]), plan.cap)], V[m, :min(int(N[m]), plan.cap)]) for m in range(rows)]
        keep = os.sched_getaffinity(0)
        os.sched_setaffinity(0, {min(keep)})
        try:
            t0 = time.perf_counter()
            reps = 0
            while reps < 3 or time.perf_counter() - t0 < 2.0:
                oracle.aggregate(lists, d)
                reps += 1
            dt = (time.perf_counter() - t0) / reps
        finally:
            os.sched_setaffinity(0, keep)
        cell["cpu_baseline"] = {"value": dt * 1e6, "unit": "us per aggregation", "cores": 1, "kind": "oracle",
                                "sample": f"{reps} aggregations of the same {rows} lists on one host core"}
    return cell


def main():
    args = parse()
    if args.summarize_pmc:
        wl_name = {"c1": "c1_normal_d65536", "c2": "c2_laplace_16x1048576", "c3": "c3_logreg_256x4194304",
                   "c4": "c4_resnet50_d25557032", "c5": "c5_student_t2_outliers_d268435456"}[args.workload]
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], wl_name)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the sparsifier runs each "
              "worker's rows on its own GPU and has no multi-GPU step to time", file=sys.stderr)
        sys.exit(2)
    if args.cells:
        cells(args)
        return
    if args.stream_probe:
        stream_probe()
        return
    if args.workload == "all":
        print("--workload all needs --cells", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_1710_09854_amd as gs
    import workloads

    assert torch.cuda.is_available(), "needs a GPU"
    dev = torch.device("cuda:0")
    wl = workloads.CONFIGS[args.workload]()
    solvers = [args.solver] if args.solver else wl.solvers
    combos = [(s, r) for s in solvers
              for r in ([args.rho] if args.rho is not None else (VARIANCE_EPS if s == "variance" else wl.rhos))]
    rhos = sorted({r for _, r in combos})
    seg = None
    if args.per_layer:
        g, seg, seeds = layer_setup(args, wl, dev)
        rows, d = seg.segs, seg.max_len
        n_elems = seg.total
    else:
        g = torch.from_numpy(wl.g).to(dev)
        rows, d = wl.rows, wl.d
        n_elems = rows * d
        seeds = torch.tensor([s - (1 << 64) if s >= (1 << 63) else s for s in wl.seeds], dtype=torch.int64,
                             device=dev)
    def make_plans(library):
        out = []
        for solver, rho in combos:
            plan = gs.Plan(rows, d, solver=solver, iters=wl.iters, cap_per_row=capacity(gs, d, solver, rho),
                           hybrid=args.hybrid, dense_q=args.dense_q, segments=seg, library=library,
                           probs=args.probs)
            out.append((plan, torch.full((rows,), rho, dtype=torch.float64, device=dev)))
        return out

    plans = make_plans(None)  # the product library

    def step(ps):
        for plan, rho_dev in ps:
            plan.run(g, rho_dev, seeds)

    if args.copy_probe:
        src = torch.empty(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step(plans)
    torch.cuda.synchronize()
    for plan, _ in plans:
        fl = plan.flags.cpu().numpy()
        assert not (fl & ~gs.FLAG_OVERFLOW).any(), f"unexpected flags {fl}"

    # the timed region: K steps through the product library, no timer armed
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(plans)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    nnz_tot, out_bytes = 0, 0
    for plan, _ in plans:
        n, ob = plan.survivors_and_bytes()
        nnz_tot += n
        out_bytes += ob

    # kernel times: the same steps through the measurement build (same kernels), every launch
    # stamped at its start and end by its own dispatch
    iplans = make_plans(gs.instr_lib())
    step(iplans)
    torch.cuda.synchronize()
    for (a, _), (b, _) in zip(plans, iplans):
        assert torch.equal(a.lam, b.lam) and torch.equal(a.nnz, b.nnz), "the two builds disagree"
    reps = args.steps
    prof = gs.KernelProfiler(reps * len(iplans) * 16)
    torch.cuda.synchronize()
    for _ in range(reps):
        step(iplans)
    ktimes = prof.read()
    prof.close()
    del iplans
    kernels = {}
    for name in _class_order():
        ms, n = ktimes[name]
        if n:
            kernels[name] = {"us_per_step": 1e3 * ms / reps, "launches_per_step": n / reps,
                             "avg_us": 1e3 * ms / n}
    kernel_us_per_step = sum(v["us_per_step"] for v in kernels.values())
    # survivors are identical in every step (same seeds), so per-step bytes are exact
    elements_per_step = n_elems * len(plans)
    ms_per_step = elapsed * 1e3 / args.steps
    value = elements_per_step / (elapsed / args.steps)
    alg_bytes_per_step = 4.0 * elements_per_step + out_bytes
    # the roofline kernel: the sampling / compaction pass (or the probabilities pass), whose
    # algorithmic bytes are the whole step's (g read once, the output written once)
    rk = "k_probs" if args.probs else "k_sample"
    rk_ms, rk_n = ktimes[rk]
    avg_launch_ms = rk_ms / max(rk_n, 1)
    alg_per_launch = alg_bytes_per_step / len(plans)
    achieved = alg_per_launch / (avg_launch_ms * 1e-3) / 1e9
    default_cells = args.solver is None and args.rho is None and not (args.hybrid or args.per_layer or args.probs)
    traffic = traffic_for(wl.name, rk) if default_cells else None
    entry = ("probabilities p = min(lambda |g|, 1)" if args.probs else
             ("hybrid coding Q_A (index, value) + Q_B (index | sign)" + (" + dense ternary vector" if args.dense_q
                                                                        else "")) if args.hybrid
             else "ascending (int32 index, fp32 value) pairs")
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
        "config": {"workload": wl.name + ("_per_layer" if args.per_layer else ""), "rows": rows, "d": d,
                   "solvers": solvers, "rho": rhos, "greedy_iters": wl.iters, "calls_per_step": len(plans),
                   "seeds": ("per-layer Philox keys 4000+layer" if args.per_layer else
                             "per-row Philox keys " + ("1000+r" if args.workload == "c2" else str(wl.seeds[0]))),
                   "parallelism": ("single GPU, 54 layers (rows: segments, d: the longest) in one segmented call"
                                   if args.per_layer else "single GPU, rows batched in one call"),
                   "output": entry},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": rk + (" (probabilities: 4 B read + 4 B written per coordinate)" if args.probs else
                                     " (Philox sampling, amplification, " +
                                     ("hybrid Q_A / Q_B coding" if args.hybrid else "compaction") +
                                     "; 4 B read per coordinate + the output)"),
                     "algorithmic_bytes_per_launch": alg_per_launch,
                     "avg_launch_ms": avg_launch_ms, "launches": rk_n,
                     "timing": "HIP start/stop events stamped by each launch's dispatch (hipExtLaunchKernelGGL), "
                               "measurement build, averaged over the launches of %d steps" % reps},
    }
    # the whole path: algorithmic bytes (g read once, the output written once) over the step time
    # and over the summed kernel time, and, when the counter summary matches this kernel source,
    # the bytes the kernels actually moved
    path = {"algorithmic_bytes_per_step": alg_bytes_per_step,
            "algorithmic_GBps": alg_bytes_per_step / (ms_per_step * 1e-3) / 1e9,
            "kernel_us_per_step": kernel_us_per_step}
    path["algorithmic_frac"] = path["algorithmic_GBps"] / HBM_PEAK_GBS
    path["algorithmic_frac_kernel_time"] = alg_bytes_per_step / (kernel_us_per_step * 1e-6) / 1e9 / HBM_PEAK_GBS
    if default_cells:
        per_kernel = {k: traffic_for(wl.name, k) for k in kernels}
        if all(v is not None for v in per_kernel.values()):
            moved = sum(per_kernel[k] * kernels[k]["launches_per_step"] for k in kernels)
            path["measured_bytes_per_step"] = moved
            path["measured_GBps"] = moved / (ms_per_step * 1e-3) / 1e9
            path["measured_frac"] = path["measured_GBps"] / HBM_PEAK_GBS
            path["measured_GBps_kernel_time"] = moved / (kernel_us_per_step * 1e-6) / 1e9
            path["measured_frac_kernel_time"] = path["measured_GBps_kernel_time"] / HBM_PEAK_GBS
    line["path"] = path
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, combos, args.cpu_seconds, per_layer=args.per_layer and not args.probs,
                                            probs=args.probs)
    line["kernels"] = kernels
    line["nnz_per_step"] = nnz_tot
    line["src_sha"] = src_hash()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
