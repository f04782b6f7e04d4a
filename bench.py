"""Benchmark of the tuner's hot path on one MI355X: configurations evaluated per second
(cost model + feasibility filter + per-bucket and per-group reductions) and the FP64
vector roofline fraction of the evaluation kernel.

One step = one mist_eval_space over the whole space of the workload (default llama42b-d128-hw64:
Llama L60 h8192 GQA-8, D=128, 64 hardware samples in one launch, 29,939,155,200 configurations,
66,496 groups, the largest workload), inputs resident on the GPU.
Prints one JSON line; its "alpha_frontier" field times the same space with weight samples of
Eq. 4 added (the per-group (t, d) argmins), and its "exact_frontier" field the exact
(unbucketed) time-vs-memory staircase of every group on the evaluated space.  The CPU baseline is the plain oracle timed on this host over a
bounded, seeded sample of the same workload's groups.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "candidate configs evaluated/sec (eval+filter+reduce); % of FP64 vector peak"
FP64_VECTOR_PEAK_TFLOPS = 78.6   # 256 CUs x 128 FP64 FLOP/clk (64 FMA lanes) x 2.4 GHz
# VALU issue: 256 CUs x 4 SIMDs, one wave64 VALU instruction per SIMD every 4 clocks at 2.4 GHz
VALU_ISSUE_PEAK = 256 * 4 * 2.4e9 / 4
FLOPS_FILE = os.path.join(ROOT, "tests", "golden", "flops_per_config.json")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2503_19050_amd", "csrc", "mist_kernels.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def flops_per_config(name: str):
    """(FP64 operations of the definition per configuration with every level shared among the
    configurations below it, as the oracle's nested loops evaluate it: the algorithmic unit; the
    same for one configuration evaluated on its own, every level repeated)."""
    try:
        with open(FLOPS_FILE) as f:
            w = json.load(f)["workloads"][name]
            return w["flops_per_config_shared_levels"], w["flops_per_config"]
    except (OSError, KeyError, ValueError):
        return None, None


def counter_record(name: str, field: str = "executed_fp64_per_config"):
    """A per-configuration figure of the evaluation kernel from the committed rocprofv3
    instruction counters, if they were taken on the current kernel source:
    executed_fp64_per_config = 64 x (ADD + MUL + TRANS + 2 FMA) F64 wave instructions per
    configuration, valu_per_config = 64 x SQ_INSTS_VALU per configuration."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)[name]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("kernel_sha") != kernel_hash():
        return None
    return rec.get(field)


def traffic_record(name: str, n_launch_configs: int):
    """HBM bytes per evaluation launch from the committed rocprofv3 counter runs, if they
    were taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)[name]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("kernel_sha") != kernel_hash():
        return None
    return rec.get("bytes_per_launch")


def _oracle_for(wl: dict, seconds: float, shard: int, n_shards: int):
    """The oracle over this shard's share of the groups (a seeded random order dealt round robin)
    until about ``seconds`` of work: (groups, configurations, seconds)."""
    import numpy as np
    from oracle import oracle as O

    o = O.Oracle(wl)
    order = np.random.default_rng(2025).permutation(o.n_groups)[shard::n_shards]
    keys = o.group_keys()
    done = configs = 0
    t0 = time.perf_counter()
    for g in order:
        o.run(int(g), int(g) + 1)
        done += 1
        configs += keys[int(g)]["size"]
        if time.perf_counter() - t0 >= seconds:
            break
    return done, configs, time.perf_counter() - t0, o.n_groups


def _oracle_shard(job):
    return _oracle_for(*job)


def host_cpu() -> dict:
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count() or 1
    return {"cpu_model": model, "nproc": usable, "cpu_count": os.cpu_count()}


def cpu_baseline(wl: dict, seconds: float, shards: int) -> dict:
    """The oracle as it stands: one process (one thread) over seeded random groups until about
    ``seconds`` of work; then, when ``shards`` > 1, that many single-threaded processes over
    disjoint groups for the same time, as the parity runs over the large workloads use it."""
    done, configs, dt, n_groups = _oracle_for(wl, seconds, 0, 1)
    host = host_cpu()
    rec = {
        "value": configs / dt, "unit": "configs/s", "cores": 1, "kind": "oracle",
        "sample": "%d of %d groups of %s in seeded random order, %d configs, %.1f s" % (
            done, n_groups, wl["name"], configs, dt),
        **host,
    }
    if shards > 1:
        import multiprocessing as mp
        with mp.get_context("spawn").Pool(shards) as pool:
            parts = pool.map(_oracle_shard, [(wl, seconds, i, shards) for i in range(shards)], chunksize=1)
        total = sum(p[1] for p in parts)
        wall = max(p[2] for p in parts)
        rec["sharded"] = {"value": total / wall, "unit": "configs/s", "processes": shards,
                          "sample": "%d groups, %d configs over %d single-threaded oracle processes, "
                                    "%.1f s" % (sum(p[0] for p in parts), total, shards, wall)}
    return rec


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llama42b-d128-hw64",
                    choices=["gpt1.3b-d8", "gpt2.7b-d16", "llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--cpu-shards", type=int, default=0,
                    help="single-threaded oracle processes of the sharded CPU baseline (0: the usable "
                         "CPUs, at most 16; 1: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--alphas", type=int, default=8,
                    help="after the headline run, also time the space with this many weight samples of "
                         "Eq. 4 (alpha = k/(n-1)); 0 skips it")
    ap.add_argument("--exact-runs", type=int, default=10,
                    help="after the headline run, time this many exact (non-bucketed) frontier passes "
                         "(mist_eval_pareto_exact) on the evaluated space; 0 skips them")
    ap.add_argument("--probe-fp64", action="store_true",
                    help="instead of the benchmark, run the FP64 instruction-mix probe (one kernel per "
                         "instruction kind with a known count, for reading the profiler's FP64 counters) "
                         "and print the expected counts")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="after the timed region, copy a buffer of this many MiB on the device "
                         "(a plain copy kernel of known size, to scale the HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the evaluation of one space runs on a single device "
              "(sharding the groups over several GPUs needs no exchange and is not run here)", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2503_19050_amd import mist
    from paper_2503_19050_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.probe_fp64:
        n_threads, reps = 256 * 1024, 64
        want = {}
        for kind in mist.PROBE_KINDS:
            want[kind] = mist.probe_fp64(kind, n_threads, reps)
        print(json.dumps({"probe": "fp64 instruction mix", "kernel": "k_probe<kind>",
                          "kinds": mist.PROBE_KINDS, "wave_instructions_per_dispatch": want}))
        return 0
    props = torch.cuda.get_device_properties(0)
    wl = W.workload(args.workload)

    t0 = time.perf_counter()
    S = mist.from_workload(wl)
    torch.cuda.synchronize()
    build_ms = (time.perf_counter() - t0) * 1e3
    info = S.launch_info()
    log("workload", wl["name"], S.n_configs, "configs", S.n_groups, "groups", info)

    for _ in range(args.warmup):
        S.eval()
    torch.cuda.synchronize()

    S.set_timing(True)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        S.eval()
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    k1_ms, k2_ms, n = S.read_timing()
    assert n == args.steps
    S.set_timing(False)

    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib * (1 << 20) // 8
        src = torch.ones(n, dtype=torch.float64, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    t0 = time.perf_counter()
    best = S.best_array()
    extract_ms = (time.perf_counter() - t0) * 1e3
    feasible = int(np.count_nonzero(best["id"] != np.uint64(mist.MIST_NONE)))

    ms_per_step = total_ms / args.steps
    value = S.n_configs / (ms_per_step / 1e3)
    k1_avg = k1_ms / n
    k2_avg = k2_ms / n
    fpc, fscratch = flops_per_config(wl["name"])
    roofline = None
    if fpc is not None:
        # Algorithmic FLOPs: the definition's FP64 operations as the oracle's nested loops
        # perform them (each level once per combination of the digits it depends on).
        achieved = fpc * S.n_configs / (k1_avg / 1e3) / 1e12
        traffic = traffic_record(wl["name"], S.n_configs)
        roofline = {"bound": "alu", "achieved": achieved, "peak": FP64_VECTOR_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": achieved / FP64_VECTOR_PEAK_TFLOPS, "traffic": traffic,
                    "kernel": "k_eval", "flops_per_config": fpc,
                    "flops_unit": "FP64 operations of the cost model per configuration with every loop level "
                                  "shared, as the oracle evaluates it (fma = 2)",
                    # Labelled extras: the count of the same definition with every level repeated
                    # per configuration (work neither the oracle nor the kernel does, so no
                    # fraction of peak is formed from it), and what the kernel executes by the
                    # instruction counters.
                    "flops_per_config_from_scratch": fscratch}
        executed = counter_record(wl["name"])
        if executed is not None:
            roofline["executed_fp64_per_config"] = executed
            roofline["frac_executed"] = executed * S.n_configs / (k1_avg / 1e3) / 1e12 / FP64_VECTOR_PEAK_TFLOPS
        valu = counter_record(wl["name"], "valu_per_config")
        if valu is not None:
            # The issue limit the kernel meets: executed wave64 VALU instructions per second
            # against the chip's issue rate.
            roofline["valu_per_config"] = valu
            roofline["valu_issue_frac"] = valu * S.n_configs / 64 / (k1_avg / 1e3) / VALU_ISSUE_PEAK

    exact = None
    if args.exact_runs > 0:
        S.eval_pareto_exact()   # first pass allocates the candidate buffers
        torch.cuda.synchronize()
        runs = []
        for _ in range(args.exact_runs):
            t0 = time.perf_counter()
            S.eval_pareto_exact()
            torch.cuda.synchronize()
            runs.append((time.perf_counter() - t0) * 1e3)
        runs.sort()
        ms = runs[len(runs) // 2]
        # The row's rate: configurations of the space per second of the whole pass.  Tiles that
        # cannot hold a candidate are skipped, so it is not an evaluation rate and no FP64 peak
        # fraction is derived from it.
        exact = {"ms_per_run": ms, "runs": len(runs), "value": S.n_configs / (ms / 1e3), "unit": "configs/s",
                 **S.exact_info(),
                 "what": "exact time-vs-memory frontier of every group after the evaluation: candidate filter, "
                         "live tiles, one candidate pass of the evaluation kernel over them (candidates past a tile's window go to an "
                         "overflow pool; a tile with a candidate that finds no place in either is evaluated again), exact "
                         "pre-filter, segmented sort by memory, scan; host "
                         "wall time including its one synchronisation"}

    alpha = None
    if args.alphas > 0:
        A = args.alphas
        wa = dict(wl)
        wa["space"] = dict(wl["space"], alphas=[k / (A - 1) if A > 1 else 0.5 for k in range(A)])
        SA = mist.from_workload(wa)
        for _ in range(args.warmup):
            SA.eval()
        torch.cuda.synchronize()
        SA.set_timing(True)
        start.record()
        for _ in range(args.steps):
            SA.eval()
        end.record()
        torch.cuda.synchronize()
        a_total = start.elapsed_time(end)
        a_k1, a_k2, a_n = SA.read_timing()
        SA.set_timing(False)
        a_fpc = None if fpc is None else fpc + 3.0 * A   # + per sample: (1-alpha)*d and one fma (shared levels)
        a_k1_avg = a_k1 / a_n
        alpha = {"n_alphas": A, "value": S.n_configs / (a_total / args.steps / 1e3), "unit": "configs/s",
                 "ms_per_step": a_total / args.steps, "eval_kernel_ms": a_k1_avg, "reduce_kernel_ms": a_k2 / a_n,
                 "flops_per_config": a_fpc,
                 "frac": None if a_fpc is None else a_fpc * S.n_configs / (a_k1_avg / 1e3) / 1e12 / FP64_VECTOR_PEAK_TFLOPS}
        SA.close()

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline: oracle for about %.0f s" % args.cpu_seconds)
        shards = args.cpu_shards or min(16, host_cpu()["nproc"])
        cpu = cpu_baseline(wl, args.cpu_seconds, shards)

    rec = {
        "metric": METRIC, "value": value, "unit": "configs/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "%s: %s" % (wl["name"], wl["desc"]), "configs": S.n_configs,
                   "groups": S.n_groups, "buckets": S.n_buckets, "tiles": info["tiles"],
                   "block": info["block"], "strips_per_tile": info["strips_per_tile"]},
        "eval_kernel_ms": k1_avg, "reduce_kernel_ms": k2_avg, "space_build_ms": build_ms,
        "extract_best_ms": extract_ms, "feasible_groups": feasible,
        "device": {"name": props.name, "cus": props.multi_processor_count,
                   "arch": getattr(props, "gcnArchName", "")},
        "roofline": roofline, "cpu_baseline": cpu, "alpha_frontier": alpha, "exact_frontier": exact,
    }
    S.close()
    print(json.dumps(rec))
    return 0


if __name__ == "__main__":
    sys.exit(main())
