"""Calibrates the cost model's constants on the current device with libmist.

Mist takes compute times from an operator database benchmarked on the target hardware
(Sec. 5.2.1) and fits the slowdown factors of its interference model to benchmarked co-runs of
computation and communication kernels (Sec. 5.2.2).  This script runs both on one MI355X:

1. the operator database for one workload's model: the efficiency of one layer's forward
   GEMMs per microbatch size (mist_measure_eta), which replaces the efficiency formula;
2. the co-run benchmark over a few shapes (mist_corun_measure) and the least-squares factors
   (mist_fit_phi);
3. a check of the fitted model on co-runs it was not fitted on: every stream given a different
   amount of work, all four starting together; the measured time until the last one ends is
   compared with Algorithm 1's prediction (mist_interference) from the streams' solo times.

It writes one JSON file with the measurements and a ready hardware sample ("hw": eta_max = 0
with the measured table, the fitted factors, the measured host link rate, the device memory).
One device cannot exercise a GPU-GPU link: that stream is a copy kernel on a few workgroups
(the footprint of a collective's kernel), and link_bw keeps the nominal value given on the
command line.

    python -m paper_2503_19050_amd.calibrate --workload gpt2.7b-d16 --out calib.json
"""
from __future__ import annotations

import os

# One hardware queue per benchmark stream: a stream that shares a queue with another would
# wait behind it.  HIP reads this when it starts, so it is set before anything loads HIP.
os.environ.setdefault("GPU_MAX_HW_QUEUES", "8")

import argparse  # noqa: E402
import datetime  # noqa: E402
import json  # noqa: E402
import sys  # noqa: E402

import numpy as np  # noqa: E402

from paper_2503_19050_amd import mist  # noqa: E402
from paper_2503_19050_amd import workloads as W  # noqa: E402

MI355X_BF16_DENSE = 2.5e15   # FLOP/s, dense bf16 matrix peak
MI355X_XGMI_LINK = 153e9     # bytes/s per xGMI link and direction (nominal, not measured here)

SHAPES = [
    # (GEMM m, n, k, bytes per copy unit): transformer-sized GEMMs and transfer chunks
    (4096, 4096, 4096, 64 << 20),
    (8192, 8192, 8192, 256 << 20),
    (16384, 8192, 4096, 128 << 20),
]


def corun_shapes():
    return [{"gemm_m": m, "gemm_n": n, "gemm_k": k, "g2g_bytes": b, "h2d_bytes": b, "d2h_bytes": b}
            for m, n, k, b in SHAPES]


def validate(C, shapes, samples, phi, rng, n_runs):
    """Held-out co-runs: all four streams with different unit counts; measured makespan against
    Algorithm 1 on the solo times."""
    solo = {}
    for x in samples:
        solo[(x["shape"], x["stream"])] = x["solo_s"]
    out = []
    for r in range(n_runs):
        k = int(rng.integers(0, len(shapes)))
        s = [solo[(k, j)] for j in range(4)]
        # aim each stream at a random share of 10-60 ms of solo work
        units = [int(np.clip(round(rng.uniform(0.01, 0.06) / s[j]), 1, mist.CORUN_MAX_UNITS)) for j in range(4)]
        t = C.run(15, shapes[k], units)
        measured = max(t[j][-1] for j in range(4)) - min(t[j][0] for j in range(4))
        x = [units[j] * s[j] for j in range(4)]
        pred = mist.interference(phi, x)
        out.append({"shape": k, "units": units, "solo_work_s": x, "measured_s": measured, "predicted_s": pred,
                    "rel_err": (pred - measured) / measured,
                    "no_interference_rel_err": (max(x) - measured) / measured})
        print("  check %d: shape %d units %s measured %.2f ms predicted %.2f ms (%.1f %%), max-of-streams %.2f ms"
              % (r, k, units, 1e3 * measured, 1e3 * pred, 100 * (pred - measured) / measured, 1e3 * max(x)),
              flush=True)
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="gpt2.7b-d16", choices=W.WORKLOADS + ["tiny", "tiny_llama"])
    ap.add_argument("--tp", type=int, default=1)
    ap.add_argument("--peak", type=float, default=MI355X_BF16_DENSE)
    ap.add_argument("--link", type=float, default=MI355X_XGMI_LINK)
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--target", type=float, default=0.02, help="seconds of work per stream and co-run")
    ap.add_argument("--g2g-blocks", type=int, default=16)
    ap.add_argument("--checks", type=int, default=12)
    ap.add_argument("--out", required=True)
    args = ap.parse_args()

    import torch
    if not torch.cuda.is_available():
        print("calibration needs a GPU", file=sys.stderr)
        return 2
    prop = torch.cuda.get_device_properties(0)
    wl = W.workload(args.workload)
    model, mb = wl["model"], wl["space"]["mb"]

    print("operator database: %s, TP %d, microbatches %s" % (args.workload, args.tp, mb), flush=True)
    eta, sec = mist.measure_eta(model, mb, args.tp, args.peak, args.reps)
    for b, e, s in zip(mb, eta, sec):
        print("  b=%-3d eta %.3f  (%.3f ms per layer forward GEMMs)" % (b, e, 1e3 * s), flush=True)

    shapes = corun_shapes()
    big = {k: max(s[k] for s in shapes) for k in shapes[0]}
    print("co-run benchmark: %d shapes, %.0f ms per stream" % (len(shapes), 1e3 * args.target), flush=True)
    with mist.Corun(big, g2g_blocks=args.g2g_blocks) as C:
        samples = C.measure(shapes, target_s=args.target)
        phi = mist.fit_phi(samples)
        for mask in range(3, 16):
            if bin(mask).count("1") >= 2:
                print("  phi[%2d] = %s" % (mask, np.array2string(phi[mask], precision=3)), flush=True)
        rng = np.random.default_rng(0)
        checks = validate(C, shapes, samples, phi, rng, args.checks)

    h2d = [s["h2d_bytes"] / x["solo_s"] for x in samples for i, s in enumerate(shapes)
           if x["shape"] == i and x["stream"] == 2]
    d2h = [s["d2h_bytes"] / x["solo_s"] for x in samples for i, s in enumerate(shapes)
           if x["shape"] == i and x["stream"] == 3]
    pcie = float(min(np.median(h2d), np.median(d2h)))
    err = np.array([c["rel_err"] for c in checks])
    err0 = np.array([c["no_interference_rel_err"] for c in checks])
    print("model check: mean |error| %.1f %% (max %.1f %%); without interference %.1f %%"
          % (100 * np.abs(err).mean(), 100 * np.abs(err).max(), 100 * np.abs(err0).mean()), flush=True)

    out = {
        "what": "libmist calibration: operator efficiency per microbatch and fitted slowdown factors",
        "date": datetime.datetime.now(datetime.timezone.utc).isoformat(timespec="seconds"),
        "command": "python -m paper_2503_19050_amd.calibrate " + " ".join(sys.argv[1:]),
        "device": {"name": prop.name, "arch": getattr(prop, "gcnArchName", ""), "cus": prop.multi_processor_count,
                   "memory_bytes": prop.total_memory},
        "workload": args.workload, "model": model, "tp": args.tp, "peak_flops": args.peak,
        "eta": {"mb": list(mb), "eta": eta.tolist(), "seconds": sec.tolist()},
        "corun": {"g2g_blocks": args.g2g_blocks, "target_s": args.target, "shapes": shapes, "samples": samples},
        "phi": phi.tolist(),
        "pcie": {"h2d_bytes_per_s": float(np.median(h2d)), "d2h_bytes_per_s": float(np.median(d2h))},
        "check": {"runs": checks, "mean_abs_rel_err": float(np.abs(err).mean()),
                  "max_abs_rel_err": float(np.abs(err).max()),
                  "mean_abs_rel_err_without_interference": float(np.abs(err0).mean())},
        "hw": {"flops": args.peak, "mem_bytes": float(prop.total_memory), "pcie_bw": pcie, "link_bw": args.link,
               "eta_max": 0.0, "n_half": 0.0, "eta_tab": eta.tolist(), "phi": phi.tolist()},
    }
    with open(args.out, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", args.out, flush=True)
    return 0


def hw_from_calibration(path: str) -> dict:
    """The hardware sample a calibration file holds (for a workload's "hws" list; its efficiency
    table belongs to the model and microbatch list it was measured for)."""
    with open(path) as f:
        return json.load(f)["hw"]


if __name__ == "__main__":
    sys.exit(main())
