"""Writes plan_llama13b-d64.npz: the planner's candidate points of llama13b-d64 for plans of one
and two stages, from the oracle alone.  For every group with PP in {1, 2}: the group's best
configuration and the one each weight sample alpha = 0, 1/7, ..., 1 selects (Eq. 4), with the
oracle's t and d of each (Eq. 5-6).  The GPU planner test plans on the library's own points and
compares the plan with the exhaustive search over these.

Run: python tests/golden/make_plan_golden.py   (calls only oracle/; all cores; a few minutes)
"""

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import oracle as O  # noqa: E402
from oracle import plan_oracle as PO  # noqa: E402
from paper_2503_19050_amd import workloads as W  # noqa: E402

NAME = "llama13b-d64"
ALPHAS = [k / 7.0 for k in range(8)]
PPS = (1, 2)


def main():
    t0 = time.time()
    wl = W.workload(NAME)
    wl["space"] = dict(wl["space"], alphas=ALPHAS)
    keys = O.Oracle(wl).group_keys()
    groups = [g for g, k in enumerate(keys) if k["PP"] in PPS]
    per_hw = PO.candidates_groups(wl, ALPHAS, groups, procs=os.cpu_count())
    rows = [(hw, G, PP, k, l, i, t, d) for hw, cand in sorted(per_hw.items())
            for (G, PP, k, l), pts in sorted(cand.items()) for (t, d, i) in pts]
    cols = list(zip(*rows))
    path = os.path.join(HERE, "plan_%s.npz" % NAME)
    np.savez_compressed(path, hw=np.array(cols[0], np.int32), G=np.array(cols[1], np.int32),
                        PP=np.array(cols[2], np.int32), k=np.array(cols[3], np.int32),
                        l=np.array(cols[4], np.int32), id=np.array(cols[5], np.uint64),
                        t=np.array(cols[6], np.float64), d=np.array(cols[7], np.float64),
                        alphas=np.array(ALPHAS), pps=np.array(PPS, np.int32))
    print(NAME, len(groups), "groups", len(rows), "points", "%.0f s" % (time.time() - t0), flush=True)


if __name__ == "__main__":
    main()
