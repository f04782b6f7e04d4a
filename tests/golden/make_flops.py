"""Writes flops_per_config.json: FP64 operations of the cost-model definition per
configuration, counted by the oracle's counting build (add/sub/mul 1, fma 2,
min/max/compare 0) with each loop level counted once per combination of its digits.

c1 and c2 are counted over every group; c3-c5 over every 16th group (the count per
configuration depends on the data only through Algorithm 1's pattern changes).

Run: python tests/golden/make_flops.py   (calls only oracle/)
"""

import json
import os
import sys
from concurrent.futures import ProcessPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import oracle as O  # noqa: E402
from paper_2503_19050_amd import workloads as W  # noqa: E402


def _count(args):
    name, g = args
    o = O.Oracle(W.workload(name))
    return o.count_flops(g, g + 1)


def main():
    out = {"cite": "counting build of oracle/mist_oracle.cpp; see the module docstring", "workloads": {}}
    with ProcessPoolExecutor(max_workers=os.cpu_count()) as ex:
        for name in W.WORKLOADS:
            o = O.Oracle(W.workload(name))
            stride = 1 if name in ("c1", "c2") else 16
            groups = list(range(0, o.n_groups, stride))
            res = list(ex.map(_count, [(name, g) for g in groups], chunksize=4))
            flops = sum(r[0] for r in res)
            configs = sum(r[1] for r in res)
            out["workloads"][name] = {"flops_per_config": flops / configs, "groups_counted": len(groups),
                                      "group_stride": stride, "configs_counted": configs}
            print(name, flops / configs, configs, flush=True)
    with open(os.path.join(HERE, "flops_per_config.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
