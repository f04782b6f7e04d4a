"""Pins of the oracle's exact (non-bucketed) time-vs-memory frontier: a configuration is on it
when no other feasible configuration with no more memory and no larger objective comes before
it in (mem, obj, id) order.  Checked here by an all-pairs dominance test on the per-configuration
dump (independent of the oracle's sort-and-scan), and against the bucketed staircase and the
group's best."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W


def _cases():
    tight = W.workload("tiny")
    tight["hws"][0]["mem_bytes"] = 3.0e7
    return [W.workload("tiny"), W.workload("tiny_llama"), tight]


@pytest.mark.parametrize("wl", _cases(), ids=["tiny", "tiny_llama", "tight"])
def test_exact_frontier_all_pairs(wl):
    o = O.Oracle(wl)
    keys = o.group_keys()
    dump = o.dump(0, o.n_groups)
    res = o.run()
    rng = np.random.default_rng(2)
    groups = sorted(set(rng.choice(o.n_groups, size=min(12, o.n_groups), replace=False).tolist()) | {0})
    for g in groups:
        k = keys[g]
        rows = dump[k["base"]:k["base"] + k["size"]]
        ids = k["base"] + np.arange(k["size"], dtype=np.uint64)
        feas = rows[:, 4] >= 0
        mem, obj, fid = rows[feas, 2], rows[feas, 3], ids[feas]
        on = np.zeros(len(fid), dtype=bool)
        for i in range(len(fid)):
            before = (mem < mem[i]) | ((mem == mem[i]) & ((obj < obj[i]) | ((obj == obj[i]) & (fid < fid[i]))))
            on[i] = not np.any(before & (obj <= obj[i]))
        want = np.nonzero(on)[0]
        want = want[np.lexsort((fid[want], obj[want], mem[want]))]
        got = o.pareto_exact(g)
        assert np.array_equal(got["id"], fid[want])
        assert np.array_equal(got["mem"], mem[want]) and np.array_equal(got["obj"], obj[want])
        if len(want) == 0:
            assert res["best_id"][g] == O.NONE
            continue
        assert np.all(np.diff(got["mem"]) > 0) and np.all(np.diff(got["obj"]) < 0)
        assert got["obj"][-1] == res["best_obj"][g]
        # every bucket on the bucketed staircase holds an exact frontier point with its objective
        NB = wl["space"]["n_buckets"]
        M = wl["hws"][k["hw"]]["mem_bytes"]
        for j in range(NB):
            if int(res["frontier"][g]) >> j & 1:
                lo = (M * float(j)) / NB if j > 0 else 0.0
                hi = (M * float(j + 1)) / NB if j < NB - 1 else M
                inb = (got["mem"] > lo) & (got["mem"] <= hi)
                assert np.any(inb & (got["obj"] == res["bucket_obj"][g][j]))
