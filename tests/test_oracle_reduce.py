"""Brute-force check of the oracle's reductions (feasible argmin per memory
bucket, overall argmin, bucketed time-vs-memory staircase) on tiny spaces.

The expected values are recomputed here from the oracle's per-configuration
dump with sorting, independently of the oracle's own reduction loop.
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W


def _cases():
    tight = W.workload("tiny")
    tight["hws"][0]["mem_bytes"] = 3.0e7          # most groups infeasible
    loose = W.workload("tiny")
    loose["hws"][0]["mem_bytes"] = 1.0e12         # everything in bucket 0
    one = W.workload("tiny")
    one["space"]["n_buckets"] = 1
    return [W.workload("tiny"), W.workload("tiny_llama"), tight, loose, one]


@pytest.mark.parametrize("wl", _cases(), ids=["tiny", "tiny_llama", "tight", "loose", "nb1"])
def test_reductions_match_brute_force(wl):
    o = O.Oracle(wl)
    NB = wl["space"]["n_buckets"]
    res = o.run()
    keys = o.group_keys()
    dump = o.dump(0, o.n_groups)
    n_feasible_groups = 0
    for gi, key in enumerate(keys):
        rows = dump[key["base"]:key["base"] + key["size"]]
        ids = key["base"] + np.arange(key["size"], dtype=np.uint64)
        mem, obj, bucket = rows[:, 2], rows[:, 3], rows[:, 4].astype(int)
        M = wl["hws"][key["hw"]]["mem_bytes"]
        # feasibility is the Eq. 4 constraint
        assert np.array_equal(bucket >= 0, mem <= M)
        # bucket j holds memory in (E_{j-1}, E_j], E_j = M (j+1) / NB
        NBf = float(NB)
        for j in np.unique(bucket[bucket >= 0]):
            lo = (M * float(j)) / NBf if j > 0 else 0.0
            hi = (M * float(j + 1)) / NBf if j < NB - 1 else M
            sel = mem[bucket == j]
            assert np.all(sel <= hi) and np.all(sel > lo)
        # bucket edges are increasing: more memory never lands in a lower bucket
        order = np.argsort(mem, kind="stable")
        fb = bucket[order][mem[order] <= M]
        assert np.all(np.diff(fb) >= 0)
        want_bid = np.full(NB, O.NONE, dtype=np.uint64)
        want_bobj = np.full(NB, np.inf)
        for j in range(NB):
            sel = np.nonzero(bucket == j)[0]
            if len(sel):
                k = sel[np.lexsort((ids[sel], obj[sel]))[0]]
                want_bid[j], want_bobj[j] = ids[k], obj[k]
        assert np.array_equal(res["bucket_id"][gi], want_bid)
        assert np.array_equal(res["bucket_obj"][gi], want_bobj)
        feas = np.nonzero(bucket >= 0)[0]
        if len(feas):
            n_feasible_groups += 1
            k = feas[np.lexsort((ids[feas], obj[feas]))[0]]
            assert res["best_id"][gi] == ids[k] and res["best_obj"][gi] == obj[k]
        else:
            assert res["best_id"][gi] == O.NONE and res["best_obj"][gi] == np.inf
        # staircase: a bucket is kept when it beats every lower bucket strictly
        mask = 0
        for j in range(NB):
            lower = want_bobj[:j]
            if want_bid[j] != O.NONE and (len(lower) == 0 or want_bobj[j] < lower.min()):
                mask |= 1 << j
        assert int(res["frontier"][gi]) == mask
    assert n_feasible_groups > 0
