"""Pins of the oracle's weight-sampled argmin (Eq. 4 with sampled alpha): per group and sample,
the feasible configuration minimising alpha*G*t + (1-alpha)*d, lowest id on ties.

The expected values are recomputed here from the oracle's per-configuration dump (t, d, mem,
bucket) with exact rational arithmetic for the fused multiply-add (fractions.Fraction, then one
correctly rounded conversion), independently of the oracle's reduction loop; the special
weights 0, 1/2 and 1 are pinned against d, the tuner's own objective and t.
"""

from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

ALPHAS = [0.0, 0.125, 0.3, 0.5, 0.9, 1.0]


def _fma(a, b, c):
    return float(Fraction(a) * Fraction(b) + Fraction(c))


def _cases():
    tight = W.workload("tiny")
    tight["hws"][0]["mem_bytes"] = 3.0e7          # most groups infeasible
    return [W.workload("tiny"), W.workload("tiny_llama"), tight]


@pytest.mark.parametrize("wl", _cases(), ids=["tiny", "tiny_llama", "tight"])
def test_alpha_argmin_matches_brute_force(wl):
    o = O.Oracle(wl)
    res = o.run_alpha(ALPHAS)
    keys = o.group_keys()
    dump = o.dump(0, o.n_groups)
    rng = np.random.default_rng(5)
    # every group for the first sample, a few groups for the rest (rational arithmetic is slow)
    checked = 0
    for gi, key in enumerate(keys):
        rows = dump[key["base"]:key["base"] + key["size"]]
        ids = key["base"] + np.arange(key["size"], dtype=np.uint64)
        feas = np.nonzero(rows[:, 4] >= 0)[0]
        for a, alpha in enumerate(ALPHAS):
            if a > 0 and rng.random() > 0.15:
                continue
            if len(feas) == 0:
                assert res["id"][gi, a] == O.NONE and res["obj"][gi, a] == np.inf
                continue
            aG = alpha * float(key["G"])
            beta = 1.0 - alpha
            v = np.array([_fma(aG, rows[k, 0], beta * rows[k, 1]) for k in feas])
            k = feas[np.lexsort((ids[feas], v))[0]]
            assert res["id"][gi, a] == ids[k], (gi, alpha)
            assert res["obj"][gi, a] == v[np.searchsorted(feas, k)], (gi, alpha)
            checked += 1
    assert checked > 0


@pytest.mark.parametrize("name", ["tiny", "tiny_llama"])
def test_special_weights(name):
    """alpha = 1/2 halves the tuner's objective fma(G, t, d) exactly (scaling by 2^-1 commutes
    with rounding), so its argmin is the group's best; alpha = 1 ranks by t, alpha = 0 by d."""
    o = O.Oracle(W.workload(name))
    res = o.run_alpha([0.5, 1.0, 0.0])
    best = o.run()
    assert np.array_equal(res["id"][:, 0], best["best_id"])
    feasible = best["best_id"] != O.NONE
    assert np.array_equal(res["obj"][feasible, 0], 0.5 * best["best_obj"][feasible])
    keys = o.group_keys()
    dump = o.dump(0, o.n_groups)
    for gi, key in enumerate(keys):
        rows = dump[key["base"]:key["base"] + key["size"]]
        ids = key["base"] + np.arange(key["size"], dtype=np.uint64)
        feas = np.nonzero(rows[:, 4] >= 0)[0]
        if len(feas) == 0:
            continue
        kt = feas[np.lexsort((ids[feas], rows[feas, 0]))[0]]   # least t (G is fixed in a group)
        kd = feas[np.lexsort((ids[feas], rows[feas, 1]))[0]]   # least d
        assert res["id"][gi, 1] == ids[kt]
        assert res["obj"][gi, 1] == float(key["G"]) * rows[kt, 0]
        assert res["id"][gi, 2] == ids[kd] and res["obj"][gi, 2] == rows[kd, 1]


def test_weights_validated():
    o = O.Oracle(W.workload("tiny"))
    for bad in ([], [1.5], [-0.1], [float("nan")], [0.5] * 17):
        with pytest.raises(ValueError):
            o.run_alpha(bad)
