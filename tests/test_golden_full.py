"""The stored whole-space oracle digests (tests/golden/full_<workload>.npz): their counts match
the oracle's enumeration, and the digest reacts to a change in any word it covers."""

import os
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
sys.path.insert(0, GOLDEN)
from digest import group_digests  # noqa: E402


@pytest.mark.parametrize("name", ["llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
def test_stored_digests_match_the_enumeration(name):
    gold = np.load(os.path.join(GOLDEN, "full_%s.npz" % name))
    o = O.Oracle(W.workload(name))
    assert int(gold["n_groups"]) == o.n_groups
    assert int(gold["n_configs"]) == o.n_configs
    assert int(gold["n_buckets"]) == o.n_buckets
    assert gold["digest"].shape == (o.n_groups,)
    # a group without a feasible configuration has the empty outputs; every other group's
    # outputs name its own ids, so their digests differ
    NB = o.n_buckets
    empty = group_digests(np.full((1, NB), O.NONE, dtype=np.uint64), np.full((1, NB), np.inf),
                          np.zeros(1, dtype=np.uint64), np.full(1, O.NONE, dtype=np.uint64), np.full(1, np.inf))[0]
    rest = gold["digest"][gold["digest"] != empty]
    assert len(rest) > 0 and len(np.unique(rest)) == len(rest)


def test_digest_sees_every_word():
    r = O.Oracle(W.workload("tiny")).run()
    base = group_digests(r["bucket_id"], r["bucket_obj"], r["frontier"], r["best_id"], r["best_obj"])
    g = int(np.argmax(r["frontier"] != 0))
    for key in ["bucket_id", "bucket_obj", "frontier", "best_id", "best_obj"]:
        m = {k: np.array(v, copy=True) for k, v in r.items()}
        a = m[key].view(np.uint64)
        idx = (g, 3) if a.ndim == 2 else (g,)
        a[idx] ^= np.uint64(1)  # one bit of one word
        d = group_digests(m["bucket_id"], m["bucket_obj"], m["frontier"], m["best_id"], m["best_obj"])
        assert d[g] != base[g], key
        assert np.array_equal(np.delete(d, g), np.delete(base, g)), key


def test_stored_plan_points_are_the_oracles():
    """tests/golden/plan_llama13b-d64.npz: every stored point decodes to its group's key and
    carries the oracle's own t and d; every group with PP = 1 or 2 and a feasible configuration
    has at least one point."""
    z = np.load(os.path.join(GOLDEN, "plan_llama13b-d64.npz"))
    wl = W.workload("llama13b-d64")
    wl["space"] = dict(wl["space"], alphas=[float(a) for a in z["alphas"]])
    o = O.Oracle(wl)
    ids = z["id"]
    vals = o.eval_ids(ids)
    assert np.array_equal(vals[:, 0], z["t"]) and np.array_equal(vals[:, 1], z["d"])
    for r in range(0, len(ids), 7):
        c = o.decode(int(ids[r]))
        assert (c["hw"], c["G"], c["PP"], c["k"], c["l"]) == (z["hw"][r], z["G"][r], z["PP"][r], z["k"][r], z["l"][r])
    keys = {(k["hw"], k["G"], k["PP"], k["k"], k["l"]) for k in o.group_keys() if k["PP"] in (1, 2)}
    have = set(zip(z["hw"].tolist(), z["G"].tolist(), z["PP"].tolist(), z["k"].tolist(), z["l"].tolist()))
    assert have <= keys and len(have) > 0.5 * len(keys)
