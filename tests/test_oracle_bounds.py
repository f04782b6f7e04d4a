"""The lower bound the exact frontier's candidate pass relies on, checked on the oracle (CPU).

With every slowdown factor at least 1 (the host rejects smaller ones), a stream's standalone time
falls in each round of Algorithm 1 (Sec. 5.2.2) by at most the round's length, so the returned time
is at least every stream's own time (up to rounding); hence a configuration's objective G t + (T1 - t) (Eq. 4-6) is
at least (G - 1) t + max(H2D, D2H) of its first microbatch.  The candidate pass compares that bound,
lowered by a relative 2^-30, with its bucket's threshold; these tests check that the computed values
keep the bound by a wide margin: on random stream vectors with random factor tables (up to 50, far
above the seeded ones, with absent and tiny streams), and on every configuration of small spaces.
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

MARGIN = 1.0 - 2.0 ** -30   # the candidate pass's relative margin


def _random_phi(rng, top):
    phi = 1.0 + (top - 1.0) * rng.random((16, 4)) ** 3
    for m in range(16):            # single-stream and empty patterns carry no slowdown
        if bin(m).count("1") < 2:
            phi[m] = 1.0
    return phi


@pytest.mark.parametrize("top", [1.0, 1.5, 50.0])
def test_interference_is_at_least_every_stream(top):
    rng = np.random.default_rng(int(top * 10))
    for _ in range(3000):
        phi = _random_phi(rng, top)
        X = rng.random(4) * 10.0 ** rng.integers(-6, 3, size=4)
        X[rng.random(4) < 0.25] = 0.0   # absent streams
        T = O.interference(X, phi)
        # In real arithmetic T >= max X; rounding can leave T an ulp or so below it, far inside
        # the pass's margin.
        assert T * (1.0 + 2.0 ** -40) >= X.max(), (X.tolist(), T)


def test_interference_bound_is_tight_without_slowdown():
    """With all factors 1 the streams overlap perfectly: the time is exactly the longest one
    (the bound cannot be raised in general)."""
    rng = np.random.default_rng(5)
    phi = np.ones((16, 4))
    for _ in range(500):
        X = rng.random(4)
        assert O.interference(X, phi) == X.max()


@pytest.mark.parametrize("name, mod", [("tiny", None), ("tiny_llama", None), ("tiny", "large"), ("gpt1.3b-d8", None)])
def test_objective_bound_on_every_configuration(name, mod):
    wl = W.workload(name)
    if mod == "large":
        rng = np.random.default_rng(3)
        for h in wl["hws"]:
            h["phi"] = [[float(x) for x in row] for row in _random_phi(rng, 50.0)]
    o = O.Oracle(wl)
    keys = o.group_keys()
    n = min(o.n_configs, 4000)
    ids = np.unique(np.linspace(0, o.n_configs - 1, n).astype(np.uint64))
    bases = np.array([k["base"] for k in keys], dtype=np.uint64)
    for cid in ids:
        t = o.terms(int(cid))
        G = keys[int(np.searchsorted(bases, cid, side="right")) - 1]["G"]
        first = max(t["C"], t["G2Gf"], t["H2Df"], t["D2Hf"])
        assert t["T1"] * (1.0 + 2.0 ** -40) >= first, (int(cid), t["T1"], first)
        assert t["t"] * (1.0 + 2.0 ** -40) >= max(t["C"], t["G2Gs"], t["H2Ds"], t["D2Hs"]), int(cid)
        lb = ((G - 1) * t["t"] + max(t["H2Df"], t["D2Hf"])) * MARGIN
        assert t["obj"] >= lb, (int(cid), t["obj"], lb)
