"""The inter-stage planner (Eq. 1-3) of libmist against the exhaustive planner of the oracle
(oracle/plan_oracle.py), on the host: seeded random candidate sets (missing groups, negative
deltas, repeated points, stage times that tie in real arithmetic but round apart) and the
oracle's own frontier points of the tiny spaces.  The optimum value is unique; the plan attaining
it is checked for validity (several plans may tie).  The planner minimises Eq. 2 in its suffix
form exactly (bit for bit against the exhaustive search in that form); its stage-order value is
within 1e-12 of the exhaustive stage-order minimum."""

import numpy as np
import pytest

from oracle import plan_oracle as PO
from paper_2503_19050_amd import mist
from paper_2503_19050_amd import workloads as W


def _check(plan, cand, n_layers, pp, want):
    if want is None:
        assert plan is None
        return
    assert plan is not None
    assert abs(plan["F"] - want[0]) <= 1e-12 * abs(want[0])
    G, PP = plan["G"], plan["PP"]
    assert (pp == 0 or PP == pp) and len(plan["stages"]) == PP
    assert sum(st["l"] for st in plan["stages"]) == n_layers
    for i, st in enumerate(plan["stages"]):
        assert st["k"] == PP - i
        assert (st["t"], st["d"], st["id"]) in cand[(G, PP, PP - i, st["l"])]
    # the reported value is Eq. 2 of the plan's own points, in stage order
    ts, ds = [st["t"] for st in plan["stages"]], [st["d"] for st in plan["stages"]]
    assert plan["F"] == PO.plan_value(G, ts, ds)
    # the plan is the exact minimum of the suffix form, the one the planner prunes in
    want_s = PO.best_plan(cand, n_layers, pp, value=PO.plan_value_suffix)
    assert PO.plan_value_suffix(G, ts, ds) == want_s[0]


def _random_instance(rng):
    L = int(rng.integers(1, 8))
    cand = {}
    nid = 0
    pool = [(float(rng.uniform(0.1, 2.0)), float(rng.uniform(-0.5, 1.0))) for _ in range(6)]
    for G in rng.choice([1, 2, 3, 8], size=int(rng.integers(1, 3)), replace=False):
        for PP in range(1, min(L, 4) + 1):
            if rng.random() < 0.3:
                continue
            for k in range(1, PP + 1):
                for l in range(1, L - PP + 2):
                    n = int(rng.integers(0, 4))
                    pts = []
                    for _ in range(n):
                        t, d = pool[int(rng.integers(0, len(pool)))] if rng.random() < 0.3 else \
                            (float(rng.uniform(0.1, 2.0)), float(rng.uniform(-0.5, 1.0)))
                        pts.append((t, d, nid))
                        nid += 1
                    if pts:
                        cand[(int(G), PP, k, l)] = pts
    return L, cand


def _near_tie_instance(rng):
    """Stage times and deltas from a few decimal values (not representable in binary), so that
    many plans tie in real arithmetic and their values differ only by rounding."""
    L = int(rng.integers(2, 7))
    tv = [0.1, 0.2, 0.3, 0.6, 0.7, 1.1]
    dv = [0.0, 0.1, 0.3, -0.1, 0.7]
    cand = {}
    nid = 0
    for G in (1, 3, 7):
        for PP in range(1, min(L, 4) + 1):
            for k in range(1, PP + 1):
                for l in range(1, L - PP + 2):
                    pts = []
                    for _ in range(int(rng.integers(1, 4))):
                        pts.append((tv[int(rng.integers(0, len(tv)))] * l, dv[int(rng.integers(0, len(dv)))], nid))
                        nid += 1
                    cand[(G, PP, k, l)] = pts
    return L, cand


def _as_points(cand):
    return [dict(G=G, PP=PP, k=k, l=l, id=i, t=t, d=d) for (G, PP, k, l), v in cand.items() for (t, d, i) in v]


@pytest.mark.parametrize("seed", range(300))
def test_random_instances(seed):
    rng = np.random.default_rng(1000 + seed)
    L, cand = _random_instance(rng)
    for pp in (0, 1, 2, 3):
        plan = mist.plan_points(_as_points(cand), L, pp)
        _check(plan, cand, L, pp, PO.best_plan(cand, L, pp))


@pytest.mark.parametrize("seed", range(60))
def test_near_tie_instances(seed):
    rng = np.random.default_rng(5000 + seed)
    L, cand = _near_tie_instance(rng)
    for pp in (0, 2, 3):
        plan = mist.plan_points(_as_points(cand), L, pp)
        _check(plan, cand, L, pp, PO.best_plan(cand, L, pp))


def test_rounding_forms_differ():
    """The two evaluation orders of Eq. 2 do round apart on the near-tie values (otherwise the
    near-tie instances would not exercise the difference)."""
    rng = np.random.default_rng(5000)
    seen = 0
    for _ in range(2000):
        ts = [float(rng.choice([0.1, 0.2, 0.3, 0.6, 0.7, 1.1])) for _ in range(3)]
        ds = [float(rng.choice([0.0, 0.1, 0.3, -0.1, 0.7])) for _ in range(3)]
        seen += PO.plan_value(3, ts, ds) != PO.plan_value_suffix(3, ts, ds)
    assert seen > 0


@pytest.mark.parametrize("name", ["tiny", "tiny_llama"])
def test_oracle_frontier_points(name):
    wl = W.workload(name)
    L = wl["model"]["n_layers"]
    per_hw = PO.candidates(wl, alphas=[0.0, 0.2, 0.5, 0.8, 1.0])
    for hw, cand in per_hw.items():
        for pp in (0, 1, 2, 4):
            plan = mist.plan_points(_as_points(cand), L, pp)
            _check(plan, cand, L, pp, PO.best_plan(cand, L, pp))


def test_invalid_points_rejected():
    with pytest.raises(mist.MistError):
        mist.plan_points([dict(G=1, PP=2, k=3, l=1, id=0, t=1.0, d=0.0)], 2)
    with pytest.raises(mist.MistError):
        mist.plan_points([dict(G=1, PP=1, k=1, l=1, id=0, t=float("nan"), d=0.0)], 1)
    with pytest.raises(mist.MistError):
        mist.plan_points([], 0)
    assert mist.plan_points([], 3) is None
