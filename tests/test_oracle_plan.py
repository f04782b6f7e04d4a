"""Pins of the oracle's inter-stage planner (Eq. 1-3): hand-computed values of Eq. 2, the
one-stage case that reduces to the intra-stage objective G*t + d, and small instances whose
optimum follows from the structure of Eq. 2 by hand."""
import pytest

from oracle import oracle as O
from oracle import plan_oracle as PO
from paper_2503_19050_amd import workloads as W


def test_plan_value_by_hand():
    # F = (G-1) max t + sum t + max_i (d_i - sum_{j<i} t_j), dyadic values (exact)
    assert PO.plan_value(4, [1.0, 2.0, 1.0], [0.5, 0.25, 0.0]) == 3 * 2.0 + 4.0 + 0.5
    assert PO.plan_value(1, [0.5], [0.25]) == 0.75
    # a late stage's delta is hidden behind the earlier stages' time
    assert PO.plan_value(2, [1.0, 1.0], [0.0, 0.75]) == 1.0 + 2.0 + 0.0
    # a negative delta on the first stage: the maximum takes the later (less negative) stage
    assert PO.plan_value(3, [1.0, 0.5], [-0.5, 0.25]) == 2.0 + 1.5 - 0.5


def test_one_stage_plan_is_the_intra_stage_objective():
    """With PP = 1 Eq. 2 is G*t + d of the single stage, so the best one-stage plan of each G is the
    best configuration of group (G, 1, 1, L), the tuner's own objective."""
    wl = W.workload("tiny")
    o = O.Oracle(wl)
    L = wl["model"]["n_layers"]
    keys = o.group_keys()
    best = o.run()
    cand = PO.candidates(wl)[0]
    Gs = sorted({k["G"] for k in keys if k["PP"] == 1})
    assert Gs
    for G in Gs:
        sub = {key: v for key, v in cand.items() if key[0] == G}
        plan = PO.best_plan(sub, L, pp=1)
        g = next(i for i, k in enumerate(keys) if (k["G"], k["PP"], k["k"], k["l"]) == (G, 1, 1, L))
        assert plan is not None and plan[2] == 1
        assert abs(plan[0] - best["best_obj"][g]) <= 1e-15 * best["best_obj"][g]


def test_small_instance_by_hand():
    """L = 2, G = 2.  One stage (PP = 1, l = 2): t = 3, d = 0 -> F = 6.  Two stages (l = 1 each):
    stage 1 (k = 2) offers (1, 0.5) or (0.75, 2); stage 2 (k = 1) offers (1, 0) or (2, -1).
    F(1,0.5 | 1,0) = 1 + 2 + max(0.5, -1) = 3.5; F(1,0.5 | 2,-1) = 2 + 3 + max(0.5, -2) = 5.5;
    F(0.75,2 | 1,0) = 1 + 1.75 + max(2, -0.75) = 4.75; F(0.75,2 | 2,-1) = 2 + 2.75 + 2 = 6.75.
    The optimum is 3.5 with two stages."""
    cand = {(2, 1, 1, 2): [(3.0, 0.0, 1)],
            (2, 2, 2, 1): [(1.0, 0.5, 2), (0.75, 2.0, 3)],
            (2, 2, 1, 1): [(1.0, 0.0, 4), (2.0, -1.0, 5)]}
    F, G, PP, parts, ids = PO.best_plan(cand, 2)
    assert (F, G, PP, parts, ids) == (3.5, 2, 2, [1, 1], [2, 4])
    assert PO.best_plan(cand, 2, pp=1)[0] == 6.0
    # no plan when a stage has no candidate
    assert PO.best_plan({(2, 2, 2, 1): [(1.0, 0.0, 1)]}, 2) is None


@pytest.mark.parametrize("L", [3, 4])
def test_layer_split_follows_the_bottleneck(L):
    """Stage times proportional to the layer count (t = l, d = 0) with G = 4 and PP = 2: F =
    3 max(l1, l2) + L, minimal at the most even split."""
    cand = {}
    for l in range(1, L):
        cand[(4, 2, 2, l)] = [(float(l), 0.0, 10 + l)]
        cand[(4, 2, 1, l)] = [(float(l), 0.0, 20 + l)]
    F, G, PP, parts, ids = PO.best_plan(cand, L, pp=2)
    assert F == 3 * ((L + 1) // 2) + L
    assert max(parts) == (L + 1) // 2
