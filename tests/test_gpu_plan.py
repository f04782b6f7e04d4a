"""The inter-stage planner on evaluated spaces (mist_plan_pipeline: frontier points gathered on
the GPU, exact dynamic program on the host) against the exhaustive planner over the oracle's
own frontier points: computed in the test for the small spaces, stored for llama13b-d64's one-
and two-stage plans."""

import sys

import numpy as np
import pytest

from oracle import plan_oracle as PO
from paper_2503_19050_amd import workloads as W

pytestmark = pytest.mark.gpu

ALPHAS = [0.0, 0.2, 0.5, 0.8, 1.0]


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "a GPU is required"
    torch.cuda.init()
    return torch


@pytest.mark.parametrize("name,pps", [("tiny", (0, 1, 2, 4)), ("tiny_llama", (0, 1, 2, 4)), ("gpt1.3b-d8", (1, 2))])
def test_plan_matches_exhaustive_search(name, pps, torch_cuda):
    from paper_2503_19050_amd import mist
    wl = W.workload(name)
    wl["space"] = dict(wl["space"], alphas=ALPHAS)
    S = mist.from_workload(wl)
    S.eval()
    torch_cuda.cuda.synchronize()
    L = wl["model"]["n_layers"]
    per_hw = PO.candidates(wl, alphas=ALPHAS)
    for hw in range(len(wl["hws"])):
        cand = per_hw.get(hw, {})
        for pp in pps:
            plan = S.plan(hw, pp)
            want = PO.best_plan(cand, L, pp)
            say(name, "hw", hw, "pp", pp, "plan", None if plan is None else (plan["G"], plan["PP"], plan["F"]))
            if want is None:
                assert plan is None
                continue
            assert abs(plan["F"] - want[0]) <= 1e-12 * abs(want[0])
            G, PP = plan["G"], plan["PP"]
            assert plan["hw"] == hw and (pp == 0 or PP == pp)
            assert sum(st["l"] for st in plan["stages"]) == L
            for i, st in enumerate(plan["stages"]):
                assert (st["t"], st["d"], st["id"]) in cand[(G, PP, PP - i, st["l"])]
                cfg = S.decode(st["id"])
                assert (cfg["G"], cfg["PP"], cfg["k"], cfg["l"], cfg["hw"]) == (G, PP, PP - i, st["l"], hw)
            assert plan["F"] == PO.plan_value(G, [st["t"] for st in plan["stages"]],
                                              [st["d"] for st in plan["stages"]])
    S.close()


def _golden_candidates(path):
    z = np.load(path)
    cand = {}
    for r in range(len(z["id"])):
        key = (int(z["G"][r]), int(z["PP"][r]), int(z["k"][r]), int(z["l"][r]))
        cand.setdefault(int(z["hw"][r]), {}).setdefault(key, []).append(
            (float(z["t"][r]), float(z["d"][r]), int(z["id"][r])))
    return cand, [float(a) for a in z["alphas"]], [int(p) for p in z["pps"]]


def test_plan_full_size(torch_cuda):
    """llama13b-d64 with eight weight samples, plans of one and two stages: the library's plan
    (points gathered and re-evaluated on the GPU, dynamic program on the host) against the
    exhaustive search over the oracle's own points of those groups
    (tests/golden/make_plan_golden.py).  F within 1e-12, every stage one of the oracle's points,
    the layers summing to the model's; the best plan over every PP is no worse."""
    from paper_2503_19050_amd import mist
    import os
    cand_hw, alphas, pps = _golden_candidates(os.path.join(os.path.dirname(__file__), "golden",
                                                            "plan_llama13b-d64.npz"))
    wl = W.workload("llama13b-d64")
    wl["space"] = dict(wl["space"], alphas=alphas)
    L = wl["model"]["n_layers"]
    S = mist.from_workload(wl)
    S.eval()
    for hw, cand in cand_hw.items():
        for pp in pps:
            plan = S.plan(hw, pp)
            want = PO.best_plan(cand, L, pp)
            say("llama13b-d64 hw", hw, "pp", pp, "plan", plan["G"], plan["F"], "oracle", want[1], want[0])
            assert abs(plan["F"] - want[0]) <= 1e-12 * abs(want[0])
            G, PP = plan["G"], plan["PP"]
            assert plan["hw"] == hw and PP == pp
            assert sum(st["l"] for st in plan["stages"]) == L
            for i, st in enumerate(plan["stages"]):
                assert (st["t"], st["d"], st["id"]) in cand[(G, PP, PP - i, st["l"])]
            ts, ds = [st["t"] for st in plan["stages"]], [st["d"] for st in plan["stages"]]
            assert plan["F"] == PO.plan_value(G, ts, ds)
            assert PO.plan_value_suffix(G, ts, ds) == PO.best_plan(cand, L, pp, value=PO.plan_value_suffix)[0]
    best = S.plan(0, 0)
    say("llama13b-d64 plan", best["G"], best["PP"], best["F"], [st["l"] for st in best["stages"]])
    assert sum(st["l"] for st in best["stages"]) == L
    assert best["F"] == PO.plan_value(best["G"], [st["t"] for st in best["stages"]],
                                      [st["d"] for st in best["stages"]])
    assert all(best["F"] <= S.plan(0, pp)["F"] * (1 + 1e-12) for pp in pps)
    S.close()
