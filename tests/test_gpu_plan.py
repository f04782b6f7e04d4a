"""The inter-stage planner on evaluated spaces (mist_plan_pipeline: frontier points gathered on
the GPU, exact dynamic program on the host) against the exhaustive planner over the oracle's
own frontier points."""

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


def test_plan_full_size(torch_cuda):
    """llama13b-d64 with weight samples: a plan exists, uses every layer once and its value is Eq. 2 of its
    points; no single-stage plan is better."""
    from paper_2503_19050_amd import mist
    wl = W.workload("llama13b-d64")
    wl["space"] = dict(wl["space"], alphas=[k / 7.0 for k in range(8)])
    S = mist.from_workload(wl)
    S.eval()
    plan = S.plan(0, 0)
    one = S.plan(0, 1)
    say("llama13b-d64 plan", plan["G"], plan["PP"], plan["F"], [st["l"] for st in plan["stages"]])
    assert sum(st["l"] for st in plan["stages"]) == wl["model"]["n_layers"]
    assert plan["F"] == PO.plan_value(plan["G"], [st["t"] for st in plan["stages"]],
                                      [st["d"] for st in plan["stages"]])
    assert one is None or plan["F"] <= one["F"]
    S.close()
