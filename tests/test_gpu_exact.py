"""GPU exact (non-bucketed) time-vs-memory frontier against the oracle's sort-and-scan, through
the C ABI: the same ids, objectives and memory, in the same order, for every checked group."""

import os
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "a GPU is required"
    torch.cuda.init()
    return torch


def _tight():
    wl = W.workload("tiny")
    wl["hws"][0]["mem_bytes"] = 3.0e7
    wl["name"] = "tight"
    return wl


PROCS = max(1, min(16, os.cpu_count() or 1))


@pytest.mark.parametrize("name", ["tiny", "tiny_llama", "tight", "gpt1.3b-d8", "gpt2.7b-d16", "llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
def test_exact_frontier(name, torch_cuda):
    """Every group of the small spaces and of gpt2.7b-d16; for the Llama workloads seeded random
    groups plus the groups with the most candidates and the most pre-filter survivors (those past
    the sort's in-LDS capacity of 4,096 take its merge path)."""
    from paper_2503_19050_amd import mist
    wl = _tight() if name == "tight" else W.workload(name)
    S = mist.from_workload(wl)
    S.eval()
    S.eval_pareto_exact()
    torch_cuda.cuda.synchronize()
    o = O.Oracle(wl)
    if name in ("tiny", "tiny_llama", "tight", "gpt1.3b-d8", "gpt2.7b-d16"):
        groups = list(range(o.n_groups))
    else:
        rng = np.random.default_rng(4)
        size = 100 if name == "llama7b-d32" else 6
        cand, kept = S.exact_group_sizes()
        top = set(int(g) for g in np.argsort(-cand, kind="stable")[:4]) | \
            set(int(g) for g in np.argsort(-kept, kind="stable")[:4])
        big = np.flatnonzero(kept > 4096)
        if big.size:
            top |= set(int(g) for g in rng.choice(big, size=min(4, big.size), replace=False))
        say(name, "largest groups", sorted(top), "kept", [int(kept[g]) for g in sorted(top)])
        groups = sorted({0, o.n_groups - 1} | top |
                        set(int(g) for g in rng.choice(o.n_groups, size=size, replace=False)))
    ref = O.pareto_exact_groups(wl, groups, procs=PROCS if len(groups) > 16 else 1)
    best = S.best(0, S.n_groups)
    total = 0
    for g in groups:
        got = S.pareto_exact(g)
        want = ref[g]
        assert [r["id"] for r in got] == [int(i) for i in want["id"]], g
        assert [r["obj"] for r in got] == list(want["obj"]) and [r["mem"] for r in got] == list(want["mem"]), g
        if got:
            assert got[-1]["obj"] == best[g]["obj"]
        total += len(got)
    say(name, "groups", len(groups), "frontier points", total)
    S.close()


def _many_ratios(seed: int, R: int) -> dict:
    """A random space with R offload ratios: a subset of the eighths of [0, 1] (odd seeds, R <= 9)
    or R uniform values in [0, 1] (the first replaced by 0 for seeds divisible by 4)."""
    wl = W.random_space(seed)
    rng = np.random.default_rng(seed)
    if R <= 9 and seed % 2:
        rs = np.sort(rng.choice(9, size=R, replace=False)) / 8.0
    else:
        rs = np.sort(rng.uniform(0.0, 1.0, R))
        if seed % 4 == 0:
            rs[0] = 0.0
    wl["space"]["ratios"] = [float(x) for x in rs]
    return wl


@pytest.mark.parametrize("R, seed", [(7, 501), (8, 502), (9, 503), (9, 504), (11, 503), (13, 517), (16, 521)])
def test_exact_frontier_many_ratios(R, seed, torch_cuda):
    """Spaces with seven or more offload ratios, whose activation ratios the candidate pass takes
    in several blocks, with a lower bound per strip and per block: every group against the
    oracle."""
    from paper_2503_19050_amd import mist
    wl = _many_ratios(seed, R)
    assert len(set(wl["space"]["ratios"])) == R
    S = mist.from_workload(wl)
    S.eval()
    S.eval_pareto_exact()
    torch_cuda.cuda.synchronize()
    o = O.Oracle(wl)
    assert 0 < o.n_configs == S.n_configs
    best = S.best(0, S.n_groups)
    total = 0
    for g in range(o.n_groups):
        got, want = S.pareto_exact(g), o.pareto_exact(g)
        assert [r["id"] for r in got] == [int(i) for i in want["id"]], g
        assert [r["obj"] for r in got] == list(want["obj"]) and [r["mem"] for r in got] == list(want["mem"]), g
        if got:
            assert got[-1]["obj"] == best[g]["obj"]
        total += len(got)
    say("R", R, "seed", seed, "configurations", o.n_configs, "groups", o.n_groups, "frontier points", total)
    S.close()


def test_exact_and_plan_states(torch_cuda):
    """The exact frontier needs an evaluation first and is read only after its own pass; a
    space without weight samples still plans from each group's best."""
    from paper_2503_19050_amd import mist
    S = mist.from_workload(W.workload("tiny"))
    with pytest.raises(mist.MistError) as e:
        S.eval_pareto_exact()
    assert e.value.status == -4
    S.eval()
    with pytest.raises(mist.MistError) as e:
        S.pareto_exact(0)
    assert e.value.status == -4
    S.eval_pareto_exact()
    assert S.pareto_exact(0)
    with pytest.raises(mist.MistError):
        S.pareto_exact(S.n_groups)
    plan = S.plan(0)
    assert plan is not None and sum(st["l"] for st in plan["stages"]) == W.workload("tiny")["model"]["n_layers"]
    with pytest.raises(mist.MistError):
        S.plan(1)      # no such hardware sample
    S.eval()           # a new evaluation invalidates the exact frontier
    with pytest.raises(mist.MistError):
        S.pareto_exact(0)
    S.close()


def test_exact_frontier_of_an_empty_space_on_reused_blocks(torch_cuda):
    """A space without configurations launches no kernel of the candidate pass, so nothing
    clears the overflow pool's counter: its count must not be read from the block, whatever the
    allocator's block held before (here blocks just freed with every byte 0x01)."""
    from paper_2503_19050_amd import mist
    wl = W.random_space(158)
    assert O.Oracle(wl).n_configs == 0
    for _ in range(3):
        junk = [torch_cuda.full((n,), 1, dtype=torch_cuda.uint8, device="cuda") for n in (256, 512, 4096) * 64]
        torch_cuda.cuda.synchronize()
        del junk
        S = mist.from_workload(wl)
        S.eval()
        S.eval_pareto_exact()
        torch_cuda.cuda.synchronize()
        info = S.exact_info()
        assert info["candidates"] == 0 and info["kept"] == 0 and info["tiles_again"] == 0, info
        assert S.n_groups == 0
        S.close()


@pytest.mark.parametrize("name", ["tight", "gpt1.3b-d8", "gpt2.7b-d16"])
def test_candidate_windows_do_not_change_results(name, torch_cuda):
    """The frontier does not depend on the candidate windows: windows as large as their tiles
    (no tile evaluated twice), the default, small ones (many tiles evaluated twice) and windows
    of one slot (every tile with two or more candidates evaluated twice); each space evaluated
    twice in a row, against the oracle on a sample of groups."""
    from paper_2503_19050_amd import mist
    wl = _tight() if name == "tight" else W.workload(name)
    o = O.Oracle(wl)
    rng = np.random.default_rng(11)
    groups = sorted({0, o.n_groups - 1} | set(int(g) for g in rng.choice(o.n_groups, size=min(12, o.n_groups),
                                                                           replace=False)))
    want = {g: o.pareto_exact(g) for g in groups}
    sizes = {}
    for window in (1, 0, 64, 1 << 30):
        say(name, "cand_window", window)
        w = dict(wl, space=dict(wl["space"], cand_window=window))
        S = mist.from_workload(w)
        for _ in range(2):
            S.eval()
            S.eval_pareto_exact()
            info = S.exact_info()
            say("  ", info)
            assert 0 <= info["kept"] <= info["candidates"]
            assert 0 <= info["tiles_again"] <= info["tiles_live"]
            if window == 1:
                assert info["tiles_again"] == 0  # a window as large as its tile never overflows
            sizes.setdefault((info["candidates"], info["kept"]), []).append(window)
            for g in groups:
                got = S.pareto_exact(g)
                assert [r["id"] for r in got] == [int(i) for i in want[g]["id"]], (window, g)
                assert [r["obj"] for r in got] == list(want[g]["obj"]), (window, g)
                assert [r["mem"] for r in got] == list(want[g]["mem"]), (window, g)
        S.close()
    assert len(sizes) == 1, sizes  # the same candidates and survivors whatever the windows


def test_exact_frontier_on_several_streams(torch_cuda):
    """Calls on different streams, one after another, give the oracle's frontier; a space
    destroyed right after a call on another stream waits for it."""
    from paper_2503_19050_amd import mist
    wl = W.workload("gpt1.3b-d8")
    o = O.Oracle(wl)
    S = mist.from_workload(wl)
    S.eval()
    streams = [torch_cuda.cuda.Stream(), torch_cuda.cuda.Stream()]
    for st in streams + streams[::-1]:
        S.eval_pareto_exact(stream=st)
    for g in range(o.n_groups):
        want = o.pareto_exact(g)
        got = S.pareto_exact(g)
        assert [r["id"] for r in got] == [int(i) for i in want["id"]], g
        assert [r["obj"] for r in got] == list(want["obj"]), g
    S.eval_pareto_exact(stream=streams[1])
    S.close()
    torch_cuda.cuda.synchronize()


def test_evaluations_and_exact_frontier_interleaved_on_streams(torch_cuda):
    """Evaluations and exact frontiers alternating between two streams with no synchronisation
    by the caller: the library orders them, and the results are the oracle's."""
    from paper_2503_19050_amd import mist
    wl = W.workload("gpt1.3b-d8")
    o = O.Oracle(wl)
    want_best = o.run()
    S = mist.from_workload(wl)
    s1, s2 = torch_cuda.cuda.Stream(), torch_cuda.cuda.Stream()
    S.eval(stream=s1)
    S.eval(stream=s2)
    S.eval_pareto_exact(stream=s1)
    S.eval(stream=s2)
    S.eval_pareto_exact(stream=s2)
    best = S.best(0, S.n_groups)
    assert [b["id"] for b in best] == [int(i) for i in want_best["best_id"]]
    for g in range(0, o.n_groups, 7):
        want = o.pareto_exact(g)
        assert [r["id"] for r in S.pareto_exact(g)] == [int(i) for i in want["id"]], g
    S.close()
