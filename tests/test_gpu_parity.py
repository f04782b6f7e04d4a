"""GPU (libmist, HIP on gfx950) against the CPU oracle, through the C ABI.

Bar: identical argmin ids, bucket tables and frontier bits, and every cost value within
1e-12 relative (the kernels follow the same IEEE operation sequence, so the values are
compared bit for bit).  The full-size Llama workloads (llama7b-d32, llama13b-d64,
llama42b-d128-hw64) run in the benchmark's launch configuration; every group is compared with the oracle's stored whole-space run (one digest
per group), and the oracle recomputes a sample of whole groups and single configurations in
full.
"""

import os
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

pytestmark = pytest.mark.gpu

PROCS = max(1, min(16, os.cpu_count() or 1))
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "a GPU is required"
    torch.cuda.init()
    return torch


def _space(wl, torch_cuda, allocator="torch"):
    from paper_2503_19050_amd import mist
    say("space", wl["name"], wl["desc"])
    return mist.from_workload(wl, allocator=allocator)


def _eval(S, torch_cuda):
    S.eval()
    torch_cuda.cuda.synchronize()


def _compare_groups(S, ref, groups):
    ids, objs, masks = S.buckets(0, S.n_groups)
    best = S.best(0, S.n_groups)
    gi = np.asarray(groups, dtype=np.int64)
    assert np.array_equal(ids[gi], ref["bucket_id"]), "bucket ids differ"
    assert np.array_equal(objs[gi], ref["bucket_obj"]), "bucket objectives differ"
    assert np.array_equal(masks[gi], ref["frontier"]), "frontier bits differ"
    bid = np.array([best[g]["id"] for g in groups], dtype=np.uint64)
    bobj = np.array([best[g]["obj"] for g in groups])
    assert np.array_equal(bid, ref["best_id"]) and np.array_equal(bobj, ref["best_obj"])


def _compare_ids(S, o, ids):
    got = S.eval_ids(ids)
    want = o.eval_ids(ids)
    rel = np.abs(got - want) / np.maximum(np.abs(want), 1e-300)
    assert np.all(rel <= 1e-12), "max relative error %g" % rel.max()
    assert np.array_equal(got, want), "values are not bitwise equal"


def _sample_ids(o, rng, n):
    keys = o.group_keys()
    edges = []
    for k in keys[:: max(1, len(keys) // 50)]:
        edges += [k["base"], k["base"] + k["size"] - 1]
    edges += [0, o.n_configs - 1]
    rand = rng.integers(0, o.n_configs, size=n, dtype=np.uint64)
    return np.unique(np.concatenate([np.array(edges, dtype=np.uint64), rand]))


@pytest.mark.parametrize("name", ["tiny", "tiny_llama", "gpt1.3b-d8", "gpt2.7b-d16"])
def test_full_parity_small(name, torch_cuda):
    wl = W.workload(name)
    S = _space(wl, torch_cuda)
    o = O.Oracle(wl)
    assert (S.n_configs, S.n_groups) == (o.n_configs, o.n_groups)
    _eval(S, torch_cuda)
    say("oracle", name, o.n_configs, "configs on", PROCS, "processes")
    groups = list(range(o.n_groups))
    ref = O.run_groups(wl, groups, procs=PROCS) if name == "gpt2.7b-d16" else o.run()
    _compare_groups(S, ref, groups)
    _compare_ids(S, o, _sample_ids(o, np.random.default_rng(1), 3000))
    S.close()


@pytest.mark.parametrize("name", ["llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
def test_full_size_sampled_parity(name, torch_cuda):
    wl = W.workload(name)
    S = _space(wl, torch_cuda)
    o = O.Oracle(wl)
    assert (S.n_configs, S.n_groups) == (o.n_configs, o.n_groups)
    _eval(S, torch_cuda)
    keys = o.group_keys()
    sizes = np.array([k["size"] for k in keys])
    rng = np.random.default_rng(7)
    groups = {int(np.argmax(sizes)), int(np.argmin(sizes)), 0, o.n_groups - 1}
    groups |= set(int(g) for g in rng.choice(o.n_groups, size=10, replace=False))
    groups = sorted(groups)
    say("oracle", name, "groups", groups, "configs", int(sizes[groups].sum()))
    ref = O.run_groups(wl, groups, procs=PROCS)
    _compare_groups(S, ref, groups)
    _compare_ids(S, o, _sample_ids(o, rng, 3000))
    S.close()


@pytest.mark.parametrize("name", ["llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
def test_full_parity_large(name, torch_cuda):
    """Every group of the full-size workloads against the oracle's whole-space run, stored as
    one digest per group by tests/golden/make_full_oracle.py (which calls only the oracle)."""
    sys.path.insert(0, GOLDEN)
    from digest import group_digests
    gold = np.load(os.path.join(GOLDEN, "full_%s.npz" % name))
    wl = W.workload(name)
    S = _space(wl, torch_cuda)
    assert (S.n_configs, S.n_groups, S.n_buckets) == (int(gold["n_configs"]), int(gold["n_groups"]),
                                                      int(gold["n_buckets"]))
    _eval(S, torch_cuda)
    ids, objs, masks = S.buckets(0, S.n_groups)
    best = S.best(0, S.n_groups)
    bid = np.array([b["id"] for b in best], dtype=np.uint64)
    bobj = np.array([b["obj"] for b in best], dtype=np.float64)
    got = group_digests(ids, objs, masks, bid, bobj)
    bad = np.flatnonzero(got != gold["digest"])
    assert bad.size == 0, "%d of %d groups differ from the oracle, first %s" % (bad.size, S.n_groups, bad[:8])
    say(name, "all", S.n_groups, "groups match the oracle's whole-space run")
    S.close()


def test_results_api_consistent(torch_cuda):
    """mist_get_best / mist_get_pareto agree with the bucket table and with per-id values."""
    wl = W.workload("gpt1.3b-d8")
    S = _space(wl, torch_cuda)
    o = O.Oracle(wl)
    _eval(S, torch_cuda)
    ids, objs, masks = S.buckets()
    best = S.best()
    for g in range(0, S.n_groups, 97):
        b = best[g]
        if b["id"] == 0xFFFFFFFFFFFFFFFF:
            continue
        t, d, mem, obj = o.eval_ids([b["id"]])[0]
        assert (b["t"], b["d"], b["mem"], b["obj"]) == (t, d, mem, obj)
        assert ids[g][b["bucket"]] == b["id"]
        cfg = o.decode(b["id"])
        for k in ("G", "PP", "k", "l", "b", "tp", "dp"):
            assert b["cfg"][k] == cfg[k]
        assert (b["cfg"]["zero"], b["cfg"]["ckpt"]) == (cfg["zero"], cfg["ckpt"])
        par = S.pareto(g)
        assert [p["id"] for p in par] == [int(ids[g][j]) for j in range(S.n_buckets) if int(masks[g]) >> j & 1]
        objs_p = [p["obj"] for p in par]
        assert all(x > y for x, y in zip(objs_p, objs_p[1:]))
    S.close()


def test_deterministic_and_rerunnable(torch_cuda):
    wl = W.workload("gpt2.7b-d16")
    S = _space(wl, torch_cuda)
    _eval(S, torch_cuda)
    a = S.buckets()
    s2 = torch_cuda.cuda.Stream()
    with torch_cuda.cuda.stream(s2):
        S.eval(s2)
    s2.synchronize()
    b = S.buckets()
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    S.close()


def test_edge_spaces(torch_cuda):
    """Budget too small for anything, a single bucket, a single ratio, ragged tiles."""
    cases = []
    wl = W.workload("tiny")
    wl["hws"][0]["mem_bytes"] = 1.0e6
    cases.append(wl)
    wl = W.workload("tiny")
    wl["space"]["n_buckets"] = 1
    cases.append(wl)
    wl = W.workload("tiny")
    wl["space"]["ratios"] = [0.0]
    cases.append(wl)
    wl = W.workload("tiny_llama")
    wl["space"]["ratios"] = [0.0, 0.3, 0.6, 1.0]
    wl["space"]["n_buckets"] = 7
    wl["model"]["flash"] = 0
    cases.append(wl)
    for wl in cases:
        S = _space(wl, torch_cuda)
        o = O.Oracle(wl)
        _eval(S, torch_cuda)
        _compare_groups(S, o.run(), list(range(o.n_groups)))
        _compare_ids(S, o, _sample_ids(o, np.random.default_rng(3), 500))
        S.close()
    # nothing feasible: sentinel results
    S = _space(cases[0], torch_cuda)
    _eval(S, torch_cuda)
    for b in S.best():
        assert b["id"] == 0xFFFFFFFFFFFFFFFF and b["obj"] == float("inf") and b["bucket"] == -1
    assert S.pareto(0) == []
    S.close()


def test_error_paths(torch_cuda):
    from paper_2503_19050_amd import mist
    S = _space(W.workload("tiny"), torch_cuda, allocator=None)
    with pytest.raises(mist.MistError) as e:
        S.best(0, 1)
    assert e.value.status == -4
    with pytest.raises(mist.MistError) as e:
        S.eval_ids([S.n_configs])
    assert e.value.status == -5
    _eval(S, torch_cuda)
    with pytest.raises(mist.MistError) as e:
        S.best(S.n_groups, 1)
    assert e.value.status == -5
    S.close()


@pytest.mark.parametrize("R", list(range(1, 17)))
def test_every_ratio_count(R, torch_cuda):
    """The evaluation kernel is compiled per ratio count R (1..16, with activation-ratio blocks
    that change shape with R): every variant — buckets, weight samples and the exact frontier's
    candidate pass — against the oracle on a small space, every group in full."""
    from paper_2503_19050_amd import mist
    wl = W.workload("tiny")
    wl["space"]["ratios"] = [i / (R - 1) for i in range(R)] if R > 1 else [0.0]
    wl["space"]["mb"] = [1, 2]
    wl["space"]["n_devices"] = 2
    wl["space"]["global_batch"] = 32
    alphas = [0.0, 0.3, 1.0]
    wl["space"]["alphas"] = alphas
    o = O.Oracle(wl)
    say("R", R, o.n_configs, "configs")
    S = mist.from_workload(wl)
    S.eval()
    S.eval_pareto_exact()
    torch_cuda.cuda.synchronize()
    _compare_groups(S, o.run(), list(range(o.n_groups)))
    ref = o.run_alpha(alphas)
    res = S.alpha(0, S.n_groups)
    assert np.array_equal(np.array([[r["id"] for r in row] for row in res], dtype=np.uint64), ref["id"])
    assert np.array_equal(np.array([[r["obj"] for r in row] for row in res]), ref["obj"])
    for g in range(o.n_groups):
        got, want = S.pareto_exact(g), o.pareto_exact(g)
        assert [r["id"] for r in got] == [int(i) for i in want["id"]], g
        assert [r["obj"] for r in got] == list(want["obj"]), g
    _compare_ids(S, o, _sample_ids(o, np.random.default_rng(R), 300))
    S.close()


def test_launch_geometry_does_not_change_results(torch_cuda):
    """The reductions are order-independent lexicographic minima: other tile sizes and other grid
    sizes (many more claims per wave) give bit-identical buckets, best results, weight-sample
    argmins and exact frontiers."""
    from paper_2503_19050_amd import mist

    def outputs(wl):
        S = mist.from_workload(wl)
        S.eval()
        S.eval_pareto_exact()
        torch_cuda.cuda.synchronize()
        ids, objs, masks = S.buckets(0, S.n_groups)
        al = S.alpha(0, S.n_groups)
        aid = np.array([[r["id"] for r in row] for row in al], dtype=np.uint64)
        ex = [[r["id"] for r in S.pareto_exact(g)] for g in range(0, S.n_groups, max(1, S.n_groups // 40))]
        info = S.launch_info()
        S.close()
        return (ids, objs, masks, aid, ex), info

    for name, variants in (("gpt2.7b-d16", [{"tile_configs": 2048}, {"tile_configs": 65536, "max_blocks": 37}]),
                           ("tiny", [{"max_blocks": 1}, {"tile_configs": 100000}])):
        wl = W.workload(name)
        wl["space"]["alphas"] = [0.2, 0.7]
        ref, info0 = outputs(wl)
        for v in variants:
            w2 = W.workload(name)
            w2["space"]["alphas"] = [0.2, 0.7]
            w2["space"].update(v)
            got, info = outputs(w2)
            say(name, v, "tiles", info0, "->", info)
            for a, b in zip(ref[:4], got[:4]):
                assert np.array_equal(a, b), (name, v)
            assert ref[4] == got[4], (name, v)


def test_allocator_failure_is_reported(torch_cuda):
    """An allocator that returns NULL (after a given number of successful calls) makes
    mist_space_create fail with MIST_E_NOMEM and release what it had allocated."""
    import ctypes
    from paper_2503_19050_amd import mist
    L = mist.load()
    wl = W.workload("tiny")
    S = mist.from_workload(wl)          # descriptors built by the binding
    model, hw, space = S._model, S._hw, S._space
    S.close()
    for ok_calls in (0, 3):
        live = {}
        calls = [0]

        def alloc(nbytes, stream, ctx):
            calls[0] += 1
            if calls[0] > ok_calls:
                return None
            t = torch_cuda.empty(int(nbytes), dtype=torch_cuda.uint8, device="cuda")
            live[t.data_ptr()] = t
            return t.data_ptr()

        def free(ptr, ctx):
            live.pop(ptr, None)

        cb = (mist.ALLOC_FN(alloc), mist.FREE_FN(free))
        al = mist.Allocator(cb[0], cb[1], None)
        h = ctypes.c_void_p()
        rc = L.mist_space_create(ctypes.byref(model), hw, len(wl["hws"]), ctypes.byref(space), ctypes.byref(al),
                                 ctypes.byref(h))
        assert rc == -2 and "allocation" in L.mist_last_error().decode()
        assert not live, "buffers left behind"


def test_allocator_sees_the_stream_of_first_use(torch_cuda):
    """The allocator callback is told the stream each block is first used on: the null stream
    for the space's own buffers, the call's stream for the exact frontier's buffers and the
    temporaries of mist_eval_ids; every block is returned by mist_space_destroy."""
    import ctypes
    from paper_2503_19050_amd import mist
    L = mist.load()
    wl = W.workload("tiny")
    S = mist.from_workload(wl)
    model, hw, space = S._model, S._hw, S._space
    S.close()
    live, seen = {}, []

    def alloc(nbytes, stream, ctx):
        t = torch_cuda.empty(int(nbytes), dtype=torch_cuda.uint8, device="cuda")
        live[t.data_ptr()] = t
        seen.append(int(stream or 0))
        return t.data_ptr()

    def free(ptr, ctx):
        live.pop(ptr, None)

    cb = (mist.ALLOC_FN(alloc), mist.FREE_FN(free))
    al = mist.Allocator(cb[0], cb[1], None)
    h = ctypes.c_void_p()
    assert L.mist_space_create(ctypes.byref(model), hw, len(wl["hws"]), ctypes.byref(space), ctypes.byref(al),
                               ctypes.byref(h)) == 0
    assert seen and set(seen) == {0}
    side = torch_cuda.cuda.Stream()
    handle = side.cuda_stream
    del seen[:]
    assert L.mist_eval_space(h, ctypes.c_void_p(handle)) == 0
    assert seen == []                      # evaluation allocates nothing
    assert L.mist_eval_pareto_exact(h, ctypes.c_void_p(handle)) == 0
    assert seen and set(seen) == {handle}
    del seen[:]
    ids = np.arange(5, dtype=np.uint64)
    out = np.empty(20)
    assert L.mist_eval_ids(h, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), 5,
                           out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ctypes.c_void_p(handle)) == 0
    assert len(seen) == 2 and set(seen) == {handle}
    L.mist_space_destroy(h)
    assert not live, "buffers left behind"


@pytest.mark.parametrize("chunk", range(8))
def test_random_small_spaces(chunk, torch_cuda):
    """Seeded random small spaces (GPT and grouped-query Llama shapes, flash or not, device counts
    1-8 including 3 and 6, random microbatch subsets, 1-6 ratios from the eighths of [0, 1], 1-64
    buckets, both layer rules, one or two hardware samples with budgets from 1 MB to 10 GB,
    0-3 weight samples), each with a random launch geometry (tile size, grid cap) and candidate
    window: buckets, best, frontier bits, weight samples and exact frontiers of every group, and
    sampled per-configuration values, against the oracle."""
    from paper_2503_19050_amd import mist
    n = 0
    for seed in range(chunk * 25, chunk * 25 + 25):
        wl = W.random_space(seed)
        rng = np.random.default_rng(seed)
        wl["space"]["cand_window"] = int(rng.choice([0, 1, 3, 64, 1 << 30]))
        wl["space"]["tile_configs"] = int(rng.choice([0, 0, 64, 1000, 100000]))
        wl["space"]["max_blocks"] = int(rng.choice([0, 0, 1, 7, 37]))
        o = O.Oracle(wl)
        if o.n_configs > 1_500_000:
            continue
        say("random space", seed, o.n_configs, "configs", o.n_groups, "groups", "window", wl["space"]["cand_window"],
            "tile", wl["space"]["tile_configs"], "grid cap", wl["space"]["max_blocks"])
        S = mist.from_workload(wl)
        S.eval()
        S.eval_pareto_exact()
        torch_cuda.cuda.synchronize()
        if o.n_configs == 0:  # no (b, TP) pair fits the batch: every call succeeds, results empty
            assert S.n_groups == 0 and S.best() == [] and S.alpha() == []
            assert S.plan(0) is None
            with pytest.raises(mist.MistError):
                S.pareto(0)
            S.close()
            continue
        _compare_groups(S, o.run(), list(range(o.n_groups)))
        alphas = wl["space"].get("alphas", [])
        if alphas:
            ref = o.run_alpha(alphas)
            res = S.alpha(0, S.n_groups)
            assert np.array_equal(np.array([[r["id"] for r in row] for row in res], dtype=np.uint64), ref["id"])
            assert np.array_equal(np.array([[r["obj"] for r in row] for row in res]), ref["obj"])
        for g in range(o.n_groups):
            got, want = S.pareto_exact(g), o.pareto_exact(g)
            assert [r["id"] for r in got] == [int(i) for i in want["id"]], (seed, g)
            assert [r["obj"] for r in got] == list(want["obj"]), (seed, g)
        _compare_ids(S, o, _sample_ids(o, np.random.default_rng(seed), 300))
        S.close()
        n += 1
    assert n >= 15
