"""GPU weight-sampled argmins (Eq. 4 with sampled alpha) against the CPU oracle, through the
C ABI: identical ids and bitwise-equal weighted values for every group and sample."""

import os
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

pytestmark = pytest.mark.gpu

PROCS = max(1, min(16, os.cpu_count() or 1))
ALPHAS = [k / 7.0 for k in range(8)] + [0.5]   # 0, 1/7, ..., 1 and the tuner's own weight


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "a GPU is required"
    torch.cuda.init()
    return torch


def _space(wl, alphas):
    from paper_2503_19050_amd import mist
    wl = dict(wl)
    wl["space"] = dict(wl["space"], alphas=list(alphas))
    say("space", wl["name"], wl["desc"], "alphas", len(alphas))
    return mist.from_workload(wl)


def _gpu_alpha(S, groups=None):
    res = S.alpha(0, S.n_groups)
    if groups is not None:
        res = [res[g] for g in groups]
    ids = np.array([[r["id"] for r in row] for row in res], dtype=np.uint64)
    objs = np.array([[r["obj"] for r in row] for row in res], dtype=np.float64)
    return ids, objs, res


@pytest.mark.parametrize("name", ["tiny", "tiny_llama", "gpt1.3b-d8", "gpt2.7b-d16"])
def test_alpha_parity_full(name, torch_cuda):
    wl = W.workload(name)
    S = _space(wl, ALPHAS)
    S.eval()
    torch_cuda.cuda.synchronize()
    o = O.Oracle(wl)
    if name == "gpt2.7b-d16":
        ref = O.run_alpha_groups(wl, ALPHAS, range(o.n_groups), procs=PROCS)
    else:
        ref = o.run_alpha(ALPHAS)
    ids, objs, res = _gpu_alpha(S)
    assert np.array_equal(ids, ref["id"]), "ids differ in %d places" % int((ids != ref["id"]).sum())
    assert np.array_equal(objs, ref["obj"]), "weighted values differ"
    # each result's t, d, mem and configuration are the re-evaluated configuration's
    for g in range(0, S.n_groups, max(1, S.n_groups // 20)):
        for a, r in enumerate(res[g]):
            if r["id"] == O.NONE:
                continue
            t, d, mem, obj = S.eval_ids(np.array([r["id"]], dtype=np.uint64))[0]
            assert (r["t"], r["d"], r["mem"]) == (t, d, mem)
            assert r["bucket"] >= 0 and r["cfg"]["G"] == o.group_keys(g, 1)[0]["G"]
    S.close()


@pytest.mark.parametrize("name", ["llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
def test_alpha_parity_sampled(name, torch_cuda):
    wl = W.workload(name)
    S = _space(wl, ALPHAS)
    S.eval()
    torch_cuda.cuda.synchronize()
    o = O.Oracle(wl)
    rng = np.random.default_rng(11)
    groups = sorted({0, o.n_groups - 1} | set(int(g) for g in rng.choice(o.n_groups, size=8, replace=False)))
    say("oracle", name, "groups", groups)
    ref = O.run_alpha_groups(wl, ALPHAS, groups, procs=PROCS)
    ids, objs, _ = _gpu_alpha(S, groups)
    assert np.array_equal(ids, ref["id"]) and np.array_equal(objs, ref["obj"])
    S.close()


def test_alpha_half_is_the_best_and_buckets_unchanged(torch_cuda):
    """alpha = 1/2 weighs fma(G, t, d) by exactly one half, so its argmin is each group's best;
    evaluating the samples leaves the bucket tables, best and frontier as without them."""
    from paper_2503_19050_amd import mist
    wl = W.workload("gpt2.7b-d16")
    S = _space(wl, ALPHAS)
    S.eval()
    P = mist.from_workload(wl)
    P.eval()
    torch_cuda.cuda.synchronize()
    ids, objs, _ = _gpu_alpha(S)
    best = S.best(0, S.n_groups)
    bid = np.array([b["id"] for b in best], dtype=np.uint64)
    bobj = np.array([b["obj"] for b in best])
    half = ALPHAS.index(0.5)
    assert np.array_equal(ids[:, half], bid)
    assert np.array_equal(objs[:, half], np.where(bid == O.NONE, np.inf, 0.5 * bobj))
    for a, b in zip(S.buckets(0, S.n_groups), P.buckets(0, P.n_groups)):
        assert np.array_equal(a, b)
    assert [r["id"] for r in P.best(0, P.n_groups)] == list(bid)
    with pytest.raises(mist.MistError):
        P.alpha(0, 1)   # no samples in this space
    S.close()
    P.close()
