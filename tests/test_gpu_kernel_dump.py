"""The evaluation kernel's own per-configuration path against the oracle, configuration by
configuration (GPU, through the C ABI).

mist_eval_ids evaluates ids one by one with the generic form of Algorithm 1; the evaluation kernel
instead shares work across a strip (the stable time across optimizer ratios, the first round of
each call with a row known per strip, the closed form of the all-zero configuration) and chooses
per wave one of four forms of the rounds (compute and the larger host stream left after the
second round, with a per-lane third row; compute finished first, one third row; the third row
looked up per lane; the general rounds).  mist_debug_eval_tiles runs that kernel path over
listed tiles and returns t, d, mem, obj, the bucket entry it chose and the forms it took for
every configuration; here the values are compared bit for bit with the oracle's
per-configuration dump (Eq. 4-6, Algorithm 1, Sec. 5.2), the bucket with the oracle's (an
infeasible configuration must land on a sink entry, NB..64), the closed forms with the
configurations they belong to, and the full-size spaces must exercise every form.
"""

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


def _check_tiles(S, o, wl, tiles, group_cache=None):
    """Compares the kernel's values over the listed tiles with the oracle's dump of their groups;
    returns the forms of Algorithm 1 the kernel took (f1 + 8 * fs per configuration)."""
    got = S.debug_eval_tiles(tiles)
    nb = wl["space"]["n_buckets"]
    ratios = np.asarray(wl["space"]["ratios"], dtype=np.float64)
    R = len(ratios)
    keys = o.group_keys()
    row = 0
    cache = {} if group_cache is None else group_cache
    for t in tiles:
        info = S.tile_info(int(t))
        g = info["group"]
        if g not in cache:
            if len(cache) >= 4:
                cache.clear()
            cache[g] = o.dump(g, g + 1)
        ref = cache[g]
        lo = info["first_id"] - keys[g]["base"]
        n = info["n_configs"]
        want = ref[lo:lo + n]
        have = got[row:row + n]
        row += n
        bad = np.flatnonzero(np.any(have[:, :4] != want[:, :4], axis=1))
        assert bad.size == 0, "tile %d, config %d: kernel %s, oracle %s" % (
            t, info["first_id"] + bad[0], have[bad[0]].tolist(), want[bad[0]].tolist())
        feasible = want[:, 4] >= 0
        assert np.array_equal(have[feasible, 4], want[feasible, 4]), "tile %d: buckets differ" % t
        assert np.all((have[~feasible, 4] >= nb) & (have[~feasible, 4] <= 64)), "tile %d: infeasible off sink" % t
        # The closed forms belong to exactly their configurations: the first microbatch's to the one
        # whose four offload ratios are all zero, the stable time's generic rounds to activation
        # ratio 0 when that ratio is zero.
        lid = np.arange(lo, lo + n, dtype=np.int64)
        ia, io, ig, iw = lid % R, (lid // R) % R, (lid // R ** 2) % R, (lid // R ** 3) % R
        f1, fs = have[:, 5].astype(np.int64) % 8, have[:, 5].astype(np.int64) // 8
        zero = (ratios[ia] == 0) & (ratios[io] == 0) & (ratios[ig] == 0) & (ratios[iw] == 0)
        assert np.array_equal(f1 == 5, zero), "tile %d: all-zero closed form" % t
        assert np.all((f1 >= 1) & (f1 <= 5)), "tile %d: first-microbatch form" % t
        assert np.array_equal(fs == 6, (ia == 0) & (ratios[0] == 0)), "tile %d: ratio-0 stable form" % t
        assert np.all(((fs >= 1) & (fs <= 4)) | (fs == 6)), "tile %d: stable form" % t
    assert row == len(got)
    return got[:, 5].astype(np.int64)


def _unit_factors(wl):
    for h in wl["hws"]:
        h["phi"] = [[1.0] * 4 for _ in range(16)]
    return wl


def _large_factors(wl, seed):
    """Slowdown factors up to 50 (far above the seeded ones), for rounds whose scaled times
    cross differently."""
    rng = np.random.default_rng(seed)
    for h in wl["hws"]:
        h["phi"] = [[float(x) for x in 1.0 + 49.0 * rng.random(4) ** 3] for _ in range(16)]
    return wl


@pytest.mark.parametrize("name, mod", [
    ("tiny", None), ("tiny_llama", None), ("tiny", "unit"), ("tiny_llama", "unit"),
    ("tiny", "large"), ("tiny_llama", "large"), ("gpt1.3b-d8", None), ("gpt1.3b-d8", "unit"),
])
def test_every_tile_small(name, mod, torch_cuda):
    from paper_2503_19050_amd import mist
    wl = W.workload(name)
    if mod == "unit":
        wl = _unit_factors(wl)
    elif mod == "large":
        wl = _large_factors(wl, 7)
    say("kernel dump", name, mod)
    S = mist.from_workload(wl)
    o = O.Oracle(wl)
    n_tiles = S.launch_info()["tiles"]
    cache = {}
    for lo in range(0, n_tiles, 512):
        _check_tiles(S, o, wl, list(range(lo, min(n_tiles, lo + 512))), cache)
    S.close()


@pytest.mark.parametrize("name, n", [("gpt2.7b-d16", 160), ("llama7b-d32", 24), ("llama42b-d128-hw64", 24)])
def test_sampled_tiles_full_size(name, n, torch_cuda):
    """Full-size spaces in the benchmark's launch configuration: the first and the last tile (a
    small tail tile) and seeded random ones."""
    from paper_2503_19050_amd import mist
    wl = W.workload(name)
    say("kernel dump", name)
    S = mist.from_workload(wl)
    o = O.Oracle(wl)
    n_tiles = S.launch_info()["tiles"]
    rng = np.random.default_rng(11)
    # Full-size tiles come first in the tile table, then every group's small tail tiles.
    picks = {0, n_tiles - 1} | set(int(t) for t in rng.integers(0, n_tiles, size=n))
    tiles = sorted(picks, key=lambda t: (S.tile_info(t)["group"], t))   # one oracle group dump at a time
    forms = _check_tiles(S, o, wl, tiles)
    S.close()
    f1, fs = np.bincount(forms % 8, minlength=8), np.bincount(forms // 8, minlength=8)
    say("first-microbatch forms", f1.tolist(), "stable forms", fs.tolist())
    # Every form of the first-microbatch call is compared somewhere on these tiles, and on
    # gpt2.7b-d16's every form of the stable time's call as well.
    assert np.all(f1[1:6] > 0), f1.tolist()
    if name == "gpt2.7b-d16":
        assert np.all(fs[[1, 2, 3, 4, 6]] > 0), fs.tolist()


@pytest.mark.parametrize("seed", range(24))
def test_random_spaces(seed, torch_cuda):
    from paper_2503_19050_amd import mist
    wl = W.random_space(seed)
    o = O.Oracle(wl)
    if o.n_configs == 0 or o.n_configs > 400_000:
        pytest.skip("empty or large random space")
    if seed % 3 == 1:
        wl = _unit_factors(wl)
        o = O.Oracle(wl)
    say("kernel dump random", seed, o.n_configs)
    S = mist.from_workload(wl)
    n_tiles = S.launch_info()["tiles"]
    _check_tiles(S, o, wl, list(range(n_tiles)), {})
    S.close()


@pytest.mark.parametrize("chunk", range(4))
def test_random_spaces_geometry(chunk, torch_cuda):
    """Seeded random spaces (seeds 100-499 in four chunks), a third each with the seeded factors,
    unit factors and factors up to 50, each with a random tile size and grid cap (so a random
    work-item order): every configuration of every tile, and every group's bucket table, best
    and frontier."""
    from paper_2503_19050_amd import mist
    n = 0
    for seed in range(100 + 100 * chunk, 200 + 100 * chunk):
        wl = W.random_space(seed)
        if seed % 3 == 1:
            wl = _unit_factors(wl)
        elif seed % 3 == 2:
            wl = _large_factors(wl, seed)
        rng = np.random.default_rng(seed)
        wl["space"]["tile_configs"] = int(rng.choice([0, 0, 64, 1000, 100000]))
        wl["space"]["max_blocks"] = int(rng.choice([0, 0, 1, 7, 37]))
        o = O.Oracle(wl)
        if o.n_configs == 0 or o.n_configs > 400_000:
            continue
        say("kernel dump random", seed, o.n_configs, "tile", wl["space"]["tile_configs"], "grid cap",
            wl["space"]["max_blocks"])
        S = mist.from_workload(wl)
        S.eval()
        ref = o.run()
        ids, objs, masks = S.buckets()
        assert np.array_equal(ids, ref["bucket_id"]), seed
        assert np.array_equal(objs, ref["bucket_obj"]), seed
        assert np.array_equal(masks, ref["frontier"]), seed
        n_tiles = S.launch_info()["tiles"]
        cache = {}
        for lo in range(0, n_tiles, 512):
            _check_tiles(S, o, wl, list(range(lo, min(n_tiles, lo + 512))), cache)
        S.close()
        n += 1
    assert n >= 60
