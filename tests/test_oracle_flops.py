"""The FP64 operation counter behind the roofline's algorithmic unit (the counting build of the
oracle), pinned by hand.

The cost model is the written-out listing of the design notes (level by level: pair,
recomputation, ZeRO, weight, gradient, optimizer-state and activation offload, then Algorithm 1
twice and the objective of Eq. 4-6).  Counting its operations by hand (add, sub and mul 1, fma 2,
min, max and comparisons 0):

  pair level        r = (rB*iD)*iL, p2p = p2pB*iL, ar = arB*iL, FE = iF*ieta        5
  recomputation     C = fma(4l+2c, ar, fma(3l+c, Fld, Fh3)*FE)                       5
  ZeRO level        Sw, Sg, So, HWz, Obo, Obg (6 mul), G2Gs, G2Gf (2 fma)           10
  weight offload    Sww, HW, DW (3 mul), Wbuf = Wb2*(1 - om*sw) (3)                  6
  gradient offload  Swg (fma), Gbuf (3), DG, Og (2 mul)                              7
  optimizer offload S, Obuf, HX, DX (4 fma), base (1), BF (2), BB (3), H2Dx, D2Hx    16
  activation        SO (fma + mul), Mf, Mb, H2Ds, D2Hs (fma + mul each), H2Df, D2Hf,
                    d (add), obj (fma)                                               16

and Algorithm 1 (Sec. 5.2.2): an update of a combination of n running streams scales each by its
factor (n mul), leaves each (scaled - overlap) / factor (n sub, n mul) and adds the overlap
(1 add): 3n + 1; the final sum adds the four leftover times (4).
"""
import json
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

LEVEL = {"pair": 5, "ckpt": 5, "zero": 10, "wo": 6, "go": 7, "oo": 16, "ao": 16}
OUTSIDE_ALG1 = sum(LEVEL.values())  # 65
FINAL_SUM = 4


def update(n):
    return 3 * n + 1


UNIT = np.ones((16, 4))


def test_hand_count_of_the_listing():
    assert OUTSIDE_ALG1 == 65
    # All four streams running and finishing one at a time: updates of 4, 3 and 2 streams.
    assert update(4) + update(3) + update(2) + FINAL_SUM == 34


@pytest.mark.parametrize("x, phi, want", [
    ([3.0, 0.0, 0.0, 0.0], UNIT, FINAL_SUM),                       # one stream: no update
    ([0.0, 0.0, 0.0, 0.0], UNIT, FINAL_SUM),
    ([0.0, 0.0, 2.5, 0.0], UNIT, FINAL_SUM),
    ([3.0, 1.0, 0.0, 0.0], UNIT, update(2) + FINAL_SUM),          # 11
    ([1.0, 2.0, 4.0, 8.0], UNIT, update(4) + update(3) + update(2) + FINAL_SUM),   # 34
    ([1.0, 1.0, 1.0, 1.0], UNIT, update(4) + FINAL_SUM),          # all finish together: 17
    ([1.0, 2.0, 2.0, 0.0], UNIT, update(3) + update(2) + FINAL_SUM),               # 21
    ([2.0, 2.0, 1.0, 0.0], UNIT, update(3) + update(2) + FINAL_SUM),               # two finish last
    ([1.0, 1.0, 2.0, 4.0], UNIT, update(4) + update(2) + FINAL_SUM),               # two finish first
    ([0.0, 5.0, 3.0, 1.0], UNIT, update(3) + update(2) + FINAL_SUM),
])
def test_interference_count_by_hand(x, phi, want):
    assert O.count_interference(x, phi) == want


def test_interference_count_with_factors():
    """Factors change the values, not the number of updates, when the finishing order stays
    strict: 1.25-scaled compute against unit transfers."""
    phi = np.ones((16, 4))
    phi[15] = [1.25, 1.0, 1.0, 1.0]
    phi[14] = [1.0, 1.0, 1.0, 1.0]
    phi[12] = [1.0, 1.0, 1.0, 1.0]
    assert O.count_interference([8.0, 1.0, 2.0, 4.0], phi) == update(4) + update(3) + update(2) + FINAL_SUM


def _xs_xf(o, cid):
    t = o.terms(cid)
    return ([t["C"], t["G2Gs"], t["H2Ds"], t["D2Hs"]], [t["C"], t["G2Gf"], t["H2Df"], t["D2Hf"]])


def test_single_configuration_equals_the_hand_count():
    """A configuration evaluated from scratch costs the 65 operations outside Algorithm 1 plus
    Algorithm 1's count on its stable and first-microbatch stream vectors."""
    for name in ("tiny", "tiny_llama"):
        wl = W.workload(name)
        o = O.Oracle(wl)
        rng = np.random.default_rng(21)
        for cid in rng.integers(0, o.n_configs, size=40):
            cid = int(cid)
            hw = o.decode(cid)["hw"]
            phi = np.asarray(wl["hws"][hw]["phi"], dtype=np.float64)
            xs, xf = _xs_xf(o, cid)
            want = OUTSIDE_ALG1 + O.count_interference(xs, phi) + O.count_interference(xf, phi)
            assert o.count_flops_ids([cid]) == want, cid


def _unit_factor_workload(name):
    wl = W.workload(name)
    for h in wl["hws"]:
        h["phi"] = [[1.0] * 4 for _ in range(16)]
    return wl


def test_known_paths():
    """Two configurations whose path through Algorithm 1 is known without running it:
    - every ratio 0 on one device per stage and one stage (no GPU-GPU traffic, no host traffic):
      both vectors hold compute alone, so no update runs: 65 + 4 + 4 = 73;
    - unit factors (Algorithm 1 is then the maximum) and four distinct, well separated positive
      stream times in both vectors: three updates per call, 65 + 34 + 34 = 133."""
    wl = _unit_factor_workload("tiny")
    o = O.Oracle(wl)
    keys = o.group_keys()
    found_zero = found_full = False
    rng = np.random.default_rng(5)
    for g in rng.permutation(len(keys)):
        k = keys[int(g)]
        for cid in rng.integers(k["base"], k["base"] + k["size"], size=60):
            c = o.decode(int(cid))
            xs, xf = _xs_xf(o, int(cid))
            n = o.count_flops_ids([int(cid)])
            if c["PP"] == 1 and c["dp"] == 1 and (c["wo"], c["go"], c["oo"], c["ao"]) == (0, 0, 0, 0):
                assert xs[1:] == [0.0, 0.0, 0.0] and xf[1:] == [0.0, 0.0, 0.0]
                assert n == 73
                found_zero = True
            vs = sorted(xs), sorted(xf)
            if all(v[0] > 0 and all(b > a * (1 + 1e-6) for a, b in zip(v, v[1:])) for v in vs):
                assert n == 133
                found_full = True
        if found_full and found_zero:
            break
    assert found_full
    # The all-zero configuration of a single-device stage: construct it directly.
    g1 = [i for i, k in enumerate(keys) if k["PP"] == 1][0]
    for p in range(keys[g1]["n_pairs"]):
        cid = keys[g1]["base"] + p * (keys[g1]["l"] + 1) * 4 * 3 ** 4
        c = o.decode(cid)
        if c["dp"] == 1:
            assert o.count_flops_ids([cid]) == 73
            found_zero = True
    assert found_zero


def test_shared_levels_equal_the_level_instance_count():
    """orc_count_flops walks a group with every level shared among the configurations below it:
    its count is each level's operations times the level's instances (pairs P, then P(l+1), then
    x4 for ZeRO, xR for each offload ratio) plus Algorithm 1 on every configuration's vectors."""
    wl = W.workload("tiny")
    o = O.Oracle(wl)
    R = len(wl["space"]["ratios"])
    phi = np.asarray(wl["hws"][0]["phi"], dtype=np.float64)
    keys = o.group_keys()
    for g in (0, len(keys) // 3, len(keys) - 1):
        k = keys[g]
        P, l = k["n_pairs"], k["l"]
        units = P * (l + 1)
        inst = {"pair": P, "ckpt": units, "zero": 4 * units, "wo": 4 * units * R,
                "go": 4 * units * R ** 2, "oo": 4 * units * R ** 3, "ao": 4 * units * R ** 4}
        alg1 = 0
        for cid in range(k["base"], k["base"] + k["size"]):
            xs, xf = _xs_xf(o, cid)
            alg1 += O.count_interference(xs, phi) + O.count_interference(xf, phi)
        want = sum(LEVEL[n] * inst[n] for n in LEVEL) + alg1
        got, n = o.count_flops(g, g + 1)
        assert n == k["size"] == inst["ao"]
        assert got == want


def test_single_configuration_counts_add_up():
    o = O.Oracle(W.workload("tiny"))
    rng = np.random.default_rng(8)
    a = rng.integers(0, o.n_configs, size=300, dtype=np.uint64)
    b = rng.integers(0, o.n_configs, size=200, dtype=np.uint64)
    assert o.count_flops_ids(a) + o.count_flops_ids(b) == o.count_flops_ids(np.concatenate([a, b]))


def test_stored_counts():
    with open(os.path.join(GOLDEN, "flops_per_config.json")) as f:
        d = json.load(f)["workloads"]
    for name in W.WORKLOADS:
        w = d[name]
        # From scratch: 65 outside Algorithm 1 plus two calls of at most 34 and at least 4.
        assert OUTSIDE_ALG1 + 8 <= w["flops_per_config"] <= OUTSIDE_ALG1 + 68
        assert w["flops_per_config"] > w["flops_per_config_shared_levels"] > 0
    o = O.Oracle(W.workload("gpt1.3b-d8"))
    assert d["gpt1.3b-d8"]["configs_sampled"] == o.n_configs    # gpt1.3b-d8: every configuration
