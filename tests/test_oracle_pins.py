"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names what fixes the expected value: a hand derivation of
Algorithm 1, a published parameter count, the ZeRO paper's state accounting,
Korthikanti et al.'s activation accounting, Megatron's FLOP formula, ring
collective byte counts, exact scaling invariants, or brute force.
"""

import json
import math
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ULP = 2.0 ** -52


def _phi_table(entries):
    phi = np.ones((16, 4))
    for mask, vals in entries.items():
        phi[int(mask)] = vals
    return phi


# ---------------------------------------------------------------------------
# Algorithm 1
# ---------------------------------------------------------------------------
def test_interference_hand_derived_cases():
    """Algorithm 1 (Sec. 5.2.2) on hand-derived dyadic cases (exact)."""
    with open(os.path.join(GOLDEN, "interference_hand.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        got = O.interference(c["X"], _phi_table(c["phi"]))
        assert got == c["T"], (c["name"], got, c["T"])


def test_interference_unit_factors_is_max():
    """With every slowdown factor 1 the streams overlap perfectly: I(X) = max X."""
    rng = np.random.default_rng(1)
    ones = np.ones((16, 4))
    for _ in range(300):
        X = rng.integers(0, 1000, size=4).astype(float)
        X[0] = max(X[0], 1.0)
        assert O.interference(X, ones) == X.max()   # integers: every step exact
    for _ in range(300):
        X = rng.random(4) * 10.0 ** rng.integers(-6, 2, size=4)
        X[rng.random(4) < 0.3] = 0.0
        X[0] = X[0] or 1e-3
        got = O.interference(X, ones)
        assert abs(got - X.max()) <= 8 * ULP * X.max()


def test_interference_single_and_two_streams():
    """One stream: its own time.  Two streams with f1*x1 <= f2*x2: the shorter
    one finishes after f1*x1, the other's remaining standalone work
    (f2*x2 - f1*x1)/f2 then runs alone."""
    rng = np.random.default_rng(2)
    for j in range(4):
        X = np.zeros(4)
        X[j] = 3.25
        phi = 1.0 + rng.random((16, 4))
        assert O.interference(X, phi) == 3.25
    for _ in range(500):
        a, b = rng.choice(4, size=2, replace=False)
        X = np.zeros(4)
        X[a], X[b] = rng.random(2) * 5 + 0.01
        phi = 1.0 + 0.5 * rng.random((16, 4))
        mask = (1 << a) | (1 << b)
        f1, f2 = phi[mask][a], phi[mask][b]
        s1, s2 = X[a] * f1, X[b] * f2
        if s1 > s2:
            s1, s2, f1, f2 = s2, s1, f2, f1
        want = s1 + (s2 - s1) / f2
        got = O.interference(X, phi)
        assert abs(got - want) <= 4 * ULP * want
    # dyadic factors: exact
    X = np.array([3.0, 0.0, 0.0, 5.0])
    phi = np.ones((16, 4))
    phi[9][0], phi[9][3] = 2.0, 4.0      # scaled 6 and 20: 6 + (20 - 6) / 4
    assert O.interference(X, phi) == 6.0 + 3.5


def test_interference_bounds_and_scaling():
    """Slowdown factors >= 1 can only lengthen the overlapped time, which never
    exceeds the serial sum times the largest factor; doubling every time
    doubles the result bitwise (every step is linear)."""
    rng = np.random.default_rng(3)
    for _ in range(500):
        X = rng.random(4) * 10.0 ** rng.integers(-5, 1, size=4)
        X[rng.random(4) < 0.25] = 0.0
        X[0] = X[0] or 0.5
        phi = 1.0 + 0.5 * rng.random((16, 4))
        got = O.interference(X, phi)
        assert got >= X.max() * (1 - 8 * ULP)
        assert got <= X.sum() * phi.max() * (1 + 8 * ULP)
        assert O.interference(2.0 * X, phi) == 2.0 * got


# ---------------------------------------------------------------------------
# helpers to address one configuration
# ---------------------------------------------------------------------------
def _find_group(o, **key):
    for gi, k in enumerate(o.group_keys()):
        if all(k[n] == v for n, v in key.items()):
            return gi, k
    raise KeyError(key)


def _group_for(o, wl, PP, b, tp, **more):
    """The group of stage count PP holding the pair (b, TP)."""
    s = wl["space"]
    dp = s["n_devices"] // (PP * tp)
    return _find_group(o, PP=PP, G=s["global_batch"] // (b * dp), **more)


def _pairs(wl, PP, G):
    """(b, TP) pairs of a (PP, G) group in ascending order, from the space rules."""
    m, s = wl["model"], wl["space"]
    D, B = s["n_devices"], s["global_batch"]
    out = []
    for b in s["mb"]:
        for tp in range(1, D // PP + 1):
            if (D // PP) % tp or m["heads"] % tp or m["ffn"] % tp:
                continue
            if tp <= m["kv_heads"] and m["kv_heads"] % tp:
                continue
            if tp > m["kv_heads"] and tp % m["kv_heads"]:
                continue
            dp = D // (PP * tp)
            if B % (b * dp) == 0 and B // (b * dp) == G:
                out.append((b, tp))
    return sorted(out)


def _cid(wl, key, b, tp, c, z, wo, go, oo, ao):
    R = len(wl["space"]["ratios"])
    p = _pairs(wl, key["PP"], key["G"]).index((b, tp))
    local = ((((((p * (key["l"] + 1) + c) * 4 + z) * R + wo) * R + go) * R + oo) * R + ao)
    return key["base"] + local


def _llama7b_space():
    wl = W.workload("llama7b-d32")          # Llama-2-7B shapes
    wl["space"] = {"n_devices": 4, "global_batch": 64, "mb": [1, 2], "ratios": [0.0, 0.5, 1.0],
                   "n_buckets": 64, "l_rule": W.L_FULL}
    return wl


# Published parameter counts of the Llama 2 models whose shapes llama7b-d32 and llama13b-d64 use
# (Touvron et al., "Llama 2", 2023; 7B: 6,738,415,616; 13B: 13,015,864,320).
LLAMA2_7B = 6_738_415_616
LLAMA2_13B = 13_015_864_320


@pytest.mark.parametrize("name,count", [("llama7b-d32", LLAMA2_7B), ("llama13b-d64", LLAMA2_13B)])
def test_whole_model_parameters_match_published_llama2(name, count):
    """A single stage (PP = 1) without TP holds the whole model: embedding,
    L layers and LM head; with ZeRO-0 and no offload its resident states are
    16 bytes per parameter (2 + 2 + 12, ZeRO's K = 12)."""
    wl = W.workload(name)
    wl["space"] = {"n_devices": 2, "global_batch": 32, "mb": [1], "ratios": [0.0, 1.0],
                   "n_buckets": 64, "l_rule": W.L_FULL}
    o = O.Oracle(wl)
    gi, key = _group_for(o, wl, 1, 1, 1)
    T = o.terms(_cid(wl, key, 1, 1, 0, 0, 0, 0, 0, 0))
    assert T["Pst"] == count
    assert T["S"] == 16.0 * count


def test_zero_stage_state_bytes():
    """ZeRO (Rajbhandari et al., SC'20), fp16 params + fp16 grads + K = 12 bytes
    of optimizer state, sharded over DP: z0 16, z1 4 + 12/DP, z2 2 + 14/DP,
    z3 16/DP bytes per parameter."""
    wl = _llama7b_space()
    o = O.Oracle(wl)
    for tp in (1, 2, 4):
        dp = 4 // tp
        for b in (1, 2):
            gi, key = _group_for(o, wl, 1, b, tp)
            per_byte = {0: 16.0, 1: 4.0 + 12.0 / dp, 2: 2.0 + 14.0 / dp, 3: 16.0 / dp}
            for z in range(4):
                T = o.terms(_cid(wl, key, b, tp, 0, z, 0, 0, 0, 0))
                assert T["S"] == per_byte[z] * T["Pst"], (tp, z)
                if tp == 1:
                    assert T["Pst"] == LLAMA2_7B


def test_full_offload_working_buffers():
    """Full weight, gradient and optimizer offload: nothing resident; the
    double-buffered per-layer units remain: weights and gradients 2*2*Psi_buf
    bytes, the optimizer step 2*Psi_buf*(12*sigma_o + 2*sigma_g)."""
    wl = _llama7b_space()
    o = O.Oracle(wl)
    gi, key = _group_for(o, wl, 1, 1, 1)
    per_layer = (LLAMA2_7B - 2 * 32000 * 4096 - 4096) // 32   # from the published total
    for z in range(4):
        T = o.terms(_cid(wl, key, 1, 1, 0, z, 2, 2, 2, 0))
        dp = 4
        so = 1.0 / dp if z >= 1 else 1.0
        sg = 1.0 / dp if z >= 2 else 1.0
        assert T["Pbuf"] == per_layer
        assert T["S"] == 0.0
        assert T["Wbuf"] == 4.0 * per_layer
        assert T["Gbuf"] == 4.0 * per_layer
        assert T["Obuf"] == 2.0 * per_layer * (12.0 * so + 2.0 * sg)


def _gpt_small():
    wl = W.workload("gpt1.3b-d8")
    wl["space"] = {"n_devices": 4, "global_batch": 64, "mb": [1, 2, 4], "ratios": [0.0, 1.0],
                   "n_buckets": 64, "l_rule": W.L_FULL}
    return wl


@pytest.mark.parametrize("flash", [1, 0])
def test_activation_footprint_korthikanti(flash):
    """Korthikanti et al. (MLSys'23) Eq. 2 per layer with TP = t is
    sbh(10 + 24/t + 5as/(ht)) bytes; removing the dropout masks (2sbh and
    a s^2 b/t, dropout disabled in Sec. 6.1) leaves sbh(8 + 24/t) + 2as^2b/t,
    and FlashAttention drops the stored softmax (2as^2b/t).  A fully
    recomputed layer keeps only its input, 2sbh."""
    wl = _gpt_small()
    wl["model"]["flash"] = flash
    m = wl["model"]
    h, s, a, L = m["hidden"], m["seq"], m["heads"], m["n_layers"]
    o = O.Oracle(wl)
    for PP, k, l in [(2, 1, 5), (4, 2, 7), (1, 1, 24)]:
        for gk in o.group_keys():
            if gk["PP"] == PP and gk["k"] == k and gk["l"] == l:
                key = gk
                break
        for b, tp in _pairs(wl, PP, key["G"]):
            ke = min(k, key["G"])
            T = o.terms(_cid(wl, key, b, tp, 0, 0, 0, 0, 0, 0))
            per_layer = s * b * h * 8 + s * b * h * 24 // tp + (0 if flash else 2 * a * s * s * b // tp)
            assert T["Amb"] == l * per_layer
            assert T["Stash_plus_Off"] == float(ke * l * per_layer)
            T = o.terms(_cid(wl, key, b, tp, l, 0, 0, 0, 0, 0))
            assert T["Amb"] == 2 * s * b * h * l
            assert T["Rc"] == float(per_layer)


def test_forward_flops_megatron():
    """Narayanan et al. (SC'21): a GPT layer's forward pass is
    24bsh^2 + 4bs^2h FLOPs (split over TP ranks); an iteration with full
    recomputation costs 96 B s L h^2 (1 + s/(6h) + V/(16 L h)) FLOPs."""
    wl = _gpt_small()
    m = wl["model"]
    h, s, L, V = m["hidden"], m["seq"], m["n_layers"], m["vocab"]
    o = O.Oracle(wl)
    for b, tp in [(b, tp) for b in wl["space"]["mb"] for tp in (1, 2, 4)]:
        gi, key = _group_for(o, wl, 1, b, tp)
        T = o.terms(_cid(wl, key, b, tp, 0, 0, 0, 0, 0, 0))
        assert T["Fl"] == (24 * b * s * h * h + 4 * b * s * s * h) // tp
        if tp == 1:
            T = o.terms(_cid(wl, key, b, tp, L, 0, 0, 0, 0, 0))
            megatron = 96 * b * s * L * h * h + 16 * b * s * s * L * h + 6 * b * s * h * V
            assert T["work_c"] == megatron


def test_ring_collective_bytes():
    """Ring all-reduce moves 2(n-1)/n of the buffer per rank; an all-gather or
    reduce-scatter (n-1)/n (Patarasuk and Yuan, 2009).  TP all-reduces carry a
    (b, s, h) fp16 activation; a ZeRO AG/RS carries the stage's fp16 tensors."""
    wl = _llama7b_space()
    m = wl["model"]
    h, s = m["hidden"], m["seq"]
    o = O.Oracle(wl)
    link = wl["hws"][0]["link_bw"]
    for b, tp in [(1, 1), (1, 2), (2, 1), (2, 2)]:
        gi, key = _group_for(o, wl, 2, b, tp, k=2)
        dp = 2 // tp
        T = o.terms(_cid(wl, key, b, tp, 0, 0, 0, 0, 0, 0))
        ar = 2 * (tp - 1) / tp * b * s * h * 2
        rs = (dp - 1) / dp * 2 * T["Pst"]
        assert abs(T["ar"] * link - ar) <= 4 * ULP * max(ar, 1)
        assert abs(T["r"] * link - rs) <= 4 * ULP * max(rs, 1)
        assert abs(T["p2p"] * link - b * s * h * 2) <= 4 * ULP * b * s * h * 2   # first stage: one send
        if tp == 1:
            assert T["ar"] == 0.0


def test_doubling_rates_halves_times_bitwise():
    """Every time term is (work) x (1/rate): doubling FLOP/s, PCIe and link
    rates halves t, d and the objective exactly, leaves memory, the ids and the
    frontier unchanged."""
    wl = W.workload("tiny")
    fast = W.scaled(wl, flops=2.0, pcie=2.0, link=2.0)
    a, b = O.Oracle(wl), O.Oracle(fast)
    ids = np.arange(0, a.n_configs, 97, dtype=np.uint64)
    va, vb = a.eval_ids(ids), b.eval_ids(ids)
    assert np.array_equal(vb[:, [0, 1, 3]] * 2.0, va[:, [0, 1, 3]])
    assert np.array_equal(vb[:, 2], va[:, 2])
    ra, rb = a.run(), b.run()
    assert np.array_equal(ra["best_id"], rb["best_id"])
    assert np.array_equal(ra["bucket_id"], rb["bucket_id"])
    assert np.array_equal(ra["frontier"], rb["frontier"])
    assert np.array_equal(rb["best_obj"] * 2.0, ra["best_obj"])


def test_single_replica_makes_zero_levels_identical():
    """With DP = 1 there is nothing to shard: every ZeRO level gives the same
    time and memory, so the lowest id (ZeRO-0) wins the tie."""
    wl = W.workload("tiny")
    o = O.Oracle(wl)
    R = len(wl["space"]["ratios"])
    D = wl["space"]["n_devices"]
    dump = None
    for gi, key in enumerate(o.group_keys()):
        pairs = _pairs(wl, key["PP"], key["G"])
        d = o.dump(gi, gi + 1)
        per_c = 4 * R ** 4
        for p, (b, tp) in enumerate(pairs):
            if D // (key["PP"] * tp) != 1:
                continue
            blk = d[p * (key["l"] + 1) * per_c:(p + 1) * (key["l"] + 1) * per_c]
            blk = blk.reshape(key["l"] + 1, 4, R ** 4, 5)
            for z in range(1, 4):
                assert np.array_equal(blk[:, z], blk[:, 0])
            dump = True
    assert dump
    r = o.run()
    for gi, bid in enumerate(r["best_id"]):
        if bid == O.NONE:
            continue
        cfg = o.decode(int(bid))
        if cfg["dp"] == 1:
            assert cfg["zero"] == 0


def test_optimizer_offload_time_plausible():
    """Plausibility only: the paper reports about 7 s to offload the optimizer
    states of a 7B model at PP = 4 on L4 GPUs (Sec. 3.2).  With PCIe Gen3 x16
    (about 16 GB/s) the first-microbatch state traffic of the first of four
    stages must be within an order of magnitude of that."""
    wl = W.workload("llama7b-d32")
    wl["hws"] = [W.hw_sample(0, {"flops": 121e12, "mem_bytes": 24e9, "pcie_bw": 16e9, "link_bw": 12.5e9})]
    wl["space"] = {"n_devices": 8, "global_batch": 64, "mb": [1], "ratios": [0.0, 1.0],
                   "n_buckets": 64, "l_rule": W.L_FULL}
    o = O.Oracle(wl)
    gi, key = _group_for(o, wl, 4, 1, 1, k=4, l=8)
    T = o.terms(_cid(wl, key, 1, 1, 0, 0, 0, 0, 1, 0))
    extra = T["H2Dx"] + T["D2Hx"]
    assert 0.7 <= extra <= 70.0, extra


# ---------------------------------------------------------------------------
# enumeration
# ---------------------------------------------------------------------------
# Exact sizes of the five workloads under the enumeration rules (space
# descriptor: PP | D with PP <= L; TP | D/PP, TP | heads, TP | ffn; G = B/(b DP)
# integral; k = 1..PP; stage sizes per rule; 4 ZeRO levels; c = 0..l; R^4).
TABLE = {
    "gpt1.3b-d8": (1_686_400, 1_514),
    "gpt2.7b-d16": (273_952_500, 4_527),
    "llama7b-d32": (4_218_539_292, 5_370),
    "llama13b-d64": (20_314_621_756, 9_634),
    "llama42b-d128-hw64": (29_939_155_200, 66_496),
}


def _count_by_brute_force(wl):
    m, s = wl["model"], wl["space"]
    D, L, R = s["n_devices"], m["n_layers"], len(s["ratios"])
    groups = configs = 0
    for PP in range(1, D + 1):
        if D % PP or PP > L:
            continue
        Gs = {}
        for b in s["mb"]:
            for tp in range(1, D // PP + 1):
                if (D // PP) % tp or m["heads"] % tp or m["ffn"] % tp:
                    continue
                if (tp <= m["kv_heads"] and m["kv_heads"] % tp) or (tp > m["kv_heads"] and tp % m["kv_heads"]):
                    continue
                dp = D // (PP * tp)
                if s["global_batch"] % (b * dp) == 0:
                    Gs.setdefault(s["global_batch"] // (b * dp), []).append((b, tp))
        if s["l_rule"] == W.L_FULL:
            ls = [L] if PP == 1 else range(1, L - PP + 2)
        else:
            ls = sorted({L // PP, -(-L // PP)})
        for G, ps in Gs.items():
            for k in range(PP):
                for l in ls:
                    groups += 1
                    configs += len(ps) * (l + 1) * 4 * R ** 4
    return configs * len(wl["hws"]), groups * len(wl["hws"])


@pytest.mark.parametrize("name", ["gpt1.3b-d8", "gpt2.7b-d16", "llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
def test_space_sizes(name):
    wl = W.workload(name)
    o = O.Oracle(wl)
    assert (o.n_configs, o.n_groups) == TABLE[name]
    assert _count_by_brute_force(wl) == TABLE[name]


@pytest.mark.parametrize("name", ["tiny", "tiny_llama"])
def test_decode_matches_dump_order(name):
    """Ids are canonical: decoding an id and evaluating it alone gives the
    same values as the id's row in the full in-order dump."""
    wl = W.workload(name)
    o = O.Oracle(wl)
    dump = o.dump(0, o.n_groups)
    assert len(dump) == o.n_configs
    rng = np.random.default_rng(5)
    ids = rng.integers(0, o.n_configs, size=400).astype(np.uint64)
    ev = o.eval_ids(ids)
    assert np.array_equal(ev, dump[ids.astype(np.int64), :4])
    keys = o.group_keys()
    for cid in ids[:100]:
        c = o.decode(int(cid))
        key = next(k for k in keys if k["base"] <= cid < k["base"] + k["size"])
        assert (c["hw"], c["G"], c["PP"], c["k"], c["l"]) == (key["hw"], key["G"], key["PP"], key["k"], key["l"])
        assert c["dp"] * c["tp"] * c["PP"] == wl["space"]["n_devices"]
        assert wl["space"]["global_batch"] == c["G"] * c["b"] * c["dp"]
        assert _cid(wl, key, c["b"], c["tp"], c["ckpt"], c["zero"], c["wo"], c["go"], c["oo"], c["ao"]) == cid
