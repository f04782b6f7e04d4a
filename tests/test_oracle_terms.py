"""Scenario pins of every cost-model term of the oracle.

Each scenario switches on one mechanism of the overlap-centric schedule
(Sec. 5.1: offloading, ZeRO sharding, recomputation, pipelining, the
repositioned optimizer step) and checks the oracle's term against the closed
form that mechanism fixes: bytes moved once or twice per microbatch, a
double-buffered per-layer unit, a ring collective's (n-1)/n, a Megatron FLOP
count divided by the effective rate, Eq. 4-6's objective.
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

ULP = 2.0 ** -52


def close(a, b, ulps=8):
    return abs(a - b) <= ulps * ULP * max(abs(a), abs(b), 1e-300)


def _wl(arch="gpt"):
    if arch == "gpt":
        wl = W.workload("gpt1.3b-d8")
        wl["space"] = {"n_devices": 8, "global_batch": 128, "mb": [1, 2, 4], "ratios": [0.0, 0.5, 1.0],
                       "n_buckets": 64, "l_rule": W.L_FULL}
    else:
        wl = W.workload("llama42b-d128-hw64")
        wl["hws"] = wl["hws"][:1]
        wl["space"] = {"n_devices": 16, "global_batch": 256, "mb": [1, 2], "ratios": [0.0, 0.5, 1.0],
                       "n_buckets": 64, "l_rule": W.L_FULL}
    return wl


class Space:
    """Addresses configurations of a workload by their knob values."""

    def __init__(self, wl):
        self.wl = wl
        self.o = O.Oracle(wl)
        self.keys = self.o.group_keys()
        self.s = wl["space"]
        self.m = wl["model"]
        self.hw = wl["hws"][0]
        self.R = len(self.s["ratios"])

    def pairs(self, PP, G):
        m, s = self.m, self.s
        D = s["n_devices"]
        out = []
        for b in s["mb"]:
            for tp in range(1, D // PP + 1):
                if (D // PP) % tp or m["heads"] % tp or m["ffn"] % tp:
                    continue
                if (tp <= m["kv_heads"] and m["kv_heads"] % tp) or (tp > m["kv_heads"] and tp % m["kv_heads"]):
                    continue
                dp = D // (PP * tp)
                if s["global_batch"] % (b * dp) == 0 and s["global_batch"] // (b * dp) == G:
                    out.append((b, tp))
        return sorted(out)

    def terms(self, PP, k, l, b, tp, c=0, z=0, wo=0, go=0, oo=0, ao=0):
        dp = self.s["n_devices"] // (PP * tp)
        G = self.s["global_batch"] // (b * dp)
        key = next(x for x in self.keys if (x["PP"], x["G"], x["k"], x["l"]) == (PP, G, k, l))
        p = self.pairs(PP, G).index((b, tp))
        R = self.R
        local = ((((((p * (l + 1) + c) * 4 + z) * R + wo) * R + go) * R + oo) * R + ao)
        T = self.o.terms(key["base"] + local)
        T["G"], T["dp"] = G, dp
        return T


@pytest.fixture(scope="module")
def gpt():
    return Space(_wl("gpt"))


@pytest.fixture(scope="module")
def llama():
    return Space(_wl("llama"))


def test_single_stage_no_overlap(gpt):
    """PP = 1, DP = 1, nothing offloaded: no stream but compute runs, so
    t = C, d = 0 and the objective is G * C (Eq. 4-6); peak memory is the
    16 bytes/parameter of model states, the in-flight activations and the fp32
    logits."""
    S = gpt
    m = S.m
    h, s, V = m["hidden"], m["seq"], m["vocab"]
    T = S.terms(1, 1, 24, 1, 8)
    assert T["dp"] == 1
    assert T["t"] == T["C"] and T["T1"] == T["C"] and T["d"] == 0.0
    assert T["obj"] == T["G"] * T["C"]
    # the logits: fp32, b x s x ceil(V / TP)
    assert T["Xl"] == 4 * 1 * s * -(-V // 8)
    assert T["Mfwd"] == T["Mbwd"] == 16.0 * T["Pst"] + T["Amb"] + T["Xl"]


@pytest.mark.parametrize("b,tp", [(1, 1), (2, 1), (4, 2)])
def test_compute_time_is_flops_over_effective_rate(gpt, b, tp):
    """C = (fwd + 2 x bwd + recomputed fwd) FLOPs / (F * eta(b)) plus the TP
    all-reduces on the critical path: two per layer forward, two backward,
    two per recomputed layer (Megatron-LM's f/g operators)."""
    S = gpt
    m, hw = S.m, S.hw
    s = m["seq"]
    eta = hw["eta_max"] * b * s / (b * s + hw["n_half"])
    for PP, k, l in [(2, 2, 9), (4, 1, 6)]:
        for c in (0, 3):
            T = S.terms(PP, k, l, b, tp, c=c)
            fl = (3 * l + c) * T["Fl"] + 3 * T["Fh"]
            want = fl / (hw["flops"] * eta) + (4 * l + 2 * c) * T["ar"]
            assert close(T["C"], want, 16), (PP, k, l, c, T["C"], want)
            if tp == 1:
                assert T["ar"] == 0.0


def test_recomputation_memory(gpt):
    """Recomputing c layers keeps only their inputs during the forward pass;
    in the backward pass one recomputed layer's full activations are live."""
    S = gpt
    for c in (1, 4, 9):
        T0 = S.terms(2, 2, 9, 2, 2, c=0)
        T = S.terms(2, 2, 9, 2, 2, c=c)
        assert T["Amb"] == (9 - c) * T["afull"] + c * T["ack"]
        assert T["Mbwd"] - T["Mfwd"] == T["afull"]
        assert T0["Mbwd"] == T0["Mfwd"]


def test_inflight_stash_and_pipeline_sends(gpt):
    """Stage k of PP holds k in-flight microbatches under 1F1B (at most G);
    middle stages send and receive a (b, s, h) activation, end stages one of
    the two, a single stage none."""
    S = gpt
    m = S.m
    bsh2 = 1 * m["seq"] * m["hidden"] * 2
    link = S.hw["link_bw"]
    for PP in (2, 4):
        for k in range(1, PP + 1):
            T = S.terms(PP, k, 5, 1, 1)
            ke = min(k, T["G"])
            assert T["Stash_plus_Off"] == ke * T["Amb"]
            sends = (k > 1) + (k < PP)
            assert close(T["p2p"] * link, sends * bsh2)
    assert S.terms(1, 1, 24, 1, 1)["p2p"] == 0.0


def test_stage_parameters_placement(gpt):
    """First stage (k = PP) holds the embedding and learned positions, the
    last (k = 1) the LM head and final norm; a GPT layer has 12h^2 + 4h
    parameters (no biases), split 12h^2/TP + 4h over TP ranks."""
    S = gpt
    m = S.m
    h, s, V = m["hidden"], m["seq"], m["vocab"]
    for tp in (1, 2):
        Vr = -(-V // tp)
        layer = 12 * h * h // tp + 4 * h
        first = S.terms(4, 4, 3, 1, tp)
        mid = S.terms(4, 2, 3, 1, tp)
        last = S.terms(4, 1, 3, 1, tp)
        assert mid["Psi"] == layer
        assert mid["Pst"] == 3 * layer
        assert first["Pst"] == 3 * layer + Vr * h + s * h
        assert last["Pst"] == 3 * layer + Vr * h + 2 * h
        assert first["Pbuf"] == max(layer, Vr * h + s * h)


@pytest.mark.parametrize("z", [0, 1, 2, 3])
def test_zero_collective_traffic(gpt, z):
    """ZeRO traffic on the GPU-GPU stream, in units of one ring AG or RS of the
    stage's fp16 tensors: per microbatch ZeRO-2 reduce-scatters gradients and
    ZeRO-3 also all-gathers weights for forward and backward (3 per
    microbatch); the first microbatch adds the gradient all-reduce (2, ZeRO-0),
    the reduce-scatter plus parameter all-gather (ZeRO-1), or the all-gather of
    updated parameters (ZeRO-2)."""
    S = gpt
    T = S.terms(2, 2, 7, 1, 1, z=z)
    assert T["dp"] == 4
    per_mb = {0: 0, 1: 0, 2: 1, 3: 3}[z]
    first = {0: 2, 1: 2, 2: 2, 3: 3}[z]
    assert close(T["G2Gs"], per_mb * T["r"] + T["p2p"])
    assert close(T["G2Gf"], first * T["r"] + T["p2p"])
    link = S.hw["link_bw"]
    assert close(T["r"] * link, 3 / 4 * 2 * T["Pst"])


def test_weight_offload(gpt):
    """Offloaded weights are fetched for the forward and again for the
    backward of every microbatch and written back once after the optimizer
    step; a double-buffered fp16 per-layer unit holds what is fetched."""
    S = gpt
    P = S.hw["pcie_bw"]
    for z in (0, 3):
        T = S.terms(2, 2, 7, 1, 1, z=z, wo=2)
        sw = 1 / T["dp"] if z == 3 else 1.0
        assert close(T["H2Ds"] * P, 2 * 2 * T["Pst"] * sw)
        assert T["D2Hs"] == 0.0 and T["H2Dx"] == 0.0
        assert close(T["D2Hx"] * P, 2 * T["Pst"] * sw)
        assert T["Wbuf"] == 2 * 2 * T["Pbuf"]
        half = S.terms(2, 2, 7, 1, 1, z=z, wo=1)
        assert close(half["Wbuf"], 2 * 2 * T["Pbuf"] * (1 - 0.5 * sw))
        assert close(half["S"], 0.5 * 2 * T["Pst"] * sw + 2 * T["Pst"] * (1 / T["dp"] if z >= 2 else 1)
                     + 12 * T["Pst"] * (1 / T["dp"] if z >= 1 else 1))


def test_gradient_and_optimizer_offload(gpt):
    """Offloaded gradients leave the GPU every microbatch and come back for the
    optimizer step before the first forward, which also fetches and writes
    back offloaded optimizer states (12 bytes/parameter, sharded from
    ZeRO-1 on); the step's working unit is a double-buffered layer of both."""
    S = gpt
    P = S.hw["pcie_bw"]
    for z in range(4):
        T = S.terms(2, 2, 7, 1, 1, z=z, go=2)
        sg = 1 / T["dp"] if z >= 2 else 1.0
        assert close(T["D2Hs"] * P, 2 * T["Pst"] * sg)
        assert close(T["H2Dx"] * P, 2 * T["Pst"] * sg)
        assert T["Gbuf"] == 2 * 2 * T["Pbuf"]
        assert close(T["Obuf"], 2 * T["Pbuf"] * 2 * sg)
        T = S.terms(2, 2, 7, 1, 1, z=z, oo=2)
        so = 1 / T["dp"] if z >= 1 else 1.0
        assert close(T["H2Dx"] * P, 12 * T["Pst"] * so)
        assert close(T["D2Hx"] * P, 12 * T["Pst"] * so)
        assert T["H2Ds"] == 0.0 and T["D2Hs"] == 0.0
        assert close(T["Obuf"], 2 * T["Pbuf"] * 12 * so)
        # the optimizer-step unit is live in the first forward, the gradient
        # unit (for sharded gradients) in the backward
        assert close(T["Mfwd"] - T["Mbwd"], T["Obuf"] - T["Gbuf"], 64)
        assert T["Gbuf"] == 2 * 2 * T["Pbuf"] * (1 - sg)


def test_activation_offload(gpt):
    """Offloaded activations leave in the forward and return in the backward
    of every microbatch; they are not stashed, and a double-buffered full
    layer of activations stages the transfers."""
    S = gpt
    P = S.hw["pcie_bw"]
    T = S.terms(2, 2, 7, 2, 1, ao=2)
    assert close(T["H2Ds"] * P, T["Amb"])
    assert close(T["D2Hs"] * P, T["Amb"])
    assert T["Stash_plus_Off"] == 2 * T["afull"]
    T = S.terms(2, 2, 7, 2, 1, ao=1)
    ke = min(2, T["G"])
    assert close(T["Stash_plus_Off"], ke * 0.5 * T["Amb"] + 0.5 * 2 * T["afull"])


def test_first_microbatch_streams(gpt):
    """The first microbatch carries the stable streams plus the once-per-step
    extras; with every slowdown factor 1 the streams overlap perfectly and
    each time is the longest stream (Algorithm 1 with unit factors)."""
    wl = _wl("gpt")
    wl["hws"][0]["phi"] = [[1.0] * 4 for _ in range(16)]
    S = Space(wl)
    for kw in [dict(z=3, wo=1, go=2), dict(z=1, oo=2, ao=1), dict(z=2, ao=2, wo=2, go=1, oo=1), dict()]:
        T = S.terms(4, 2, 5, 2, 2, **kw)
        assert T["H2Df"] == T["H2Ds"] + T["H2Dx"] and T["D2Hf"] == T["D2Hs"] + T["D2Hx"]
        assert close(T["t"], max(T["C"], T["G2Gs"], T["H2Ds"], T["D2Hs"]))
        assert close(T["T1"], max(T["C"], T["G2Gf"], T["H2Df"], T["D2Hf"]))
        assert T["d"] == T["T1"] - T["t"]
        assert close(T["obj"], T["G"] * T["t"] + T["d"], 2)


def test_gqa_kv_width(llama):
    """Grouped-query attention: K and V projections are kv_heads * d_h wide and
    split over TP ranks until TP exceeds kv_heads, after which each rank keeps
    one replicated KV head (d_h)."""
    S = llama
    m = S.m
    h, f, kv = m["hidden"], m["ffn"], m["kv_heads"]
    dh = h // m["heads"]
    for tp in (1, 2, 4, 8, 16):
        b = 1
        kvr = kv * dh // tp if tp <= kv else dh
        T = S.terms(1, 1, 60, b, tp)
        assert T["Psi"] == (2 * h * h + 3 * h * f) // tp + 2 * h * kvr + 2 * h
        assert T["atok"] == 4 * h + (2 * h + 3 * f) // tp + 2 * kvr
        assert T["Fl"] == b * m["seq"] * (2 * ((2 * h * h + 3 * h * f) // tp + 2 * h * kvr) + 4 * m["seq"] * h // tp)


def test_inflight_capped_by_accumulation_steps():
    """1F1B never holds more microbatches than a step has: a stage k deep
    stashes min(k, G) microbatches."""
    wl = _wl("gpt")
    wl["space"]["global_batch"] = 16
    wl["space"]["mb"] = [2, 4]
    S = Space(wl)
    seen_cap = False
    for k in range(1, 5):
        T = S.terms(4, k, 3, 4, 1)
        assert T["G"] == 2
        assert T["Stash_plus_Off"] == min(k, 2) * T["Amb"]
        seen_cap |= k > T["G"]
    assert seen_cap


def _two_stream(c, x, f_c, f_x):
    """Closed form of two overlapping streams (compute c, transfer x)."""
    sc, sx = c * f_c, x * f_x
    if sc <= sx:
        return sc + (sx - sc) / f_x
    return sx + (sc - sx) / f_c


def test_stream_identity_in_interference(gpt):
    """Each stream meets its own slowdown factors: a single stage without
    data parallelism overlaps compute with host->device traffic only when
    weights are offloaded (mask C+C2G) and with device->host traffic only when
    gradients are offloaded (mask C+G2C)."""
    S = gpt
    phi = S.hw["phi"]
    T = S.terms(1, 1, 24, 1, 8, wo=2)
    assert T["G2Gs"] == 0.0 and T["D2Hs"] == 0.0 and T["H2Ds"] > 0.0
    want = _two_stream(T["C"], T["H2Ds"], phi[5][0], phi[5][2])
    assert close(T["t"], want, 16)
    T = S.terms(1, 1, 24, 1, 8, go=2)
    assert T["G2Gs"] == 0.0 and T["H2Ds"] == 0.0 and T["D2Hs"] > 0.0
    want = _two_stream(T["C"], T["D2Hs"], phi[9][0], phi[9][3])
    assert close(T["t"], want, 16)
    # pipelined stage: compute with GPU<->GPU sends only
    T = S.terms(2, 2, 12, 1, 4)
    assert T["dp"] == 1 and T["H2Ds"] == 0.0 and T["D2Hs"] == 0.0
    want = _two_stream(T["C"], T["G2Gs"], phi[3][0], phi[3][1])
    assert close(T["t"], want, 16)
