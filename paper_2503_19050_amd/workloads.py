"""Seeded synthetic inputs for the tuner: model, hardware and search-space descriptors.

This module only produces input data.  It holds none of the cost model's
arithmetic and imports neither the HIP binding nor the oracle, so both sides
can take their inputs from it.

The five workloads follow the paper's evaluation setting (Sec. 6.1, Table 3 and
Table 4): GPT and Llama decoders of 1.3B-42B parameters, sequence 2048-8192,
global batch scaled with the device count.  The paper's profiled operator
database and fitted interference factors are not available, so hardware
constants and slowdown factors are drawn from SplitMix64 (Steele, Lea and
Flood, OOPSLA 2014) with a fixed seed per sample.
"""

from __future__ import annotations

import copy

GPT = 0
LLAMA = 1
L_FULL = 0       # stage layer counts 1..L-PP+1 (PP = 1: L)
L_BALANCED = 1   # stage layer counts floor(L/PP) and ceil(L/PP)

MASK64 = (1 << 64) - 1


class SplitMix64:
    """SplitMix64 generator; uniform doubles are (x >> 11) * 2**-53."""

    def __init__(self, seed: int):
        self.x = seed & MASK64

    def next_u64(self) -> int:
        self.x = (self.x + 0x9E3779B97F4A7C15) & MASK64
        z = self.x
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)

    def uniform(self) -> float:
        return (self.next_u64() >> 11) * (1.0 / 9007199254740992.0)


# Stream order of the interference model: compute, GPU<->GPU, host->device,
# device->host.  A mask has bit j set when stream j co-runs.
N_STREAMS = 4


def _popcount(v: int) -> int:
    return bin(v).count("1")


def hw_sample(seed: int, preset: dict | None = None) -> dict:
    """One hardware descriptor.

    Draw order: peak FLOP/s U[100, 1000] TFLOP/s, memory U[24, 80] GB,
    PCIe U[16, 64] GB/s, link U[100, 900] GB/s, then one slowdown factor per
    (mask, member stream) for the 11 masks with at least two streams, masks
    ascending and streams ascending: compute U[1.00, 1.10], other streams
    U[1.00, 1.50].  Entries of absent streams and of single-stream masks are 1.
    ``preset`` overrides the four scalars (the factors are still drawn).
    """
    g = SplitMix64(seed)
    flops = (100.0 + 900.0 * g.uniform()) * 1e12
    mem = (24.0 + 56.0 * g.uniform()) * 1e9
    pcie = (16.0 + 48.0 * g.uniform()) * 1e9
    link = (100.0 + 800.0 * g.uniform()) * 1e9
    phi = [[1.0] * N_STREAMS for _ in range(16)]
    for mask in range(16):
        if _popcount(mask) < 2:
            continue
        for j in range(N_STREAMS):
            if mask >> j & 1:
                hi = 0.10 if j == 0 else 0.50
                phi[mask][j] = 1.0 + hi * g.uniform()
    hw = {
        "flops": flops,
        "mem_bytes": mem,
        "pcie_bw": pcie,
        "link_bw": link,
        "eta_max": 0.75,
        "n_half": 1024.0,
        "phi": phi,
    }
    if preset:
        hw.update(preset)
    return hw


def ratios(n: int) -> list[float]:
    """n offload ratios evenly spaced on [0, 1]: j / (n - 1)."""
    if n == 1:
        return [0.0]
    return [j / (n - 1) for j in range(n)]


POW2_32 = [1, 2, 4, 8, 16, 32]


def _model(arch, L, h, heads, kv, f, s, V):
    return {
        "arch": arch, "n_layers": L, "hidden": h, "heads": heads, "kv_heads": kv,
        "ffn": f, "seq": s, "vocab": V, "bytes_w": 2, "bytes_opt": 12, "flash": 1,
    }


def _space(D, mb, R, rule, nb=64):
    return {
        "n_devices": D, "global_batch": 16 * D, "mb": list(mb), "ratios": ratios(R),
        "n_buckets": nb, "l_rule": rule,
    }


# name -> (description, model, hardware list, space)
def workload(name: str) -> dict:
    """Descriptors of a named workload (one of WORKLOADS, or a tiny test space)."""
    if name == "gpt1.3b-d8":
        # GPT L24 h2048 (1.3B class), 8 devices, fixed seed-0 hardware.
        model = _model(GPT, 24, 2048, 16, 16, 8192, 2048, 50257)
        hws = [hw_sample(0, {"flops": 200e12, "mem_bytes": 24e9, "pcie_bw": 32e9, "link_bw": 100e9})]
        space = _space(8, [1, 2, 4, 8, 16], 2, L_FULL)
        desc = "GPT L24 h2048 16 heads s2048 V50257, D=8, B=128, b 1..16, ratios {0,1}"
    elif name == "gpt2.7b-d16":
        model = _model(GPT, 32, 2560, 32, 32, 10240, 2048, 50257)
        hws = [hw_sample(2)]
        space = _space(16, POW2_32, 5, L_FULL)
        desc = "GPT L32 h2560 32 heads s2048 V50257, D=16, B=256, b 1..32, 5 ratios"
    elif name == "llama7b-d32":
        model = _model(LLAMA, 32, 4096, 32, 32, 11008, 4096, 32000)
        hws = [hw_sample(3)]
        space = _space(32, POW2_32, 9, L_FULL)
        desc = "Llama L32 h4096 f11008 32 heads s4096 V32000, D=32, B=512, b 1..32, 9 ratios"
    elif name == "llama13b-d64":
        model = _model(LLAMA, 40, 5120, 40, 40, 13824, 4096, 32000)
        hws = [hw_sample(4)]
        space = _space(64, POW2_32, 11, L_FULL)
        desc = "Llama L40 h5120 f13824 40 heads s4096 V32000, D=64, B=1024, b 1..32, 11 ratios"
    elif name == "llama42b-d128-hw64":
        model = _model(LLAMA, 60, 8192, 64, 8, 22016, 8192, 32000)
        hws = [hw_sample(100 + i) for i in range(64)]
        space = _space(128, POW2_32, 9, L_BALANCED)
        desc = ("Llama L60 h8192 f22016 64 heads / 8 KV s8192 V32000, D=128, B=2048, "
                "b 1..32, 9 ratios, 64 hardware samples")
    elif name == "tiny":
        # A small GPT space whose oracle run takes well under a second.
        model = _model(GPT, 4, 256, 8, 8, 1024, 128, 1000)
        hws = [hw_sample(7, {"mem_bytes": 2.0e8})]
        space = _space(4, [1, 2, 4], 3, L_FULL, nb=16)
        desc = "tiny GPT L4 h256, D=4, 3 ratios, 16 buckets"
    elif name == "tiny_llama":
        # Small GQA Llama space with KV replication (TP > kv heads) and 2 hw samples.
        model = _model(LLAMA, 6, 512, 8, 2, 1408, 256, 2048)
        hws = [hw_sample(11, {"mem_bytes": 6.0e8}), hw_sample(12, {"mem_bytes": 3.0e8})]
        space = _space(8, [1, 2, 4], 2, L_BALANCED, nb=64)
        desc = "tiny Llama L6 h512 8 heads / 2 KV, D=8, balanced, 2 hw samples"
    else:
        raise KeyError(name)
    return {"name": name, "desc": desc, "model": model, "hws": hws, "space": space}


WORKLOADS = ["gpt1.3b-d8", "gpt2.7b-d16", "llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"]


def random_space(seed: int) -> dict:
    """A small seeded random workload for coverage: GPT or Llama (grouped-query) shapes, flash or
    not, any device count among 1, 2, 3, 4, 6, 8, a random subset of microbatch sizes, 1-6
    offload ratios drawn from the eighths of [0, 1], 1, 3, 16 or 64 buckets, either layer rule,
    one or two hardware samples with budgets from 1 MB to 10 GB (log-uniform) and 0-3 weight
    samples.  Sizes vary widely; callers bound them."""
    g = SplitMix64(0x5EED0000 + seed)

    def pick(xs):
        return xs[min(len(xs) - 1, int(g.uniform() * len(xs)))]

    arch = pick([GPT, LLAMA])
    heads = pick([4, 8, 16])
    d_h = pick([16, 32, 64])
    kv = heads if arch == GPT else pick([d for d in (1, 2, 4, 8, 16) if heads % d == 0])
    L = 2 + int(g.uniform() * 7)
    h = heads * d_h
    model = _model(arch, L, h, heads, kv, h * pick([2, 3, 4]), pick([32, 64, 128, 256]),
                   500 + int(g.uniform() * 3000))
    model["flash"] = pick([0, 1])
    D = pick([1, 2, 3, 4, 6, 8])
    mb = [b for i, b in enumerate([1, 2, 4, 8]) if g.next_u64() >> (7 + i) & 1] or [1]
    R = 1 + int(g.uniform() * 6)
    grid = [j / 8 for j in range(9)]
    ratios_ = []
    while len(ratios_) < R:
        r = pick(grid)
        if r not in ratios_:
            ratios_.append(r)
    space = {"n_devices": D, "global_batch": D * pick([4, 8, 16]), "mb": mb, "ratios": sorted(ratios_),
             "n_buckets": pick([1, 3, 16, 64]), "l_rule": pick([L_FULL, L_BALANCED])}
    n_alpha = int(g.uniform() * 4)
    if n_alpha:
        space["alphas"] = [g.uniform() for _ in range(n_alpha)]
    hws = [hw_sample(seed * 7 + i, {"mem_bytes": 10.0 ** (6.0 + 4.0 * g.uniform())})
           for i in range(1 + int(g.uniform() * 2))]
    return {"name": "random%d" % seed, "desc": "random small space %d" % seed, "model": model, "hws": hws,
            "space": space}


def with_eta_table(wl: dict, seed: int, lo: float = 0.30, hi: float = 0.90) -> dict:
    """Copy of a workload whose hardware samples take a measured-style efficiency table in place of
    the formula: eta_max = 0 and one efficiency per microbatch size drawn U[lo, hi] from
    SplitMix64(seed + sample index), in microbatch order (the shape of an operator-database
    table; the values are synthetic)."""
    out = copy.deepcopy(wl)
    n = len(out["space"]["mb"])
    for i, hw in enumerate(out["hws"]):
        g = SplitMix64(seed + i)
        hw["eta_max"] = 0.0
        hw["eta_tab"] = [lo + (hi - lo) * g.uniform() for _ in range(n)]
    return out


def scaled(wl: dict, *, flops=1.0, pcie=1.0, link=1.0, mem=1.0) -> dict:
    """Copy of a workload with every hardware sample's scalars multiplied."""
    out = copy.deepcopy(wl)
    for hw in out["hws"]:
        hw["flops"] *= flops
        hw["pcie_bw"] *= pcie
        hw["link_bw"] *= link
        hw["mem_bytes"] *= mem
    return out
