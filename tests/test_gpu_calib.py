"""Calibration on the GPU: the cost model with an efficiency table against the oracle (whole
spaces, bit for bit), and the co-run benchmark and operator database (Sec. 5.2.1-5.2.2) run
through the C ABI and return well-formed measurements.
"""
import math
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


@pytest.mark.parametrize("name", ["tiny", "tiny_llama", "gpt1.3b-d8"])
def test_eta_table_full_parity(name, torch_cuda):
    from paper_2503_19050_amd import mist
    wl = W.with_eta_table(W.workload(name), seed=77)
    say("eta table parity", name)
    o = O.Oracle(wl)
    ref = o.run()
    S = mist.from_workload(wl)
    S.eval()
    torch_cuda.cuda.synchronize()
    ids, objs, masks = S.buckets(0, S.n_groups)
    assert np.array_equal(ids, ref["bucket_id"])
    assert np.array_equal(objs, ref["bucket_obj"])
    assert np.array_equal(masks, ref["frontier"])
    best = S.best(0, S.n_groups)
    assert np.array_equal(np.array([b["id"] for b in best], dtype=np.uint64), ref["best_id"])
    rng = np.random.default_rng(2)
    cid = np.unique(rng.integers(0, o.n_configs, size=4000, dtype=np.uint64))
    assert np.array_equal(S.eval_ids(cid), o.eval_ids(cid))
    # the table changes the results: the formula's space differs
    base = O.Oracle(W.workload(name)).run()
    assert not np.array_equal(base["bucket_obj"], ref["bucket_obj"])
    S.close()


SMALL = {"gemm_m": 2048, "gemm_n": 2048, "gemm_k": 2048, "g2g_bytes": 16 << 20, "h2d_bytes": 16 << 20,
         "d2h_bytes": 16 << 20}


def test_corun_run_timestamps(torch_cuda):
    from paper_2503_19050_amd import mist
    say("corun run")
    with mist.Corun(SMALL, g2g_blocks=16) as C:
        for mask in (1, 2, 4, 8, 15, 0b0101):
            units = [3, 4, 2, 5]
            t = C.run(mask, SMALL, units)
            for j in range(4):
                if not mask >> j & 1:
                    assert len(t[j]) == 0
                    continue
                assert len(t[j]) == units[j] + 1
                assert t[j][0] >= 0.0
                assert np.all(np.diff(t[j]) > 0.0), (mask, j, t[j])
            mean, count = mist.corun_reduce(mask, t, units)
            assert all(count[j] >= 0 for j in range(4))
        with pytest.raises(mist.MistError):       # larger than the creation maximum
            C.run(1, dict(SMALL, h2d_bytes=SMALL["h2d_bytes"] * 2), [1, 1, 1, 1])
        with pytest.raises(mist.MistError):
            C.run(1, SMALL, [0, 1, 1, 1])


def test_corun_measure_and_fit(torch_cuda):
    from paper_2503_19050_amd import mist
    say("corun measure")
    shapes = [SMALL, dict(SMALL, gemm_n=1024, g2g_bytes=8 << 20, h2d_bytes=8 << 20, d2h_bytes=8 << 20)]
    with mist.Corun(SMALL, g2g_blocks=16) as C:
        samples = C.measure(shapes, target_s=0.005)
    assert len(samples) == 2 * mist.CORUN_SAMPLES_PER_SHAPE
    for x in samples:
        assert x["mask"] >> x["stream"] & 1 and bin(x["mask"]).count("1") >= 2
        assert x["units"] >= 0     # 0: starved for the whole window (corun_s is its length)
        assert 0.0 < x["solo_s"] < 1.0 and 0.0 < x["corun_s"] < 1.0
    phi = mist.fit_phi(samples)
    assert np.all(np.isfinite(phi)) and np.all(phi >= 1.0)
    # The least-squares factor sum(c*s) / sum(s^2) is a weighted mean of the samples' ratios
    # corun/solo (weights s^2), raised to 1: it lies between the smallest and the largest ratio
    # of its (mask, stream).  A starved member's ratio is at most the co-run window over one solo
    # unit, so the bound is the measurement's own, not a guess.
    for mask in range(16):
        for j in range(4):
            r = [x["corun_s"] / x["solo_s"] for x in samples if x["mask"] == mask and x["stream"] == j]
            if not r:
                continue
            lo, hi = max(1.0, min(r)), max(1.0, max(r))
            assert lo * (1 - 1e-12) <= phi[mask][j] <= hi * (1 + 1e-12), (mask, j, r, phi[mask][j])
    say("phi[15] =", phi[15])


def test_measure_eta(torch_cuda):
    from paper_2503_19050_amd import mist
    say("operator database")
    m = W.workload("tiny")["model"]
    model = dict(m, hidden=1024, heads=8, kv_heads=8, ffn=4096, seq=512)
    eta, sec = mist.measure_eta(model, [1, 2, 4], tp=1, peak_flops=2.5e15, reps=3)
    assert np.all(sec > 0.0) and np.all(np.isfinite(sec))
    # bf16 GEMMs against the bf16 dense peak: an efficiency above 1 would be a wrong count or time
    assert np.all(eta > 0.0) and np.all(eta <= 1.0), eta
    say("eta", eta)
    with pytest.raises(mist.MistError):
        mist.measure_eta(model, [1], tp=3, peak_flops=2.5e15)
