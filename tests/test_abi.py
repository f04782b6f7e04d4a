"""The C ABI without a GPU: the library loads, exports every entry point that
include/mist.h declares, and rejects invalid descriptors before touching the device."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2503_19050_amd import mist
from paper_2503_19050_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mist.h")


def _declared():
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(mist_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ["mist_space_create", "mist_eval_space", "mist_get_best", "mist_get_pareto"]:
        assert n in names
    assert set(names) == set(mist.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = mist.load()
    for n in _declared():
        assert hasattr(L, n), n


def _create(wl, **over):
    L = mist.load()
    m = dict(wl["model"])
    s = dict(wl["space"])
    hws = [dict(h) for h in wl["hws"]]
    for k, v in over.items():
        where, key = k.split("__")
        {"m": m, "s": s, "h": hws[0]}[where][key] = v
    model = mist.ModelDesc(**{k: m[k] for k, _ in mist.ModelDesc._fields_})
    hw = (mist.HwDesc * len(hws))()
    for i, h in enumerate(hws):
        for k in ("flops", "mem_bytes", "pcie_bw", "link_bw", "eta_max", "n_half"):
            setattr(hw[i], k, float(h[k]))
        for a in range(16):
            for j in range(4):
                hw[i].phi[a][j] = float(h["phi"][a][j])
    mb = np.ascontiguousarray(s["mb"], dtype=np.int32)
    r = np.ascontiguousarray(s["ratios"], dtype=np.float64)
    al = np.ascontiguousarray(s.get("alphas", []), dtype=np.float64)
    n_al = s.get("n_alphas", len(al))
    space = mist.SpaceDesc(s["n_devices"], s["global_batch"], mb.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                           len(mb), r.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), len(r),
                           s["n_buckets"], s["l_rule"], n_al,
                           al.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if len(al) else None,
                           s.get("tile_configs", 0), s.get("max_blocks", 0), s.get("cand_window", 0))
    h = ctypes.c_void_p()
    rc = L.mist_space_create(ctypes.byref(model), hw, len(hws), ctypes.byref(space), None, ctypes.byref(h))
    return rc, L.mist_last_error().decode()


@pytest.mark.parametrize("over", [
    {"m__arch": 7}, {"m__hidden": 1000, "m__heads": 3}, {"m__kv_heads": 5}, {"m__n_layers": 0},
    {"h__flops": 0.0}, {"h__mem_bytes": -1.0}, {"h__pcie_bw": float("nan")}, {"h__eta_max": 0.0},
    {"s__n_buckets": 0}, {"s__n_buckets": 65}, {"s__mb": [2, 1]}, {"s__mb": []},
    {"s__ratios": [0.0, 1.5]}, {"s__ratios": [0.5, 0.5]}, {"s__l_rule": 3}, {"s__n_devices": 0},
    {"s__ratios": [j / 16 for j in range(17)]},
    {"s__alphas": [0.5, 1.5]}, {"s__alphas": [-0.25]}, {"s__alphas": [float("nan")]},
    {"s__alphas": [0.5] * 17}, {"s__n_alphas": 2}, {"s__n_alphas": -1},
    {"s__tile_configs": -1}, {"s__max_blocks": -4}, {"s__cand_window": -1},
    # magnitude bounds: rates in [2^-200, 2^200], efficiencies in [2^-100, 2^100], non-zero
    # ratios at least 2^-100
    {"h__flops": 2.0 ** 201}, {"h__pcie_bw": 2.0 ** -201}, {"h__link_bw": 1e300},
    {"h__eta_max": 2.0 ** -101}, {"h__n_half": 2.0 ** 101}, {"s__ratios": [0.0, 2.0 ** -101, 1.0]},
])
def test_invalid_descriptors_are_rejected(over):
    rc, msg = _create(W.workload("tiny"), **over)
    assert rc == -1 and msg


def test_bad_slowdown_factor_rejected():
    wl = W.workload("tiny")
    wl["hws"][0]["phi"] = [list(r) for r in wl["hws"][0]["phi"]]
    wl["hws"][0]["phi"][15][2] = 0.5
    rc, msg = _create(wl)
    assert rc == -1 and "slowdown" in msg


def test_slowdown_factor_above_bound_rejected():
    wl = W.workload("tiny")
    wl["hws"][0]["phi"] = [list(r) for r in wl["hws"][0]["phi"]]
    wl["hws"][0]["phi"][15][1] = 2.0 ** 101
    rc, msg = _create(wl)
    assert rc == -1 and "2^100" in msg


def test_counts_beyond_exact_range_rejected():
    rc, msg = _create(W.workload("tiny"), m__hidden=1 << 30, m__heads=1, m__kv_heads=1)
    assert rc == -1 and "2^53" in msg


def test_group_beyond_32bit_local_ids_rejected():
    """Local ids within a group are 32-bit (0xFFFFFFFF marks an empty bucket): a group of 2^32 - 1
    or more configurations is refused with MIST_E_RANGE before the device is touched.  Here PP = 1
    and l = L = 20,000 layers give 20,001 x (pairs) units of 4 * 16^4 configurations each."""
    ratios = [j / 15 for j in range(16)]
    rc, msg = _create(W.workload("tiny"), m__n_layers=20000, s__ratios=ratios, s__n_devices=1,
                      s__global_batch=16)
    assert rc == -5 and "group too large" in msg and "2^32 - 2" in msg


def test_null_arguments():
    L = mist.load()
    assert L.mist_space_create(None, None, 0, None, None, None) == -1
    assert L.mist_eval_space(None, None) == -1
    assert L.mist_space_destroy(None) == 0
    assert L.mist_exact_info(None, None, None, None, None) == -1
    assert L.mist_last_error() is not None


def test_random_small_spaces_are_valid():
    """The seeded random spaces the GPU parity test draws are accepted by the oracle's checks,
    and most are small enough for it."""
    from oracle import oracle as O
    small = 0
    for seed in range(200):
        o = O.Oracle(W.random_space(seed))
        small += o.n_configs <= 1_500_000
    assert small >= 170


def test_result_conversion_matches_field_access():
    """The binding's numpy-view conversion of mist_result arrays gives the same dicts as reading
    every ctypes field."""
    import ctypes
    n = 7
    out = (mist.Result * n)()
    for i in range(n):
        out[i].id = 1000 + i
        out[i].obj = 0.5 * i
        out[i].t, out[i].d, out[i].mem = 1.0 + i, -0.25 * i, 3e9 + i
        out[i].bucket = i - 1
        out[i].cfg.hw, out[i].cfg.G, out[i].cfg.PP, out[i].cfg.ckpt = i, 2 * i, 4, i % 3
        out[i].cfg.ao, out[i].cfg.ao_idx = 0.125 * i, i
    assert mist._results_to_dicts(out, n) == [mist._struct_to_dict(out[i]) for i in range(n)]
    assert mist._results_to_dicts(out, 0) == []
    assert mist._results_to_dicts(out, 3) == [mist._struct_to_dict(out[i]) for i in range(3)]
