"""Pins of the oracle's calibration parts: the measured efficiency table of the cost model, the
co-run window reduction and the least-squares fit of the slowdown factors (Sec. 5.2.1's
operator database, Sec. 5.2.2's fitted interference model).

Expected values come from exact rational arithmetic, hand-built timelines, numpy's
least-squares solver and invariants, never from the oracle itself.
"""
import copy
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import calib_oracle as CO
from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

ULP = 2.0 ** -52


def _with_table(wl, tab):
    out = copy.deepcopy(wl)
    for h in out["hws"]:
        h["eta_max"] = 0.0
        h["eta_tab"] = list(tab)
    return out


# ---------------------------------------------------------------------------
# Efficiency table
# ---------------------------------------------------------------------------
def test_eta_table_of_ones_runs_at_peak():
    """eta = 1 for every microbatch: the compute time is the work at the peak rate plus the
    serial TP all-reduces, C = fma(4l + 2c, ar, work * (1/F)) with work < 2^53 an exact
    integer, rounded once (checked with exact rationals)."""
    wl = W.workload("tiny")
    o = O.Oracle(_with_table(wl, [1.0] * len(wl["space"]["mb"])))
    iF = 1.0 / wl["hws"][0]["flops"]
    n = 0
    for cid in range(0, o.n_configs, 211):
        T = o.terms(cid)
        cfg = o.decode(cid)
        l, c = cfg["l"], cfg["ckpt"]
        assert T["work_c"] < 2 ** 53
        inner = float(T["work_c"]) * iF
        want = float(Fraction(4 * l + 2 * c) * Fraction(T["ar"]) + Fraction(inner))
        assert T["C"] == want, (cid, T["C"], want)
        n += 1
    assert n > 50


def test_eta_table_matching_the_formula_agrees_to_rounding():
    """A table holding eta(b) = eta_max*bs/(bs + n_half) reproduces the formula's results up to
    the rounding of 1/eta (a few ulps); memory does not involve eta and is identical."""
    wl = W.workload("tiny")
    h = wl["hws"][0]
    s = wl["model"]["seq"]
    tab = [h["eta_max"] * b * s / (b * s + h["n_half"]) for b in wl["space"]["mb"]]
    a, b = O.Oracle(wl), O.Oracle(_with_table(wl, tab))
    ids = np.arange(0, a.n_configs, 53, dtype=np.uint64)
    va, vb = a.eval_ids(ids), b.eval_ids(ids)
    assert np.array_equal(va[:, 2], vb[:, 2])
    for col in (0, 3):
        rel = np.abs(va[:, col] - vb[:, col]) / np.abs(va[:, col])
        assert rel.max() <= 16 * ULP


def test_eta_table_halved_doubles_compute_without_tp():
    """Halving every eta doubles 1/eta exactly; with TP = 1 there is no all-reduce term, so the
    compute time C doubles bit for bit."""
    wl = W.workload("tiny")
    tab = [0.5, 0.625, 0.75]
    a = O.Oracle(_with_table(wl, tab))
    b = O.Oracle(_with_table(wl, [v / 2 for v in tab]))
    n = 0
    for cid in range(0, a.n_configs, 97):
        if a.decode(cid)["tp"] != 1:
            continue
        assert b.terms(cid)["C"] == 2.0 * a.terms(cid)["C"]
        n += 1
    assert n > 20


@pytest.mark.parametrize("bad", [0.0, -0.5, math.inf, math.nan])
def test_eta_table_rejects_non_positive_or_non_finite(bad):
    wl = W.workload("tiny")
    with pytest.raises(ValueError):
        O.Oracle(_with_table(wl, [0.5, bad, 0.5]))


# ---------------------------------------------------------------------------
# Co-run window
# ---------------------------------------------------------------------------
def test_corun_window_hand_timeline():
    """Stream 0 runs units [0,1],[1,2],[2,3],[3,4]; stream 1 runs [0.5,2.5],[2.5,4.5].  Both run
    in [0.5, 4]: stream 0's units 2-4 lie inside (mean 1, three units), stream 1's first unit
    only (mean 2)."""
    t = [[0.0, 1.0, 2.0, 3.0, 4.0], [0.5, 2.5, 4.5], [], []]
    mean, count = CO.corun_reduce(0b0011, t)
    assert mean[:2] == [1.0, 2.0] and count == [3, 1, 0, 0]
    assert math.isnan(mean[2]) and math.isnan(mean[3])


def test_corun_window_three_streams_and_unit_on_the_edge():
    """A unit that ends exactly at the window's end counts; one that starts before its start
    does not."""
    t = [[0.0, 2.0, 4.0, 6.0], [1.0, 3.0, 5.0, 7.0], [], [1.0, 1.5, 6.0]]
    mean, count = CO.corun_reduce(0b1011, t)
    # window [1, 6]
    assert count[0] == 2 and mean[0] == 2.0          # [2,4], [4,6]
    assert count[1] == 2 and mean[1] == 2.0          # [1,3], [3,5]
    assert count[3] == 2 and mean[3] == 2.5          # [1,1.5], [1.5,6]: (0.5 + 4.5) / 2


def test_corun_window_single_stream_is_its_whole_run():
    t = [[], [], [0.25, 1.25, 2.0, 3.5], []]
    mean, count = CO.corun_reduce(0b0100, t)
    assert count[2] == 3 and mean[2] == (3.5 - 0.25) / 3


def test_corun_window_member_without_a_whole_unit():
    t = [[0.0, 10.0], [1.0, 2.0, 3.0], [], []]
    mean, count = CO.corun_reduce(0b0011, t)
    assert count[0] == 0 and math.isnan(mean[0])
    assert count[1] == 2 and mean[1] == 1.0


# ---------------------------------------------------------------------------
# Least-squares fit
# ---------------------------------------------------------------------------
def _samples_from(phi_true, shapes, rng=None, noise=0.0):
    out = []
    for mask in range(16):
        if CO.popcount(mask) < 2:
            continue
        for j in range(4):
            if mask >> j & 1:
                for s in shapes:
                    c = phi_true[mask][j] * s
                    if rng is not None:
                        c *= 1.0 + noise * rng.standard_normal()
                    out.append((mask, j, s, c))
    return out


def test_fit_recovers_exact_factors():
    """Co-run times that are exactly phi * solo (dyadic values, exact products) give phi back
    exactly: sum(phi s^2) / sum(s^2) = phi."""
    rng = np.random.default_rng(5)
    phi_true = [[1.0] * 4 for _ in range(16)]
    for mask in range(16):
        for j in range(4):
            if CO.popcount(mask) >= 2 and mask >> j & 1:
                phi_true[mask][j] = 1.0 + int(rng.integers(0, 64)) / 64.0
    phi = CO.fit_phi(_samples_from(phi_true, [0.5, 1.0, 2.0, 4.0]))
    assert phi == phi_true


def test_fit_equals_numpy_least_squares():
    """With noise the factor is the one-parameter least-squares solution, as numpy's solver
    computes it (no intercept)."""
    rng = np.random.default_rng(9)
    phi_true = [[1.3] * 4 for _ in range(16)]
    shapes = list(rng.uniform(0.1, 3.0, size=5))
    samples = _samples_from(phi_true, shapes, rng, noise=0.05)
    phi = CO.fit_phi(samples)
    for mask in range(16):
        for j in range(4):
            rows = [(s, c) for (m, jj, s, c) in samples if m == mask and jj == j]
            if not rows:
                assert phi[mask][j] == 1.0
                continue
            A = np.array([[s] for s, _ in rows])
            y = np.array([c for _, c in rows])
            ls = np.linalg.lstsq(A, y, rcond=None)[0][0]
            assert abs(phi[mask][j] - max(1.0, ls)) <= 1e-12 * ls


def test_fit_clamps_speedups_to_one_and_leaves_unused_entries_at_one():
    phi_true = [[0.9] * 4 for _ in range(16)]
    phi = CO.fit_phi(_samples_from(phi_true, [1.0, 2.0]))
    assert all(v == 1.0 for row in phi for v in row)


def test_fit_rejects_bad_samples():
    good = _samples_from([[1.5] * 4 for _ in range(16)], [1.0])
    with pytest.raises(ValueError):
        CO.fit_phi(good[1:])                       # a member without samples
    with pytest.raises(ValueError):
        CO.fit_phi(good + [(0b0011, 2, 1.0, 1.0)])  # stream 2 is not in mask 3
    with pytest.raises(ValueError):
        CO.fit_phi(good + [(0b0011, 0, 0.0, 1.0)])  # solo time 0
    with pytest.raises(ValueError):
        CO.fit_phi(good + [(0b0011, 0, 1.0, math.inf)])
