"""The library's host-side calibration functions against the oracle (CPU, no device needed):
the co-run window reduction, the least-squares fit of the slowdown factors and Algorithm 1 on one
vector (Sec. 5.2.2).  Results must be identical bit for bit; invalid input must be rejected.
"""
import math

import numpy as np
import pytest

from oracle import calib_oracle as CO
from oracle import oracle as O
from paper_2503_19050_amd import mist


def _timeline(rng, n_units, start):
    return list(np.cumsum(np.concatenate([[start], rng.uniform(0.1, 2.0, size=n_units)])))


def test_reduce_matches_oracle_on_random_timelines():
    rng = np.random.default_rng(3)
    for _ in range(500):
        mask = int(rng.integers(1, 16))
        units = [int(rng.integers(1, 40)) if mask >> j & 1 else 0 for j in range(4)]
        t = [_timeline(rng, units[j], rng.uniform(0, 3)) if units[j] else [] for j in range(4)]
        want_mean, want_count = CO.corun_reduce(mask, t)
        mean, count = mist.corun_reduce(mask, t, units)
        assert list(count) == want_count
        for j in range(4):
            if want_count[j]:
                assert mean[j] == want_mean[j]
            else:
                assert math.isnan(mean[j])


def test_fit_matches_oracle_on_random_samples():
    rng = np.random.default_rng(4)
    for _ in range(50):
        samples = []
        for mask in range(16):
            if CO.popcount(mask) < 2:
                continue
            for j in range(4):
                if mask >> j & 1:
                    for _k in range(int(rng.integers(1, 5))):
                        s = float(rng.uniform(1e-4, 1e-1))
                        samples.append((mask, j, s, s * float(rng.uniform(0.9, 2.5))))
        rng.shuffle(samples)
        samples = [tuple(x) for x in samples]
        want = np.array(CO.fit_phi(samples))
        got = mist.fit_phi(samples)
        assert np.array_equal(got, want)


def test_interference_matches_oracle():
    rng = np.random.default_rng(6)
    for _ in range(3000):
        phi = np.ones((16, 4))
        for mask in range(16):
            for j in range(4):
                if mask >> j & 1 and CO.popcount(mask) >= 2:
                    phi[mask, j] = rng.uniform(1.0, 1.6)
        x = rng.uniform(0, 1, size=4) * 10.0 ** rng.integers(-5, 1, size=4)
        x[rng.random(4) < 0.25] = 0.0
        assert mist.interference(phi, x) == O.interference(x, phi)


def test_interference_closed_forms():
    """Two streams f1*x1 <= f2*x2: f1*x1 + (f2*x2 - f1*x1)/f2; unit factors: the maximum."""
    phi = np.ones((16, 4))
    assert mist.interference(phi, [3.0, 1.0, 2.0, 0.5]) == 3.0
    phi[0b0011] = [1.5, 1.25, 1.0, 1.0]
    got = mist.interference(phi, [1.0, 4.0, 0.0, 0.0])
    assert got == 1.5 + (5.0 - 1.5) * (1.0 / 1.25)


@pytest.mark.parametrize("bad", [
    dict(mask=0), dict(mask=16), dict(units=[0, 1, 0, 0]), dict(t=[[0.0, 2.0, 1.0], [0.0, 1.0], [], []]),
])
def test_reduce_rejects_invalid(bad):
    args = dict(mask=0b0011, t=[[0.0, 1.0, 2.0], [0.0, 1.0], [], []], units=[2, 1, 0, 0])
    args.update(bad)
    with pytest.raises(mist.MistError):
        mist.corun_reduce(args["mask"], args["t"], args["units"])


def test_fit_and_interference_reject_invalid():
    with pytest.raises(mist.MistError):
        mist.fit_phi([(3, 2, 1.0, 1.0)])            # stream 2 is not in mask 3
    with pytest.raises(mist.MistError):
        mist.fit_phi([(3, 0, -1.0, 1.0)])
    phi = np.ones((16, 4))
    with pytest.raises(mist.MistError):
        mist.interference(phi, [1.0, -1.0, 0.0, 0.0])
    phi[0b0011, 0] = 0.5
    with pytest.raises(mist.MistError):
        mist.interference(phi, [1.0, 1.0, 0.0, 0.0])
