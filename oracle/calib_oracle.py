"""Plain reference for the calibration of the cost model's constants.

TEST INFRASTRUCTURE ONLY: the tests and the smoke check call this module; the library never
does, and it shares no code with it.

Mist fits the slowdown factors of its interference model from benchmarks: co-running kernels
of several shapes and combinations are timed, and the timings train one factor per co-running
combination and participant (Sec. 5.2.2, the paragraph after Algorithm 1).  Two steps of that
fit are written out here, with plain loops:

* ``corun_reduce``: from the per-unit timestamps of one co-run (each stream repeats one unit of
  work back to back; t[j][i] is the start of unit i of stream j and t[j][i+1] its end, on one
  time base), the mean duration of each member's units that lie entirely inside the window
  in which every member runs, [max_j t[j][0], min_j t[j][-1]].  Inside that window the
  combination of running streams is exactly the mask, which is what a factor phi[mask][j]
  describes.
* ``fit_phi``: per combination of two or more streams and per member, the least-squares
  factor phi that maps solo unit times s_k to co-run unit times c_k over the sampled shapes k,
  minimising sum_k (c_k - phi * s_k)^2, i.e. phi = sum c_k s_k / sum s_k^2, raised to 1 when
  below (the model's factors are slowdowns, >= 1: a co-run unit measured faster than solo is
  noise).  Entries of absent streams and of combinations of at most one stream are 1 (they
  are never used by Algorithm 1).
"""
from __future__ import annotations

import math


def popcount(mask: int) -> int:
    return bin(mask).count("1")


def corun_reduce(mask: int, t) -> tuple[list[float], list[int]]:
    """Mean unit duration and unit count inside the all-running window, per stream.

    t[j] is the list of timestamps of stream j (len = units + 1); ignored for streams not in
    mask.  Non-members and members without a whole unit inside the window get (nan, 0).
    """
    members = [j for j in range(4) if mask >> j & 1]
    if not members:
        raise ValueError("empty mask")
    for j in members:
        if len(t[j]) < 2:
            raise ValueError("stream %d has no unit" % j)
        for i in range(len(t[j]) - 1):
            if not t[j][i] <= t[j][i + 1]:
                raise ValueError("timestamps of stream %d decrease" % j)
    lo = max(t[j][0] for j in members)
    hi = min(t[j][-1] for j in members)
    mean = [math.nan] * 4
    count = [0] * 4
    for j in members:
        total = 0.0
        n = 0
        for i in range(len(t[j]) - 1):
            if t[j][i] >= lo and t[j][i + 1] <= hi:
                total += t[j][i + 1] - t[j][i]
                n += 1
        if n:
            mean[j] = total / n
            count[j] = n
    return mean, count


def fit_phi(samples) -> list[list[float]]:
    """samples: iterable of (mask, stream, solo_seconds, corun_seconds).  Returns phi[16][4]."""
    num = [[0.0] * 4 for _ in range(16)]
    den = [[0.0] * 4 for _ in range(16)]
    seen = [[False] * 4 for _ in range(16)]
    for mask, j, s, c in samples:
        if not (1 <= mask <= 15) or not (0 <= j <= 3) or not (mask >> j & 1):
            raise ValueError("stream %d is not in mask %d" % (j, mask))
        if not (s > 0 and math.isfinite(s) and c > 0 and math.isfinite(c)):
            raise ValueError("times must be positive and finite")
        num[mask][j] += c * s
        den[mask][j] += s * s
        seen[mask][j] = True
    phi = [[1.0] * 4 for _ in range(16)]
    for mask in range(16):
        if popcount(mask) < 2:
            continue
        for j in range(4):
            if not mask >> j & 1:
                continue
            if not seen[mask][j]:
                raise ValueError("no sample for stream %d of mask %d" % (j, mask))
            phi[mask][j] = max(1.0, num[mask][j] / den[mask][j])
    return phi
