"""A 64-bit digest of one group's outputs (bucket table, frontier bits, best), for comparing
whole spaces against stored oracle results without storing every bucket.

The words hashed per group, in order: the NB bucket ids, the NB bucket objective bit
patterns, the frontier mask, the best id and the best objective's bit pattern.  Each word is
folded in with the SplitMix64 finaliser (Steele, Lea and Flood, OOPSLA 2014):
h = mix(h + word + 0x9E3779B97F4A7C15).  No arithmetic of the cost model is involved.
"""

import numpy as np

_GOLD = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def _mix(z):
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def group_digests(bucket_id, bucket_obj, frontier, best_id, best_obj) -> np.ndarray:
    """One uint64 per group; arrays as returned by the oracle and by the library."""
    bucket_id = np.ascontiguousarray(bucket_id, dtype=np.uint64)
    bits = np.ascontiguousarray(bucket_obj, dtype=np.float64).view(np.uint64)
    words = [bucket_id[:, j] for j in range(bucket_id.shape[1])]
    words += [bits[:, j] for j in range(bits.shape[1])]
    words += [np.asarray(frontier, dtype=np.uint64), np.asarray(best_id, dtype=np.uint64),
              np.ascontiguousarray(best_obj, dtype=np.float64).view(np.uint64)]
    h = np.zeros(bucket_id.shape[0], dtype=np.uint64)
    with np.errstate(over="ignore"):
        for w in words:
            h = _mix(h + w + _GOLD)
    return h
