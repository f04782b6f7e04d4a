"""The allocation-free entry point mist_eval_ids_noalloc against mist_eval_ids (GPU, through the C
ABI): the same per-configuration values, bit for bit, on two calls in a row (the second with fewer
ids, so the fixed device scratch holds the first call's values when the second starts), the
limit of the fixed scratch refused with MIST_E_RANGE, and an empty call."""

import ctypes
import sys

import numpy as np
import pytest

from paper_2503_19050_amd import workloads as W

pytestmark = pytest.mark.gpu

MAX_IDS = (4 << 20) // 40


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _call(L, S, ids, stream):
    ids = np.ascontiguousarray(ids, dtype=np.uint64)
    out = np.full((len(ids), 4), np.nan)
    rc = L.mist_eval_ids_noalloc(S.h, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), len(ids),
                                 out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ctypes.c_void_p(stream))
    return rc, out


@pytest.mark.parametrize("name", ["tiny_llama", "gpt2.7b-d16"])
def test_noalloc_matches_eval_ids(name):
    import torch
    from paper_2503_19050_amd import mist
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    L = mist.load()
    S = mist.from_workload(W.workload(name))
    stream = torch.cuda.current_stream().cuda_stream
    rng = np.random.default_rng(5)
    n1 = min(MAX_IDS, S.n_configs)
    for n in (n1, max(1, n1 // 7)):   # the second call is smaller
        ids = rng.integers(0, S.n_configs, size=n, dtype=np.uint64)
        ids[0], ids[-1] = 0, S.n_configs - 1
        say("noalloc", name, n)
        rc, got = _call(L, S, ids, stream)
        assert rc == 0, L.mist_last_error().decode()
        want = S.eval_ids(ids)
        assert np.array_equal(got, want), "values differ from mist_eval_ids"
    rc, _ = _call(L, S, np.zeros(0, dtype=np.uint64), stream)
    assert rc == 0
    S.close()


def test_noalloc_limits():
    import torch
    from paper_2503_19050_amd import mist
    torch.cuda.set_device(0)
    L = mist.load()
    S = mist.from_workload(W.workload("tiny"))
    stream = torch.cuda.current_stream().cuda_stream
    rc, _ = _call(L, S, np.zeros(MAX_IDS + 1, dtype=np.uint64), stream)
    assert rc == -5 and "at most" in L.mist_last_error().decode()
    rc, _ = _call(L, S, np.array([S.n_configs], dtype=np.uint64), stream)
    assert rc == -5
    S.close()
