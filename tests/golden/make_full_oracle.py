"""Writes full_<workload>.npz for the large workloads (llama7b-d32, llama13b-d64,
llama42b-d128-hw64): the oracle run over every group, reduced to one digest per group
(tests/golden/digest.py) plus the space's counts.  The GPU parity test evaluates the whole space
with the library and compares every group's digest.

Run: python tests/golden/make_full_oracle.py [llama7b-d32 llama13b-d64 llama42b-d128-hw64]
(calls only oracle/; all cores; llama42b-d128-hw64 takes about 8 minutes on 8 cores)
"""

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, HERE)

from digest import group_digests  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2503_19050_amd import workloads as W  # noqa: E402

_oracle = None


def _init(name):
    global _oracle
    _oracle = O.Oracle(W.workload(name))


def _run(rng):
    g0, g1 = rng
    r = _oracle.run(g0, g1)
    return g0, group_digests(r["bucket_id"], r["bucket_obj"], r["frontier"], r["best_id"], r["best_obj"])


def main(names):
    import multiprocessing as mp
    for name in names:
        t0 = time.time()
        o = O.Oracle(W.workload(name))
        step = 16
        ranges = [(g, min(g + step, o.n_groups)) for g in range(0, o.n_groups, step)]
        with mp.get_context("spawn").Pool(os.cpu_count(), initializer=_init, initargs=(name,)) as pool:
            parts = dict(pool.imap_unordered(_run, ranges, chunksize=1))
        dig = np.concatenate([parts[g0] for g0, _ in ranges])
        path = os.path.join(HERE, "full_%s.npz" % name)
        np.savez_compressed(path, digest=dig, n_groups=np.int64(o.n_groups), n_configs=np.uint64(o.n_configs),
                            n_buckets=np.int32(o.n_buckets))
        print(name, o.n_groups, "groups", o.n_configs, "configs", "%.0f s" % (time.time() - t0), flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["llama7b-d32", "llama13b-d64", "llama42b-d128-hw64"])
