"""ctypes wrapper of the plain single-threaded CPU oracle (mist_oracle.cpp).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline use it to check and time the GPU path.  It takes plain descriptor
dictionaries (model, hardware list, space) and shares no code with the HIP
library or its Python binding.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mist_oracle.cpp")
LIB = os.path.join(HERE, "liboracle.so")
# A test may point the wrapper at another build of the oracle (a planted-mistake
# variant built by the mutation test); the library is then loaded as given.
LIB_OVERRIDE = os.environ.get("MIST_ORACLE_LIB")

CXXFLAGS = ["-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
            "-Wall", "-Wextra"]

NONE = np.uint64(0xFFFFFFFFFFFFFFFF)

_lock = threading.Lock()
_lib = None


def build(force: bool = True, extra: list[str] | None = None, out: str | None = None) -> str:
    """Compiles the oracle with g++ into oracle/liboracle.so (or ``out``)."""
    out = out or LIB
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(SRC):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["g++", *CXXFLAGS, *(extra or []), SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


def lib() -> ctypes.CDLL:
    global _lib
    with _lock:
        if _lib is None:
            if LIB_OVERRIDE:
                L = ctypes.CDLL(LIB_OVERRIDE)
            else:
                build(force=False)
                L = ctypes.CDLL(LIB)
            P = ctypes.POINTER
            args = [P(_Model), P(_Hw), ctypes.c_int32, P(_Space)]
            L.orc_space_info.argtypes = args + [P(ctypes.c_uint64), P(ctypes.c_int64)]
            L.orc_group_keys.argtypes = args + [ctypes.c_int64, ctypes.c_int64, P(_GroupKey)]
            L.orc_decode.argtypes = args + [ctypes.c_uint64, P(ctypes.c_int64)]
            L.orc_eval_ids.argtypes = args + [P(ctypes.c_uint64), ctypes.c_int64, P(ctypes.c_double)]
            L.orc_eval_terms.argtypes = args + [ctypes.c_uint64, P(_Terms)]
            L.orc_dump.argtypes = args + [ctypes.c_int64, ctypes.c_int64, P(ctypes.c_double), ctypes.c_uint64]
            L.orc_run.argtypes = args + [ctypes.c_int64, ctypes.c_int64, P(ctypes.c_uint64), P(ctypes.c_double),
                                         P(ctypes.c_uint64), P(ctypes.c_double), P(ctypes.c_uint64)]
            L.orc_count_flops.argtypes = args + [ctypes.c_int64, ctypes.c_int64, P(ctypes.c_uint64),
                                                 P(ctypes.c_uint64)]
            L.orc_run_alpha.argtypes = args + [P(ctypes.c_double), ctypes.c_int32, ctypes.c_int64,
                                               ctypes.c_int64, P(ctypes.c_uint64), P(ctypes.c_double)]
            L.orc_pareto_exact.argtypes = args + [ctypes.c_int64, P(ctypes.c_uint64), P(ctypes.c_double),
                                                  P(ctypes.c_double), ctypes.c_int64, P(ctypes.c_int64)]
            L.orc_count_flops_ids.argtypes = args + [P(ctypes.c_uint64), ctypes.c_int64, P(ctypes.c_uint64)]
            L.orc_count_interference.argtypes = [P(ctypes.c_double), P(ctypes.c_double), P(ctypes.c_uint64)]
            L.orc_interference.argtypes = [P(ctypes.c_double), P(ctypes.c_double)]
            L.orc_interference.restype = ctypes.c_double
            _lib = L
        return _lib


class _Model(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int64),
                ("heads", ctypes.c_int32), ("kv_heads", ctypes.c_int32), ("ffn", ctypes.c_int64),
                ("seq", ctypes.c_int64), ("vocab", ctypes.c_int64), ("bytes_w", ctypes.c_int32),
                ("bytes_opt", ctypes.c_int32), ("flash", ctypes.c_int32)]


class _Hw(ctypes.Structure):
    _fields_ = [("flops", ctypes.c_double), ("mem_bytes", ctypes.c_double), ("pcie_bw", ctypes.c_double),
                ("link_bw", ctypes.c_double), ("eta_max", ctypes.c_double), ("n_half", ctypes.c_double),
                ("phi", ctypes.c_double * 64), ("eta_tab", ctypes.c_double * 16)]


class _Space(ctypes.Structure):
    _fields_ = [("n_devices", ctypes.c_int64), ("global_batch", ctypes.c_int64),
                ("mb", ctypes.POINTER(ctypes.c_int32)), ("n_mb", ctypes.c_int32),
                ("ratios", ctypes.POINTER(ctypes.c_double)), ("n_ratios", ctypes.c_int32),
                ("n_buckets", ctypes.c_int32), ("l_rule", ctypes.c_int32)]


class _GroupKey(ctypes.Structure):
    _fields_ = [("hw", ctypes.c_int32), ("n_pairs", ctypes.c_int32), ("G", ctypes.c_int64),
                ("PP", ctypes.c_int64), ("k", ctypes.c_int64), ("l", ctypes.c_int64),
                ("base", ctypes.c_uint64), ("size", ctypes.c_uint64)]


_TERM_INT = ["Psi", "Pst", "Pbuf", "atok", "afull", "ack", "Fl", "Fh", "Xl", "Amb", "work_c"]
_TERM_DBL = ["S", "Wbuf", "Gbuf", "Obuf", "Stash_plus_Off", "Rc", "Mfwd", "Mbwd", "Mem",
             "C", "G2Gs", "G2Gf", "H2Ds", "D2Hs", "H2Df", "D2Hf", "ar", "r", "p2p", "H2Dx", "D2Hx",
             "t", "T1", "d", "obj"]


class _Terms(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in _TERM_INT] + [(n, ctypes.c_double) for n in _TERM_DBL]


def _dp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _up(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))


class Oracle:
    """The oracle bound to one (model, hardware list, space) description."""

    def __init__(self, wl: dict):
        m, hws, s = wl["model"], wl["hws"], wl["space"]
        self.model = _Model(**{k: m[k] for k, _ in _Model._fields_})
        self.hw = (_Hw * len(hws))()
        for i, h in enumerate(hws):
            for k in ("flops", "mem_bytes", "pcie_bw", "link_bw", "eta_max", "n_half"):
                setattr(self.hw[i], k, float(h[k]))
            flat = [float(v) for row in h["phi"] for v in row]
            self.hw[i].phi[:] = flat
            tab = [float(v) for v in h.get("eta_tab", [])]
            self.hw[i].eta_tab[:len(tab)] = tab
        self.n_hw = len(hws)
        self._mb = np.ascontiguousarray(s["mb"], dtype=np.int32)
        self._ratios = np.ascontiguousarray(s["ratios"], dtype=np.float64)
        self.space = _Space(s["n_devices"], s["global_batch"],
                            self._mb.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), len(self._mb),
                            _dp(self._ratios), len(self._ratios), s["n_buckets"], s["l_rule"])
        self.n_buckets = s["n_buckets"]
        self.L = lib()
        n = ctypes.c_uint64()
        g = ctypes.c_int64()
        self._check(self.L.orc_space_info(*self._args(), ctypes.byref(n), ctypes.byref(g)))
        self.n_configs = n.value
        self.n_groups = g.value

    def _args(self):
        return (ctypes.byref(self.model), self.hw, self.n_hw, ctypes.byref(self.space))

    @staticmethod
    def _check(rc):
        if rc != 0:
            raise ValueError("oracle call failed with status %d" % rc)

    def group_keys(self, g0: int = 0, n: int | None = None) -> list[dict]:
        n = self.n_groups - g0 if n is None else n
        out = (_GroupKey * max(n, 1))()
        self._check(self.L.orc_group_keys(*self._args(), g0, n, out))
        return [{k: getattr(out[i], k) for k, _ in _GroupKey._fields_} for i in range(n)]

    def decode(self, cid: int) -> dict:
        out = (ctypes.c_int64 * 14)()
        self._check(self.L.orc_decode(*self._args(), cid, out))
        keys = ["hw", "G", "PP", "k", "l", "b", "tp", "dp", "zero", "ckpt", "wo", "go", "oo", "ao"]
        return dict(zip(keys, list(out)))

    def eval_ids(self, ids) -> np.ndarray:
        ids = np.ascontiguousarray(ids, dtype=np.uint64)
        out = np.empty((len(ids), 4), dtype=np.float64)
        self._check(self.L.orc_eval_ids(*self._args(), _up(ids), len(ids), _dp(out)))
        return out

    def terms(self, cid: int) -> dict:
        t = _Terms()
        self._check(self.L.orc_eval_terms(*self._args(), cid, ctypes.byref(t)))
        return {k: getattr(t, k) for k, _ in _Terms._fields_}

    def dump(self, g0: int, g1: int) -> np.ndarray:
        keys = self.group_keys(g0, g1 - g0)
        n = sum(k["size"] for k in keys)
        out = np.empty((n, 5), dtype=np.float64)
        self._check(self.L.orc_dump(*self._args(), g0, g1, _dp(out), n))
        return out

    def run(self, g0: int = 0, g1: int | None = None) -> dict:
        g1 = self.n_groups if g1 is None else g1
        n = g1 - g0
        NB = self.n_buckets
        res = {
            "best_id": np.empty(n, dtype=np.uint64), "best_obj": np.empty(n, dtype=np.float64),
            "bucket_id": np.empty((n, NB), dtype=np.uint64), "bucket_obj": np.empty((n, NB), dtype=np.float64),
            "frontier": np.empty(n, dtype=np.uint64),
        }
        self._check(self.L.orc_run(*self._args(), g0, g1, _up(res["best_id"]), _dp(res["best_obj"]),
                                   _up(res["bucket_id"]), _dp(res["bucket_obj"]), _up(res["frontier"])))
        return res

    def run_alpha(self, alphas, g0: int = 0, g1: int | None = None) -> dict:
        """Per group and weight sample alpha: the feasible configuration minimising
        alpha*G*t + (1-alpha)*d (Eq. 4), lowest id on ties: {"id", "obj"} of shape [n, A]."""
        g1 = self.n_groups if g1 is None else g1
        al = np.ascontiguousarray(alphas, dtype=np.float64)
        n = g1 - g0
        res = {"id": np.empty((n, len(al)), dtype=np.uint64), "obj": np.empty((n, len(al)), dtype=np.float64)}
        self._check(self.L.orc_run_alpha(*self._args(), _dp(al), len(al), g0, g1, _up(res["id"]),
                                         _dp(res["obj"])))
        return res

    def pareto_exact(self, g: int) -> dict:
        """Exact (non-bucketed) time-vs-memory frontier of group g: {"id", "obj", "mem"} in
        increasing memory, strictly decreasing objective."""
        cap = 4096
        while True:
            res = {"id": np.empty(cap, dtype=np.uint64), "obj": np.empty(cap), "mem": np.empty(cap)}
            n = ctypes.c_int64()
            rc = self.L.orc_pareto_exact(*self._args(), g, _up(res["id"]), _dp(res["obj"]), _dp(res["mem"]),
                                         cap, ctypes.byref(n))
            if rc == -5 and n.value > cap:
                cap = n.value
                continue
            self._check(rc)
            return {k: v[:n.value] for k, v in res.items()}

    def count_flops(self, g0: int = 0, g1: int | None = None) -> tuple[int, int]:
        g1 = self.n_groups if g1 is None else g1
        f = ctypes.c_uint64()
        c = ctypes.c_uint64()
        self._check(self.L.orc_count_flops(*self._args(), g0, g1, ctypes.byref(f), ctypes.byref(c)))
        return f.value, c.value

    def count_flops_ids(self, ids) -> int:
        """FP64 operations of the definition for the given configurations, each evaluated from
        scratch (no level shared between configurations)."""
        a = np.ascontiguousarray(ids, dtype=np.uint64)
        f = ctypes.c_uint64()
        self._check(self.L.orc_count_flops_ids(*self._args(), _up(a), len(a), ctypes.byref(f)))
        return f.value


def count_interference(X, phi) -> int:
    """FP64 operations the counting build of the oracle records for Algorithm 1 on one vector."""
    x = np.ascontiguousarray(X, dtype=np.float64)
    p = np.ascontiguousarray(phi, dtype=np.float64).reshape(64)
    f = ctypes.c_uint64()
    rc = lib().orc_count_interference(_dp(x), _dp(p), ctypes.byref(f))
    if rc != 0:
        raise RuntimeError("orc_count_interference failed")
    return f.value


def interference(X, phi) -> float:
    """Algorithm 1 on one 4-stream vector X with factors phi[16][4]."""
    x = np.ascontiguousarray(X, dtype=np.float64)
    p = np.ascontiguousarray(phi, dtype=np.float64).reshape(64)
    return lib().orc_interference(_dp(x), _dp(p))


# ---------------------------------------------------------------------------
# Process-parallel runs over disjoint group sets (each process single-threaded).
# ---------------------------------------------------------------------------
_worker_oracle = None


def _worker_init(wl):
    global _worker_oracle
    _worker_oracle = Oracle(wl)


def _worker_run(rng):
    g0, g1 = rng
    return g0, _worker_oracle.run(g0, g1)


def _worker_run_alpha(job):
    alphas, g0, g1 = job
    return g0, _worker_oracle.run_alpha(alphas, g0, g1)


def _worker_pareto(g):
    return g, _worker_oracle.pareto_exact(g)


def pareto_exact_groups(wl: dict, groups, procs: int = 1) -> dict:
    """Oracle.pareto_exact of each listed group (in fresh single-threaded processes when procs > 1):
    {group: result}."""
    groups = [int(g) for g in groups]
    if procs <= 1:
        o = Oracle(wl)
        return {g: o.pareto_exact(g) for g in groups}
    import multiprocessing as mp
    ctx = mp.get_context("spawn")
    with ctx.Pool(procs, initializer=_worker_init, initargs=(wl,)) as pool:
        return dict(pool.map(_worker_pareto, groups, chunksize=max(1, len(groups) // (8 * procs))))


def run_alpha_groups(wl: dict, alphas, groups, procs: int = 1) -> dict:
    """Oracle.run_alpha on the listed group indices; arrays in that order."""
    groups = [int(g) for g in groups]
    alphas = [float(a) for a in alphas]
    if procs <= 1:
        o = Oracle(wl)
        parts = [(g, o.run_alpha(alphas, g, g + 1)) for g in groups]
    else:
        import multiprocessing as mp
        ctx = mp.get_context("spawn")
        with ctx.Pool(procs, initializer=_worker_init, initargs=(wl,)) as pool:
            parts = pool.map(_worker_run_alpha, [(alphas, g, g + 1) for g in groups], chunksize=1)
    by = dict(parts)
    return {k: np.concatenate([by[g][k] for g in groups]) for k in ("id", "obj")}


def run_groups(wl: dict, groups, procs: int = 1) -> dict:
    """Runs the oracle on the listed group indices; returns arrays in that order."""
    groups = [int(g) for g in groups]
    ranges = [(g, g + 1) for g in groups]
    if procs <= 1:
        o = Oracle(wl)
        parts = [(g0, o.run(g0, g1)) for g0, g1 in ranges]
    else:
        import multiprocessing as mp
        ctx = mp.get_context("spawn")  # fresh interpreters: nothing inherited from a GPU process
        with ctx.Pool(procs, initializer=_worker_init, initargs=(wl,)) as pool:
            parts = pool.map(_worker_run, ranges, chunksize=1)
    by = dict(parts)
    keys = ["best_id", "best_obj", "bucket_id", "bucket_obj", "frontier"]
    return {k: np.concatenate([by[g][k] for g in groups]) for k in keys}
