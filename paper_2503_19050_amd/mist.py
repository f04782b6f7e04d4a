"""Python binding of libmist (include/mist.h): argument marshalling only.

Every step of the tuner's hot path runs inside libmist.so (host space build and HIP
kernels on the GPU).  PyTorch provides device memory (its caching allocator, through the
library's allocator callbacks) and the stream.  If the library is missing this module
raises; there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
import threading

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmist.so")

MIST_NONE = 0xFFFFFFFFFFFFFFFF
NONE = np.uint64(MIST_NONE)

EXPORTS = [
    "mist_space_create", "mist_eval_space", "mist_get_best", "mist_get_pareto", "mist_get_alpha",
    "mist_get_buckets",
    "mist_space_info", "mist_get_group_key", "mist_decode", "mist_eval_ids", "mist_set_timing",
    "mist_read_timing", "mist_launch_info", "mist_space_destroy", "mist_last_error",
    "mist_plan_points", "mist_plan_pipeline", "mist_eval_pareto_exact", "mist_get_pareto_exact", "mist_exact_info",
    "mist_corun_create", "mist_corun_run", "mist_corun_reduce", "mist_corun_measure", "mist_corun_destroy",
    "mist_fit_phi", "mist_interference", "mist_measure_eta", "mist_probe_fp64",
    "mist_tile_info", "mist_debug_eval_tiles", "mist_eval_ids_noalloc", "mist_exact_group_sizes",
]

PROBE_KINDS = {"add": 0, "mul": 1, "fma": 2, "min": 3, "max": 4, "cmp": 5}


class MistError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("libmist status %d: %s" % (status, msg))
        self.status = status


class ModelDesc(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int64),
                ("heads", ctypes.c_int32), ("kv_heads", ctypes.c_int32), ("ffn", ctypes.c_int64),
                ("seq", ctypes.c_int64), ("vocab", ctypes.c_int64), ("bytes_w", ctypes.c_int32),
                ("bytes_opt", ctypes.c_int32), ("flash", ctypes.c_int32)]


class HwDesc(ctypes.Structure):
    _fields_ = [("flops", ctypes.c_double), ("mem_bytes", ctypes.c_double), ("pcie_bw", ctypes.c_double),
                ("link_bw", ctypes.c_double), ("eta_max", ctypes.c_double), ("n_half", ctypes.c_double),
                ("phi", (ctypes.c_double * 4) * 16), ("eta_tab", ctypes.c_double * 16)]


class SpaceDesc(ctypes.Structure):
    _fields_ = [("n_devices", ctypes.c_int64), ("global_batch", ctypes.c_int64),
                ("mb", ctypes.POINTER(ctypes.c_int32)), ("n_mb", ctypes.c_int32),
                ("ratios", ctypes.POINTER(ctypes.c_double)), ("n_ratios", ctypes.c_int32),
                ("n_buckets", ctypes.c_int32), ("l_rule", ctypes.c_int32),
                ("n_alphas", ctypes.c_int32), ("alphas", ctypes.POINTER(ctypes.c_double)),
                ("tile_configs", ctypes.c_int64), ("max_blocks", ctypes.c_int32),
                ("cand_window", ctypes.c_int32)]


MAX_STAGES = 64
CORUN_MAX_UNITS = 256
CORUN_SAMPLES_PER_SHAPE = 28


class CorunShape(ctypes.Structure):
    _fields_ = [("gemm_m", ctypes.c_int64), ("gemm_n", ctypes.c_int64), ("gemm_k", ctypes.c_int64),
                ("g2g_bytes", ctypes.c_int64), ("h2d_bytes", ctypes.c_int64), ("d2h_bytes", ctypes.c_int64)]


class CorunSample(ctypes.Structure):
    _fields_ = [("mask", ctypes.c_int32), ("stream", ctypes.c_int32), ("shape", ctypes.c_int32),
                ("units", ctypes.c_int32), ("solo_s", ctypes.c_double), ("corun_s", ctypes.c_double)]


class StagePoint(ctypes.Structure):
    _fields_ = [("G", ctypes.c_int32), ("PP", ctypes.c_int32), ("k", ctypes.c_int32), ("l", ctypes.c_int32),
                ("id", ctypes.c_uint64), ("t", ctypes.c_double), ("d", ctypes.c_double)]


class StagePlan(ctypes.Structure):
    _fields_ = [("l", ctypes.c_int32), ("k", ctypes.c_int32), ("id", ctypes.c_uint64),
                ("t", ctypes.c_double), ("d", ctypes.c_double)]


class Plan(ctypes.Structure):
    _fields_ = [("found", ctypes.c_int32), ("hw", ctypes.c_int32), ("G", ctypes.c_int32), ("PP", ctypes.c_int32),
                ("F", ctypes.c_double), ("stage", StagePlan * MAX_STAGES)]


def _plan_dict(p: Plan) -> dict | None:
    if not p.found:
        return None
    return {"hw": p.hw, "G": p.G, "PP": p.PP, "F": p.F,
            "stages": [_struct_to_dict(p.stage[i]) for i in range(p.PP)]}


ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)
FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)


class Allocator(ctypes.Structure):
    _fields_ = [("alloc", ALLOC_FN), ("free", FREE_FN), ("ctx", ctypes.c_void_p)]


class Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ["hw", "G", "PP", "k", "l", "b", "tp", "dp", "zero", "ckpt",
                 "wo_idx", "go_idx", "oo_idx", "ao_idx"]] + \
               [(n, ctypes.c_double) for n in ["wo", "go", "oo", "ao"]]


class Result(ctypes.Structure):
    _fields_ = [("id", ctypes.c_uint64), ("obj", ctypes.c_double), ("t", ctypes.c_double),
                ("d", ctypes.c_double), ("mem", ctypes.c_double), ("bucket", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("cfg", Config)]


class GroupKey(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ["hw", "G", "PP", "k", "l", "n_pairs"]] + \
               [("base", ctypes.c_uint64), ("size", ctypes.c_uint64)]


_lib = None
_lock = threading.Lock()


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libmist.so (built by paper_2503_19050_amd.build); raises when it is missing."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(path):
            raise MistError(-3, "%s is not built; run paper_2503_19050_amd.build.build()" % path)
        L = ctypes.CDLL(path)
        P = ctypes.POINTER
        st = ctypes.c_int32
        vp = ctypes.c_void_p
        L.mist_space_create.argtypes = [P(ModelDesc), P(HwDesc), ctypes.c_int32, P(SpaceDesc), P(Allocator), P(vp)]
        L.mist_eval_space.argtypes = [vp, vp]
        L.mist_get_best.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, P(Result)]
        L.mist_get_pareto.argtypes = [vp, ctypes.c_int64, P(Result), ctypes.c_int32, P(ctypes.c_int32)]
        L.mist_get_alpha.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, P(Result)]
        L.mist_get_buckets.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, P(ctypes.c_uint64),
                                       P(ctypes.c_double), P(ctypes.c_uint64)]
        L.mist_space_info.argtypes = [vp, P(ctypes.c_uint64), P(ctypes.c_int64), P(ctypes.c_int32)]
        L.mist_get_group_key.argtypes = [vp, ctypes.c_int64, P(GroupKey)]
        L.mist_decode.argtypes = [vp, ctypes.c_uint64, P(Config)]
        L.mist_eval_ids.argtypes = [vp, P(ctypes.c_uint64), ctypes.c_int64, P(ctypes.c_double), vp]
        L.mist_eval_ids_noalloc.argtypes = [vp, P(ctypes.c_uint64), ctypes.c_int64, P(ctypes.c_double), vp]
        L.mist_set_timing.argtypes = [vp, ctypes.c_int32]
        L.mist_read_timing.argtypes = [vp, P(ctypes.c_double), P(ctypes.c_double), P(ctypes.c_int64)]
        L.mist_launch_info.argtypes = [vp, P(ctypes.c_int64), P(ctypes.c_int32), P(ctypes.c_int32)]
        L.mist_space_destroy.argtypes = [vp]
        L.mist_eval_pareto_exact.argtypes = [vp, vp]
        L.mist_get_pareto_exact.argtypes = [vp, ctypes.c_int64, P(Result), ctypes.c_int64, P(ctypes.c_int64)]
        L.mist_exact_group_sizes.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, P(ctypes.c_int64), P(ctypes.c_int64)]
        L.mist_exact_info.argtypes = [vp, P(ctypes.c_int64), P(ctypes.c_int64), P(ctypes.c_int32), P(ctypes.c_int32)]
        L.mist_plan_points.argtypes = [P(StagePoint), ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P(Plan)]
        L.mist_plan_pipeline.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, P(Plan)]
        dp = P(ctypes.c_double)
        ip = P(ctypes.c_int32)
        L.mist_corun_create.argtypes = [P(CorunShape), ctypes.c_int32, P(vp)]
        L.mist_corun_run.argtypes = [vp, ctypes.c_int32, P(CorunShape), ip, dp, ctypes.c_int32]
        L.mist_corun_reduce.argtypes = [ctypes.c_int32, dp, ctypes.c_int32, ip, dp, ip]
        L.mist_corun_measure.argtypes = [vp, P(CorunShape), ctypes.c_int32, ctypes.c_double, P(CorunSample),
                                         ctypes.c_int32, ip]
        L.mist_corun_destroy.argtypes = [vp]
        L.mist_fit_phi.argtypes = [P(CorunSample), ctypes.c_int64, dp]
        L.mist_interference.argtypes = [dp, dp, dp]
        L.mist_measure_eta.argtypes = [P(ModelDesc), ip, ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
                                       ctypes.c_int32, dp, dp]
        L.mist_tile_info.argtypes = [vp, ctypes.c_int32, P(ctypes.c_int64), P(ctypes.c_uint64), P(ctypes.c_int64)]
        L.mist_debug_eval_tiles.argtypes = [vp, P(ctypes.c_int32), ctypes.c_int32, P(ctypes.c_double),
                                            ctypes.c_int64, vp]
        L.mist_probe_fp64.argtypes = [ctypes.c_int32, vp, vp, ctypes.c_int64, ctypes.c_int32, P(ctypes.c_uint64), vp]
        L.mist_last_error.restype = ctypes.c_char_p
        for name in EXPORTS:
            if name != "mist_last_error":
                getattr(L, name).restype = st
        _lib = L
        return L


def _check(L, rc):
    if rc != 0:
        raise MistError(rc, L.mist_last_error().decode())


def _struct_to_dict(s) -> dict:
    out = {}
    for name, _ in s._fields_:
        v = getattr(s, name)
        out[name] = _struct_to_dict(v) if isinstance(v, ctypes.Structure) else v
    return out


def _results_to_dicts(out, n: int) -> list[dict]:
    """mist_result array -> list of dicts, through one numpy view (no per-field ctypes access)."""
    if n == 0:
        return []
    rows = np.ctypeslib.as_array(out)[:n].tolist()
    names = [f for f, _ in Result._fields_[:-1]]
    cnames = [f for f, _ in Config._fields_]
    return [dict(zip(names, r[:-1]), cfg=dict(zip(cnames, r[-1]))) for r in rows]


def _stream_handle(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Space:
    """A configuration space held by libmist on the current GPU.

    ``model``, ``hws`` and ``space`` are the descriptor dictionaries of
    ``paper_2503_19050_amd.workloads``.  ``allocator="torch"`` routes device memory through
    PyTorch's caching allocator; ``None`` lets the library use hipMalloc.
    """

    def __init__(self, model: dict, hws: list, space: dict, allocator: str | None = "torch"):
        self.L = load()
        self._model = ModelDesc(**{k: model[k] for k, _ in ModelDesc._fields_})
        self._hw = (HwDesc * len(hws))()
        for i, h in enumerate(hws):
            for k in ("flops", "mem_bytes", "pcie_bw", "link_bw", "eta_max", "n_half"):
                setattr(self._hw[i], k, float(h[k]))
            for m in range(16):
                for j in range(4):
                    self._hw[i].phi[m][j] = float(h["phi"][m][j])
            tab = [float(v) for v in h.get("eta_tab", [])]
            self._hw[i].eta_tab[:len(tab)] = tab
        self._mb = np.ascontiguousarray(space["mb"], dtype=np.int32)
        self._ratios = np.ascontiguousarray(space["ratios"], dtype=np.float64)
        self._alphas = np.ascontiguousarray(space.get("alphas", []), dtype=np.float64)
        self.n_alphas = len(self._alphas)
        self._space = SpaceDesc(space["n_devices"], space["global_batch"],
                                self._mb.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), len(self._mb),
                                self._ratios.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                len(self._ratios), space["n_buckets"], space["l_rule"], self.n_alphas,
                                self._alphas.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                int(space.get("tile_configs", 0)), int(space.get("max_blocks", 0)),
                                int(space.get("cand_window", 0)))
        self._alloc = None
        if allocator == "torch":
            self._alloc = self._torch_allocator()
        elif allocator is not None:
            raise ValueError("allocator must be 'torch' or None")
        h = ctypes.c_void_p()
        _check(self.L, self.L.mist_space_create(ctypes.byref(self._model), self._hw, len(hws),
                                                ctypes.byref(self._space),
                                                ctypes.byref(self._alloc) if self._alloc else None,
                                                ctypes.byref(h)))
        self.h = h
        n = ctypes.c_uint64()
        g = ctypes.c_int64()
        nb = ctypes.c_int32()
        _check(self.L, self.L.mist_space_info(self.h, ctypes.byref(n), ctypes.byref(g), ctypes.byref(nb)))
        self.n_configs, self.n_groups, self.n_buckets = n.value, g.value, nb.value

    def _torch_allocator(self):
        import torch
        device = torch.cuda.current_device()
        failures = self._alloc_failures = []

        def alloc(nbytes, stream, ctx):
            # the block joins the pool of the stream the library uses it on (NULL: the null stream)
            try:
                return torch.cuda.caching_allocator_alloc(int(nbytes), device, int(stream or 0))
            except Exception as e:  # no exception may cross the C ABI
                failures.append(e)
                return None

        def free(ptr, ctx):
            try:
                torch.cuda.caching_allocator_delete(ptr)
            except Exception as e:
                failures.append(e)

        self._cb = (ALLOC_FN(alloc), FREE_FN(free))
        return Allocator(self._cb[0], self._cb[1], None)

    # -- evaluation ---------------------------------------------------------------
    def eval(self, stream=None) -> None:
        """Enqueues the evaluation on ``stream`` (torch stream, raw handle, or current)."""
        _check(self.L, self.L.mist_eval_space(self.h, ctypes.c_void_p(_stream_handle(stream))))

    def set_timing(self, on: bool = True) -> None:
        _check(self.L, self.L.mist_set_timing(self.h, 1 if on else 0))

    def read_timing(self) -> tuple[float, float, int]:
        """(summed evaluation-kernel ms, summed reduction-kernel ms, evaluations) since the
        last read; waits for them."""
        a = ctypes.c_double()
        b = ctypes.c_double()
        n = ctypes.c_int64()
        _check(self.L, self.L.mist_read_timing(self.h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(n)))
        return a.value, b.value, n.value

    def launch_info(self) -> dict:
        t = ctypes.c_int64()
        b = ctypes.c_int32()
        u = ctypes.c_int32()
        _check(self.L, self.L.mist_launch_info(self.h, ctypes.byref(t), ctypes.byref(b), ctypes.byref(u)))
        return {"tiles": t.value, "block": b.value, "strips_per_tile": u.value}

    # -- results ------------------------------------------------------------------
    def best(self, g0: int = 0, n: int | None = None) -> list[dict]:
        n = self.n_groups - g0 if n is None else n
        return _results_to_dicts(self._best_raw(g0, n), n)

    def best_array(self, g0: int = 0, n: int | None = None) -> np.ndarray:
        """best() as a numpy structured array (the mist_result layout), without per-group dicts."""
        n = self.n_groups - g0 if n is None else n
        return np.ctypeslib.as_array(self._best_raw(g0, n))[:n]

    def _best_raw(self, g0: int, n: int):
        out = (Result * max(n, 1))()
        _check(self.L, self.L.mist_get_best(self.h, g0, n, out))
        return out

    def pareto(self, g: int) -> list[dict]:
        out = (Result * 64)()
        cnt = ctypes.c_int32()
        _check(self.L, self.L.mist_get_pareto(self.h, g, out, 64, ctypes.byref(cnt)))
        return _results_to_dicts(out, cnt.value)

    def eval_pareto_exact(self, stream=None) -> None:
        """Exact (non-bucketed) time-vs-memory frontier of every group; after eval()."""
        _check(self.L, self.L.mist_eval_pareto_exact(self.h, _stream_handle(stream)))

    def pareto_exact(self, g: int) -> list[dict]:
        """Group g's exact frontier in increasing memory (strictly decreasing objective)."""
        n = ctypes.c_int64()
        cap = 256
        while True:
            out = (Result * cap)()
            rc = self.L.mist_get_pareto_exact(self.h, g, out, cap, ctypes.byref(n))
            if rc == -5 and n.value > cap:
                cap = n.value
                continue
            _check(self.L, rc)
            return _results_to_dicts(out, n.value)

    def exact_group_sizes(self, g0: int = 0, n: int | None = None) -> tuple[np.ndarray, np.ndarray]:
        """Per-group candidates and pre-filter survivors of the last exact frontier."""
        n = self.n_groups - g0 if n is None else n
        c = np.zeros(max(n, 1), dtype=np.int64)
        k = np.zeros(max(n, 1), dtype=np.int64)
        P = ctypes.POINTER(ctypes.c_int64)
        _check(self.L, self.L.mist_exact_group_sizes(self.h, g0, n, c.ctypes.data_as(P), k.ctypes.data_as(P)))
        return c[:n], k[:n]

    def exact_info(self) -> dict:
        """Sizes of the last exact frontier: candidates, those the pre-filter kept, tiles the
        candidate pass evaluated, and tiles evaluated a second time."""
        c, k, v, t = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()
        _check(self.L, self.L.mist_exact_info(self.h, ctypes.byref(c), ctypes.byref(k), ctypes.byref(v),
                                              ctypes.byref(t)))
        return {"candidates": c.value, "kept": k.value, "tiles_live": v.value, "tiles_again": t.value}

    def plan(self, hw: int = 0, pp: int = 0) -> dict | None:
        """The inter-stage plan (Eq. 1-3) of hardware sample hw from this space's frontier
        points; pp = 0 allows every stage count.  None when no plan exists."""
        out = Plan()
        _check(self.L, self.L.mist_plan_pipeline(self.h, hw, pp, ctypes.byref(out)))
        return _plan_dict(out)

    def alpha(self, g0: int = 0, n: int | None = None) -> list[list[dict]]:
        """Per group g0..g0+n-1 and weight sample a: the feasible configuration minimising
        alpha_a*G*t + (1-alpha_a)*d (Eq. 4); obj holds that weighted value."""
        n = self.n_groups - g0 if n is None else n
        A = self.n_alphas
        out = (Result * max(n * A, 1))()
        _check(self.L, self.L.mist_get_alpha(self.h, g0, n, out))
        flat = _results_to_dicts(out, n * A)
        return [flat[i * A:(i + 1) * A] for i in range(n)]

    def buckets(self, g0: int = 0, n: int | None = None):
        """(ids[n, NB], objs[n, NB], frontier masks[n]) of groups g0..g0+n-1."""
        n = self.n_groups - g0 if n is None else n
        ids = np.empty((n, self.n_buckets), dtype=np.uint64)
        objs = np.empty((n, self.n_buckets), dtype=np.float64)
        masks = np.empty(n, dtype=np.uint64)
        _check(self.L, self.L.mist_get_buckets(self.h, g0, n,
                                               ids.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                                               objs.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                               masks.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))))
        return ids, objs, masks

    def eval_ids(self, ids, stream=None) -> np.ndarray:
        """Per-configuration (t, d, mem, obj) computed on the GPU."""
        ids = np.ascontiguousarray(ids, dtype=np.uint64)
        out = np.empty((len(ids), 4), dtype=np.float64)
        _check(self.L, self.L.mist_eval_ids(self.h, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                                            len(ids), out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                            ctypes.c_void_p(_stream_handle(stream))))
        return out

    def eval_ids_noalloc(self, ids, stream=None) -> np.ndarray:
        """eval_ids through the allocation-free entry point (at most 104,857 ids per call)."""
        ids = np.ascontiguousarray(ids, dtype=np.uint64)
        out = np.empty((len(ids), 4), dtype=np.float64)
        _check(self.L, self.L.mist_eval_ids_noalloc(self.h, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                                                    len(ids), out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                                    ctypes.c_void_p(_stream_handle(stream))))
        return out

    def tile_info(self, t: int) -> dict:
        g = ctypes.c_int64()
        f = ctypes.c_uint64()
        n = ctypes.c_int64()
        _check(self.L, self.L.mist_tile_info(self.h, t, ctypes.byref(g), ctypes.byref(f), ctypes.byref(n)))
        return {"group": g.value, "first_id": f.value, "n_configs": n.value}

    def debug_eval_tiles(self, tiles, stream=None) -> np.ndarray:
        """The evaluation kernel's own per-configuration values over the listed tiles: rows of
        (t, d, mem, obj, bucket entry, forms of Algorithm 1 as f1 + 8 * fs) in tile order, id
        order within a tile."""
        tl = np.ascontiguousarray(tiles, dtype=np.int32)
        total = sum(self.tile_info(int(t))["n_configs"] for t in tl)
        out = np.empty((max(total, 1), 6), dtype=np.float64)
        _check(self.L, self.L.mist_debug_eval_tiles(self.h, tl.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                                    len(tl), out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                                    total, _stream_handle(stream)))
        return out[:total]

    def decode(self, cid: int) -> dict:
        c = Config()
        _check(self.L, self.L.mist_decode(self.h, cid, ctypes.byref(c)))
        return _struct_to_dict(c)

    def group_key(self, g: int) -> dict:
        k = GroupKey()
        _check(self.L, self.L.mist_get_group_key(self.h, g, ctypes.byref(k)))
        return _struct_to_dict(k)

    def close(self) -> None:
        if getattr(self, "h", None):
            self.L.mist_space_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def from_workload(wl: dict, allocator: str | None = "torch") -> Space:
    return Space(wl["model"], wl["hws"], wl["space"], allocator=allocator)


def plan_points(points, n_layers: int, pp: int = 0) -> dict | None:
    """The host planner on explicit candidate points: an iterable of dicts with keys G, PP, k,
    l, id, t, d.  None when no plan exists."""
    L = load()
    pts = list(points)
    arr = (StagePoint * max(len(pts), 1))()
    for i, p in enumerate(pts):
        arr[i] = StagePoint(p["G"], p["PP"], p["k"], p["l"], p["id"], p["t"], p["d"])
    out = Plan()
    _check(L, L.mist_plan_points(arr, len(pts), n_layers, pp, ctypes.byref(out)))
    return _plan_dict(out)


# -- calibration ------------------------------------------------------------------------------
def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _iptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _shape(sh: dict) -> CorunShape:
    return CorunShape(*(int(sh[k]) for k, _ in CorunShape._fields_))


def corun_reduce(mask: int, t, units) -> tuple[np.ndarray, np.ndarray]:
    """mist_corun_reduce: t[j] are stream j's timestamps (seconds); returns (mean[4], count[4])."""
    L = load()
    u = np.zeros(4, dtype=np.int32)
    for j in range(4):
        u[j] = units[j]
    stride = int(max([u.max(), 1] + [len(x) - 1 for x in t])) + 1
    tt = np.zeros((4, stride))
    for j in range(4):
        if mask >> j & 1:
            tt[j, :len(t[j])] = t[j]
    mean = np.zeros(4)
    count = np.zeros(4, dtype=np.int32)
    _check(L, L.mist_corun_reduce(int(mask), _dptr(tt), stride, _iptr(u), _dptr(mean), _iptr(count)))
    return mean, count


def fit_phi(samples) -> np.ndarray:
    """mist_fit_phi: samples are (mask, stream, solo_s, corun_s) tuples or dicts; returns phi[16][4]."""
    L = load()
    arr = (CorunSample * max(len(samples), 1))()
    for i, x in enumerate(samples):
        if isinstance(x, dict):
            arr[i] = CorunSample(x["mask"], x["stream"], x.get("shape", 0), x.get("units", 0), x["solo_s"], x["corun_s"])
        else:
            arr[i] = CorunSample(int(x[0]), int(x[1]), 0, 0, float(x[2]), float(x[3]))
    phi = np.zeros(64)
    _check(L, L.mist_fit_phi(arr, len(samples), _dptr(phi)))
    return phi.reshape(16, 4)


def interference(phi, x) -> float:
    """mist_interference: Algorithm 1 on stream times x[4] with factors phi[16][4]."""
    L = load()
    p = np.ascontiguousarray(phi, dtype=np.float64).reshape(64)
    xx = np.ascontiguousarray(x, dtype=np.float64).reshape(4)
    out = ctypes.c_double()
    _check(L, L.mist_interference(_dptr(p), _dptr(xx), ctypes.byref(out)))
    return out.value


def probe_fp64(kind: str, n_threads: int, reps: int, stream=None) -> int:
    """Enqueues the FP64 instruction-mix probe of one kind (add, mul, fma, min, max, cmp) on the
    current (or given) stream; returns the wave-level count of the probed instruction."""
    import torch
    L = load()
    inp = torch.rand(2 * n_threads, dtype=torch.float64, device="cuda") + 0.5
    out = torch.empty(n_threads, dtype=torch.int64, device="cuda")
    n = ctypes.c_uint64()
    _check(L, L.mist_probe_fp64(PROBE_KINDS[kind], ctypes.c_void_p(inp.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                n_threads, reps, ctypes.byref(n), _stream_handle(stream)))
    torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
    return n.value


def measure_eta(model: dict, mb, tp: int, peak_flops: float, reps: int = 5) -> tuple[np.ndarray, np.ndarray]:
    """mist_measure_eta on the current device: (eta[i], seconds[i]) per microbatch size mb[i]."""
    L = load()
    m = ModelDesc(**{k: model[k] for k, _ in ModelDesc._fields_})
    b = np.ascontiguousarray(mb, dtype=np.int32)
    eta = np.zeros(len(b))
    sec = np.zeros(len(b))
    _check(L, L.mist_measure_eta(ctypes.byref(m), _iptr(b), len(b), int(tp), float(peak_flops), int(reps),
                                 _dptr(eta), _dptr(sec)))
    return eta, sec


class Corun:
    """The co-run benchmark's device state (mist_corun_create) on the current device."""

    def __init__(self, max_shape: dict, g2g_blocks: int = 16):
        self.L = load()
        h = ctypes.c_void_p()
        _check(self.L, self.L.mist_corun_create(ctypes.byref(_shape(max_shape)), int(g2g_blocks), ctypes.byref(h)))
        self.h = h

    def run(self, mask: int, shape: dict, units) -> list[np.ndarray]:
        """Timestamps (seconds after the common start) of each member's units."""
        u = np.zeros(4, dtype=np.int32)
        for j in range(4):
            u[j] = units[j]
        stride = CORUN_MAX_UNITS + 1
        t = np.zeros((4, stride))
        _check(self.L, self.L.mist_corun_run(self.h, int(mask), ctypes.byref(_shape(shape)), _iptr(u), _dptr(t),
                                             stride))
        return [t[j, :u[j] + 1].copy() if mask >> j & 1 else np.zeros(0) for j in range(4)]

    def measure(self, shapes, target_s: float = 0.02) -> list[dict]:
        arr = (CorunShape * len(shapes))(*[_shape(s) for s in shapes])
        cap = len(shapes) * CORUN_SAMPLES_PER_SHAPE
        out = (CorunSample * cap)()
        n = ctypes.c_int32()
        _check(self.L, self.L.mist_corun_measure(self.h, arr, len(shapes), float(target_s), out, cap,
                                                 ctypes.byref(n)))
        return [_struct_to_dict(out[i]) for i in range(n.value)]

    def close(self) -> None:
        if getattr(self, "h", None):
            _check(self.L, self.L.mist_corun_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
