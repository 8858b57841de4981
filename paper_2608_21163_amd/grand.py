"""Thin ctypes binding of libgrand.so (the C ABI in include/grand.h).

Argument marshalling only: every step of the update and search path runs in
the library's HIP kernels.  Arrays may be numpy arrays (host memory) or
torch tensors (host or device memory); device tensors are passed by their
data pointer, and the library runs on torch's current HIP stream.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgrand.so")
INVALID = 0xFFFFFFFF

OK, E_ARG, E_ID, E_CAPACITY, E_DEVICE, E_OOM, E_STATE = 0, -1, -2, -3, -4, -5, -6
VAMANA, CAGRA = 0, 1
F32, U8 = 0, 1
L2, IP, MIPS = 0, 1, 2
ALPHA_ON_DIST, ALPHA_ON_L2 = 0, 1
CAS_GROUPED, CAS_RACING = 0, 1
REV_FULL, REV_BATCH = 0, 1
INDEG_SCAN, INDEG_REV_BATCH, INDEG_REV_FULL = 0, 1, 2
STATIC_SCRATCH_BYTES = 8 << 20   # GRAND_STATIC_SCRATCH_BYTES

PHASES = ["validate", "stage", "search_insert", "bootstrap", "prune_fwd", "group", "rebuild", "search_delete",
          "reverse", "repair", "clear", "medoid", "search_query", "cagra_detour", "cagra_pickone"]

EXPORTED = ["grand_default_params", "grand_create", "grand_destroy", "grand_set_stream", "grand_insert_batch",
            "grand_build_cagra", "grand_delete_batch", "grand_search", "grand_search_static", "grand_count_in_edges", "grand_reader_create",
            "grand_reader_search", "grand_reader_destroy", "grand_reader_last_error", "grand_export_graph", "grand_import_graph", "grand_set_timing",
            "grand_set_counting", "grand_stats", "grand_reset_stats", "grand_last_error"]


class GrandError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"grand status {code}: {msg}")
        self.code = code


class Params(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("algo", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("metric", ctypes.c_int32), ("dim", ctypes.c_uint32), ("capacity", ctypes.c_uint32),
                ("R", ctypes.c_uint32), ("L_build", ctypes.c_uint32), ("P", ctypes.c_uint32),
                ("c", ctypes.c_uint32), ("k_repair", ctypes.c_uint32), ("max_iters", ctypes.c_uint32),
                ("alpha", ctypes.c_float), ("prune_rule", ctypes.c_int32), ("cas_mode", ctypes.c_int32),
                ("rev_mode", ctypes.c_int32), ("max_batch", ctypes.c_uint32), ("mips_norm", ctypes.c_float),
                ("device", ctypes.c_int32),
                ("stream", ctypes.c_void_p)]


class Stats(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("timing_enabled", ctypes.c_uint32),
                ("inserted", ctypes.c_uint64), ("deleted", ctypes.c_uint64), ("queried", ctypes.c_uint64),
                ("search_hops", ctypes.c_uint64 * 3), ("search_evals", ctypes.c_uint64 * 3),
                ("fwd_evals", ctypes.c_uint64), ("fwd_prunes", ctypes.c_uint64),
                ("rebuild_evals", ctypes.c_uint64), ("rebuild_prunes", ctypes.c_uint64), ("dirty", ctypes.c_uint64),
                ("rebuild_records", ctypes.c_uint64), ("records", ctypes.c_uint64), ("rev_edges", ctypes.c_uint64),
                ("repair_evals", ctypes.c_uint64), ("rebuild_rows", ctypes.c_uint64),
                ("repair_rows", ctypes.c_uint64), ("repair_records", ctypes.c_uint64),
                ("search_distinct", ctypes.c_uint64 * 3), ("search_capped", ctypes.c_uint64 * 3),
                ("phase_ms", ctypes.c_double * len(PHASES)), ("phase_calls", ctypes.c_uint64 * len(PHASES))]


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads libgrand.so; raises if it has not been built (there is no
    fallback implementation)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2608_21163_amd/build.py")
    # One HIP runtime per process: torch ships its own libamdhip64 with the
    # same soname as the system one libgrand.so links.  Loading torch first
    # makes libgrand bind to torch's copy; loading libgrand first would pull
    # in the system copy, and torch's later initialisation then finds no GPU.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    P, U32, I32, U64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint64
    lib.grand_default_params.argtypes = [P]
    lib.grand_create.argtypes = [P, P]
    lib.grand_destroy.argtypes = [P]
    lib.grand_set_stream.argtypes = [P, P]
    lib.grand_insert_batch.argtypes = [P, P, P, U32]
    lib.grand_build_cagra.restype = I32
    lib.grand_build_cagra.argtypes = [P, P, P, U32, P, U32, U32, U32]
    lib.grand_delete_batch.argtypes = [P, P, U32]
    lib.grand_search.argtypes = [P, P, U32, U32, U32, P, P]
    lib.grand_search_static.argtypes = [P, P, U32, U32, U32, P, P]
    lib.grand_count_in_edges.argtypes = [P, P, U32, I32, P, P]
    lib.grand_reader_create.argtypes = [P, P, P]
    lib.grand_reader_search.argtypes = [P, P, U32, U32, U32, P, P]
    lib.grand_reader_destroy.argtypes = [P]
    lib.grand_reader_last_error.argtypes = [P]
    lib.grand_reader_last_error.restype = ctypes.c_char_p
    lib.grand_export_graph.argtypes = [P, P, P, P, P, P, P, P]
    lib.grand_import_graph.argtypes = [P, P, P, P, P, U32]
    lib.grand_set_timing.argtypes = [P, I32]
    lib.grand_set_counting.argtypes = [P, I32]
    lib.grand_stats.argtypes = [P, P, ctypes.c_size_t]
    lib.grand_reset_stats.argtypes = [P]
    lib.grand_last_error.argtypes = [P]
    lib.grand_last_error.restype = ctypes.c_char_p
    for name in EXPORTED:
        if name not in ("grand_default_params", "grand_last_error", "grand_reader_last_error"):
            getattr(lib, name).restype = I32
    _lib = lib
    return lib


def _is_torch(x) -> bool:
    return type(x).__module__.startswith("torch")


def _ptr(x):
    """Data pointer of a numpy array or torch tensor (must be contiguous)."""
    if x is None:
        return None
    if _is_torch(x):
        assert x.is_contiguous()
        return x.data_ptr()
    assert x.flags["C_CONTIGUOUS"]
    return x.ctypes.data


def _np(x, dtype):
    return np.ascontiguousarray(x, dtype=dtype)


def params_from_config(cfg, device: int = 0, max_batch: int = 10000, rev_mode: int = REV_BATCH) -> Params:
    """grand_params from a workloads.IndexConfig."""
    p = Params()
    load_library().grand_default_params(ctypes.byref(p))
    p.algo = CAGRA if cfg.algo == "cagra" else VAMANA
    p.dtype = U8 if cfg.dtype == "u8" else F32
    p.metric = {"l2": L2, "ip": IP, "mips": MIPS}[cfg.metric]
    p.mips_norm = getattr(cfg, "mips_norm", 0.0)
    p.dim, p.capacity, p.R, p.L_build = cfg.dim, cfg.capacity, cfg.R, cfg.L_build
    p.P, p.c, p.k_repair, p.max_iters = cfg.P, cfg.c, cfg.k_repair, cfg.max_iters
    p.alpha = cfg.alpha
    p.prune_rule = ALPHA_ON_L2 if cfg.prune_rule == "alpha_on_l2" else ALPHA_ON_DIST
    p.cas_mode = CAS_RACING if cfg.cas_mode == "racing" else CAS_GROUPED
    p.rev_mode = rev_mode
    p.max_batch = max_batch
    p.device = device
    return p


class Reader:
    """grand_reader_create ... grand_reader_destroy: searches that may run on
    another host thread while the index is updated (ctypes releases the
    GIL during the call)."""

    def __init__(self, index: "GrandIndex", stream: Optional[int] = None):
        self.lib = index.lib
        self.index = index
        h = ctypes.c_void_p()
        rc = self.lib.grand_reader_create(index.h, None if stream is None else ctypes.c_void_p(stream),
                                          ctypes.byref(h))
        if rc != OK:
            raise GrandError(rc, index.last_error())
        self.h = h

    def search(self, queries, k: int, beam: int, out_ids=None, out_dists=None):
        if not _is_torch(queries):
            queries = _np(queries, self.index.np_dtype)
        nq = int(queries.shape[0])
        if out_ids is None:
            out_ids = np.zeros((nq, k), np.uint32)
            out_dists = np.zeros((nq, k), np.float32)
        rc = self.lib.grand_reader_search(self.h, _ptr(queries), nq, k, beam, _ptr(out_ids), _ptr(out_dists))
        if rc != OK:
            raise GrandError(rc, self.lib.grand_reader_last_error(self.h).decode())
        return out_ids, out_dists

    def close(self):
        if getattr(self, "h", None):
            self.lib.grand_reader_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class GrandIndex:
    """One index on one GPU (grand_create ... grand_destroy)."""

    def __init__(self, params: Params, stream: Optional[int] = None):
        self.lib = load_library()
        self.params = params
        if stream is not None:
            params.stream = stream
        h = ctypes.c_void_p()
        rc = self.lib.grand_create(ctypes.byref(params), ctypes.byref(h))
        if rc != OK:
            raise GrandError(rc, "grand_create failed")
        self.h = h
        self.np_dtype = np.uint8 if params.dtype == U8 else np.float32

    @classmethod
    def from_config(cls, cfg, **kw):
        stream = kw.pop("stream", None)
        return cls(params_from_config(cfg, **kw), stream=stream)

    def close(self):
        if getattr(self, "h", None):
            self.lib.grand_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, rc: int) -> int:
        if rc != OK:
            raise GrandError(rc, self.last_error())
        return rc

    def last_error(self) -> str:
        return self.lib.grand_last_error(self.h).decode()

    def set_stream(self, stream: int):
        self._check(self.lib.grand_set_stream(self.h, ctypes.c_void_p(stream)))

    def insert(self, ids, vecs, check: bool = True) -> int:
        if not _is_torch(ids):
            ids = _np(ids, np.uint32)
        if not _is_torch(vecs):
            vecs = _np(vecs, self.np_dtype)
        n = int(ids.shape[0])
        rc = self.lib.grand_insert_batch(self.h, _ptr(vecs), _ptr(ids), n)
        return self._check(rc) if check else rc

    def build_cagra(self, ids, vecs, init, knn: int, iters: int, sample: int, check: bool = True) -> int:
        """CAGRA graph construction over this empty CAGRA index; init is
        n x knn batch positions (the random initial neighbour lists)."""
        if not _is_torch(ids):
            ids = _np(ids, np.uint32)
        if not _is_torch(vecs):
            vecs = _np(vecs, self.np_dtype)
        if not _is_torch(init):
            init = _np(init, np.uint32)
        n = int(ids.shape[0])
        if tuple(init.shape) != (n, knn):
            raise ValueError("init must be n x knn")
        rc = self.lib.grand_build_cagra(self.h, _ptr(vecs), _ptr(ids), n, _ptr(init), knn, iters, sample)
        return self._check(rc) if check else rc

    def delete(self, ids, check: bool = True) -> int:
        if not _is_torch(ids):
            ids = _np(ids, np.uint32)
        rc = self.lib.grand_delete_batch(self.h, _ptr(ids), int(ids.shape[0]))
        return self._check(rc) if check else rc

    def search(self, queries, k: int, beam: int, out_ids=None, out_dists=None):
        """Returns (ids, dists); with out_* given (e.g. device tensors) the
        results are written there."""
        if not _is_torch(queries):
            queries = _np(queries, self.np_dtype)
        nq = int(queries.shape[0])
        if out_ids is None:
            out_ids = np.zeros((nq, k), np.uint32)
            out_dists = np.zeros((nq, k), np.float32)
        self._check(self.lib.grand_search(self.h, _ptr(queries), nq, k, beam, _ptr(out_ids), _ptr(out_dists)))
        return out_ids, out_dists

    def search_static(self, queries, k: int, beam: int, out_ids=None, out_dists=None, check: bool = True):
        """grand_search_static: the search without any device allocation.
        Returns (ids, dists), or the status code when check is False."""
        if not _is_torch(queries):
            queries = _np(queries, self.np_dtype)
        nq = int(queries.shape[0])
        if out_ids is None:
            out_ids = np.zeros((nq, k), np.uint32)
            out_dists = np.zeros((nq, k), np.float32)
        rc = self.lib.grand_search_static(self.h, _ptr(queries), nq, k, beam, _ptr(out_ids), _ptr(out_dists))
        if not check:
            return rc
        self._check(rc)
        return out_ids, out_dists

    def count_in_edges(self, ids, method: int):
        """grand_count_in_edges: (counts, GPU milliseconds of the method)."""
        ids = _np(ids, np.uint32)
        out = np.zeros(ids.shape[0], np.uint32)
        ms = ctypes.c_float(0.0)
        self._check(self.lib.grand_count_in_edges(self.h, _ptr(ids), ids.shape[0], method, _ptr(out),
                                                  ctypes.byref(ms)))
        return out, float(ms.value)

    def search_rc(self, queries, k: int, beam: int) -> int:
        q = _np(queries, self.np_dtype)
        ids = np.zeros((max(q.shape[0], 1), max(k, 1)), np.uint32)
        d = np.zeros_like(ids, dtype=np.float32)
        return self.lib.grand_search(self.h, _ptr(q), q.shape[0], k, beam, _ptr(ids), _ptr(d))

    def export(self, with_reverse: bool = False) -> dict:
        p = self.params
        cap, R = p.capacity, p.R
        adj = np.zeros((cap, R), np.uint32)
        deg = np.zeros(cap, np.uint32)
        act = np.zeros(cap, np.uint8)
        med = np.zeros(1, np.uint32)
        out = dict(adj=adj, deg=deg, active=act)
        if with_reverse:
            offs = np.zeros(cap + 1, np.uint32)
            nnz = np.zeros(1, np.uint64)
            self._check(self.lib.grand_export_graph(self.h, _ptr(adj), _ptr(deg), _ptr(act), _ptr(med), _ptr(offs),
                                                    None, _ptr(nnz)))
            srcs = np.zeros(max(int(nnz[0]), 1), np.uint32)
            self._check(self.lib.grand_export_graph(self.h, None, None, None, None, _ptr(offs), _ptr(srcs),
                                                    _ptr(nnz)))
            out["rev_offsets"] = offs
            out["rev_srcs"] = srcs[: int(nnz[0])]
        else:
            self._check(self.lib.grand_export_graph(self.h, _ptr(adj), _ptr(deg), _ptr(act), _ptr(med), None, None,
                                                    None))
        out["medoid"] = int(med[0])
        return out

    def import_graph(self, vecs, adj, deg, active, medoid: int):
        if not _is_torch(vecs):
            vecs = _np(vecs, self.np_dtype)
        self._check(self.lib.grand_import_graph(self.h, _ptr(vecs), _ptr(_np(adj, np.uint32)),
                                                _ptr(_np(deg, np.uint32)), _ptr(_np(active, np.uint8)),
                                                int(medoid)))

    def set_timing(self, on: bool = True):
        self._check(self.lib.grand_set_timing(self.h, 1 if on else 0))

    def set_counting(self, on: bool = True):
        self._check(self.lib.grand_set_counting(self.h, 1 if on else 0))

    def reset_stats(self):
        self._check(self.lib.grand_reset_stats(self.h))

    def stats(self) -> dict:
        s = Stats()
        self._check(self.lib.grand_stats(self.h, ctypes.byref(s), ctypes.sizeof(Stats)))
        arrays = ("search_hops", "search_evals", "search_distinct", "search_capped", "phase_ms", "phase_calls")
        out = {n: getattr(s, n) for n, _ in Stats._fields_ if n not in arrays}
        for i, w in enumerate(("insert", "delete", "query")):
            out[f"hops_{w}"] = s.search_hops[i]
            out[f"evals_{w}"] = s.search_evals[i]
            out[f"distinct_{w}"] = s.search_distinct[i]
            out[f"capped_{w}"] = s.search_capped[i]
        out["phase_ms"] = {n: s.phase_ms[i] for i, n in enumerate(PHASES)}
        out["phase_calls"] = {n: s.phase_calls[i] for i, n in enumerate(PHASES)}
        return out
