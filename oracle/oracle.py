"""TEST INFRASTRUCTURE ONLY: ctypes wrapper of the plain-C oracle.

The oracle (``grand_oracle.c``) is a slow CPU implementation of the paper's
batched dynamic graph-index updates, used by the tests, the smoke check and
the benchmark's CPU-baseline leg to check the GPU library.  The GPU product
path never imports this module.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "grand_oracle.c")
LIB = os.path.join(HERE, "libgrand_oracle.so")
INVALID = 0xFFFFFFFF

OK, E_ARG, E_ID, E_CAPACITY = 0, -1, -2, -3

_lib = None


def build() -> str:
    """Compile the oracle with gcc (plain C11 + OpenMP)."""
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-ffp-contract=off", "-fopenmp",
           "-shared", "-fPIC", "-o", tmp, SRC, "-lm"]
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        build()
    lib = ctypes.CDLL(LIB)
    P, U32, I32, U64, F32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint64, ctypes.c_float
    lib.oracle_create.restype = P
    lib.oracle_create.argtypes = [P]
    lib.oracle_destroy.argtypes = [P]
    lib.oracle_last_error.restype = ctypes.c_char_p
    lib.oracle_last_error.argtypes = [P]
    lib.oracle_set_threads.argtypes = [P, I32]
    lib.oracle_get_stats.argtypes = [P, P]
    lib.oracle_insert_batch.restype = I32
    lib.oracle_insert_batch.argtypes = [P, P, P, U32]
    lib.oracle_delete_batch.restype = I32
    lib.oracle_delete_batch.argtypes = [P, P, U32]
    lib.oracle_search.restype = I32
    lib.oracle_search.argtypes = [P, P, U32, U32, U32, P, P]
    lib.oracle_export_graph.restype = I32
    lib.oracle_export_graph.argtypes = [P, P, P, P, P, P, P, P]
    lib.oracle_import_graph.restype = I32
    lib.oracle_import_graph.argtypes = [P, P, P, P, P, U32]
    lib.oracle_dist.restype = F32
    lib.oracle_dist.argtypes = [P, P, P]
    lib.oracle_beam_search.restype = U32
    lib.oracle_beam_search.argtypes = [P, P, U32, U32, U32, P, P, P, P, P]
    lib.oracle_store_row.restype = I32
    lib.oracle_store_row.argtypes = [P, P, P, I32]
    lib.oracle_robust_prune.restype = U32
    lib.oracle_robust_prune.argtypes = [P, U32, P, P, U32, P]
    lib.oracle_medoid.restype = U32
    lib.oracle_medoid.argtypes = [P]
    lib.oracle_reverse_csr.restype = U64
    lib.oracle_reverse_csr.argtypes = [P, P, U32, U32, P, P]
    lib.oracle_build_cagra.restype = I32
    lib.oracle_build_cagra.argtypes = [P, P, P, U32, P, U32, U32, U32]
    lib.oracle_nn_descent.restype = I32
    lib.oracle_nn_descent.argtypes = [P, P, U32, P, U32, U32, U32, P, P]
    lib.oracle_rank_prune.restype = None
    lib.oracle_rank_prune.argtypes = [P, U32, U32, U32, P]
    lib.oracle_reverse_merge.restype = None
    lib.oracle_reverse_merge.argtypes = [P, U32, U32, P, P]
    lib.oracle_bruteforce_knn.restype = I32
    lib.oracle_bruteforce_knn.argtypes = [P, P, U32, U32, P, P]
    _lib = lib
    return lib


class _Cfg(ctypes.Structure):
    _fields_ = [("algo", ctypes.c_int32), ("dtype", ctypes.c_int32), ("metric", ctypes.c_int32),
                ("prune_rule", ctypes.c_int32),
                ("dim", ctypes.c_uint32), ("capacity", ctypes.c_uint32), ("R", ctypes.c_uint32),
                ("L_build", ctypes.c_uint32), ("P", ctypes.c_uint32), ("c", ctypes.c_uint32),
                ("k_repair", ctypes.c_uint32), ("max_iters", ctypes.c_uint32),
                ("alpha", ctypes.c_float), ("threads", ctypes.c_int32), ("mips_norm", ctypes.c_float)]


class _Stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in
                ("searches", "hops", "dist_evals", "prunes", "dirty", "records", "cap_dropped")]


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def rank_prune(lists: np.ndarray, R: int) -> np.ndarray:
    """CAGRA rank-based pruning of ascending k-NN lists (n x K positions)."""
    lists = np.ascontiguousarray(lists, np.uint32)
    n, K = lists.shape
    out = np.empty((n, R), np.uint32)
    _load().oracle_rank_prune(_ptr(lists), n, K, R, _ptr(out))
    return out


def reverse_merge(P: np.ndarray):
    """CAGRA reverse-edge merge of pruned lists (n x R positions): (lists, lengths)."""
    P = np.ascontiguousarray(P, np.uint32)
    n, R = P.shape
    out = np.empty((n, R), np.uint32)
    nout = np.empty(n, np.uint32)
    _load().oracle_reverse_merge(_ptr(P), n, R, _ptr(out), _ptr(nout))
    return out, nout


def reverse_csr(adj: np.ndarray, active: np.ndarray):
    """Exact transpose of the out-lists of active nodes, rows ascending."""
    lib = _load()
    cap, R = adj.shape
    adj = np.ascontiguousarray(adj, np.uint32)
    active = np.ascontiguousarray(active, np.uint8)
    offs = np.zeros(cap + 1, np.uint32)
    nnz = lib.oracle_reverse_csr(_ptr(adj), _ptr(active), cap, R, _ptr(offs), None)
    srcs = np.zeros(max(int(nnz), 1), np.uint32)
    lib.oracle_reverse_csr(_ptr(adj), _ptr(active), cap, R, _ptr(offs), _ptr(srcs))
    return offs, srcs[: int(nnz)]


class Oracle:
    """One oracle index.  ``cfg`` is a ``workloads.IndexConfig``."""

    def __init__(self, cfg, threads: int = 0):
        self.lib = _load()
        self.cfg = cfg
        c = _Cfg(algo=1 if cfg.algo == "cagra" else 0, dtype=1 if cfg.dtype == "u8" else 0,
                 metric={"l2": 0, "ip": 1, "mips": 2}[cfg.metric], mips_norm=cfg.mips_norm,
                 prune_rule=1 if cfg.prune_rule == "alpha_on_l2" else 0,
                 dim=cfg.dim, capacity=cfg.capacity, R=cfg.R, L_build=cfg.L_build, P=cfg.P,
                 c=cfg.c, k_repair=cfg.k_repair, max_iters=cfg.iters, alpha=cfg.alpha,
                 threads=threads)
        self._c = c
        self.h = self.lib.oracle_create(ctypes.byref(c))
        if not self.h:
            raise ValueError("oracle_create rejected the configuration")
        self.np_dtype = np.uint8 if cfg.dtype == "u8" else np.float32

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            self.lib.oracle_destroy(h)
            self.h = None

    def set_threads(self, t: int):
        self.lib.oracle_set_threads(self.h, t)

    def last_error(self) -> str:
        return self.lib.oracle_last_error(self.h).decode()

    def _vecs(self, v):
        v = np.ascontiguousarray(v, self.np_dtype)
        assert v.ndim == 2 and v.shape[1] == self.cfg.dim
        return v

    def insert(self, ids, vecs) -> int:
        ids = np.ascontiguousarray(ids, np.uint32)
        vecs = self._vecs(vecs)
        return self.lib.oracle_insert_batch(self.h, _ptr(vecs), _ptr(ids), ids.size)

    def build_cagra(self, ids, vecs, init, knn: int, iters: int, sample: int) -> int:
        """CAGRA graph construction over an empty CAGRA index (NN-Descent,
        rank-based pruning, reverse edges); init is n x knn batch positions."""
        ids = np.ascontiguousarray(ids, np.uint32)
        vecs = self._vecs(vecs)
        init = np.ascontiguousarray(init, np.uint32)
        assert init.shape == (ids.size, knn)
        return self.lib.oracle_build_cagra(self.h, _ptr(vecs), _ptr(ids), ids.size, _ptr(init), knn, iters, sample)

    def nn_descent(self, vecs, init, knn: int, iters: int, sample: int):
        """NN-Descent alone over positions 0..n-1 (an empty index's rows 0..n-1
        are overwritten); returns (ids, dists), each n x knn, ascending."""
        vecs = self._vecs(vecs)
        init = np.ascontiguousarray(init, np.uint32)
        n = vecs.shape[0]
        assert init.shape == (n, knn)
        ids = np.empty((n, knn), np.uint32)
        d = np.empty((n, knn), np.float32)
        rc = self.lib.oracle_nn_descent(self.h, _ptr(vecs), n, _ptr(init), knn, iters, sample, _ptr(ids), _ptr(d))
        if rc != 0:
            raise ValueError(self.last_error())
        return ids, d

    def delete(self, ids) -> int:
        ids = np.ascontiguousarray(ids, np.uint32)
        return self.lib.oracle_delete_batch(self.h, _ptr(ids), ids.size)

    def search(self, queries, k: int, beam: int):
        q = self._vecs(queries)
        nq = q.shape[0]
        ids = np.zeros((nq, k), np.uint32)
        d = np.zeros((nq, k), np.float32)
        rc = self.lib.oracle_search(self.h, _ptr(q), nq, k, beam, _ptr(ids), _ptr(d))
        if rc:
            raise ValueError(f"oracle_search: {rc} {self.last_error()}")
        return ids, d

    def export(self, with_reverse: bool = False) -> dict:
        cap, R = self.cfg.capacity, self.cfg.R
        adj = np.zeros((cap, R), np.uint32)
        deg = np.zeros(cap, np.uint32)
        act = np.zeros(cap, np.uint8)
        med = np.zeros(1, np.uint32)
        self.lib.oracle_export_graph(self.h, _ptr(adj), _ptr(deg), _ptr(act), _ptr(med), None, None, None)
        out = dict(adj=adj, deg=deg, active=act, medoid=int(med[0]))
        if with_reverse:
            out["rev_offsets"], out["rev_srcs"] = reverse_csr(adj, act)
        return out

    def import_graph(self, vecs, adj, deg, active, medoid: int):
        vecs = self._vecs(vecs)
        adj = np.ascontiguousarray(adj, np.uint32)
        deg = np.ascontiguousarray(deg, np.uint32)
        active = np.ascontiguousarray(active, np.uint8)
        assert vecs.shape[0] == self.cfg.capacity and adj.shape == (self.cfg.capacity, self.cfg.R)
        self.lib.oracle_import_graph(self.h, _ptr(vecs), _ptr(adj), _ptr(deg), _ptr(active), medoid)

    def dist(self, a, b) -> float:
        a = np.ascontiguousarray(a, self.np_dtype)
        b = np.ascontiguousarray(b, self.np_dtype)
        return float(self.lib.oracle_dist(self.h, _ptr(a), _ptr(b)))

    def beam_search(self, q, start: int, ell: int, max_iters: int):
        q = np.ascontiguousarray(q, self.np_dtype)
        R = self.cfg.R
        C_ids = np.zeros(ell + R + 1, np.uint32)
        C_d = np.zeros(ell + R + 1, np.float32)
        V_ids = np.zeros(max_iters + 1, np.uint32)
        V_d = np.zeros(max_iters + 1, np.float32)
        nV = np.zeros(1, np.uint32)
        nC = self.lib.oracle_beam_search(self.h, _ptr(q), start, ell, max_iters, _ptr(C_ids), _ptr(C_d),
                                         _ptr(V_ids), _ptr(V_d), _ptr(nV))
        n = int(nV[0])
        return C_ids[:nC], C_d[:nC], V_ids[:n], V_d[:n]

    def store_row(self, x, is_query: bool = False):
        """A caller row in its stored form (the MIPS augmentation appends one
        coordinate); returns (row, status)."""
        x = np.ascontiguousarray(x, self.np_dtype)
        sdim = self.cfg.dim + (1 if self.cfg.metric == "mips" else 0)
        out = np.zeros(sdim, self.np_dtype)
        rc = self.lib.oracle_store_row(self.h, _ptr(x), _ptr(out), 1 if is_query else 0)
        return out, rc

    def robust_prune(self, p: int, ids, D) -> np.ndarray:
        ids = np.ascontiguousarray(ids, np.uint32)
        D = np.ascontiguousarray(D, np.float32)
        L = np.zeros(self.cfg.R, np.uint32)
        n = self.lib.oracle_robust_prune(self.h, p, _ptr(ids), _ptr(D), ids.size, _ptr(L))
        return L[:n]

    def medoid(self) -> int:
        return int(self.lib.oracle_medoid(self.h))

    def bruteforce_knn(self, queries, k: int):
        q = self._vecs(queries)
        nq = q.shape[0]
        ids = np.zeros((nq, k), np.uint32)
        d = np.zeros((nq, k), np.float32)
        self.lib.oracle_bruteforce_knn(self.h, _ptr(q), nq, k, _ptr(ids), _ptr(d))
        return ids, d

    def stats(self) -> dict:
        s = _Stats()
        self.lib.oracle_get_stats(self.h, ctypes.byref(s))
        return {n: int(getattr(s, n)) for n, _ in s._fields_}
