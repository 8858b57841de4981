"""Seeded synthetic workloads shaped like the paper's streaming experiments.

The paper evaluates on real datasets (Section 5.1, Table 2) under streaming
patterns (Section 5.2).  None of those datasets is available here, so every
workload below is synthetic: a seeded Gaussian (or Student-t) mixture with
the dimensionality, element type and metric of the dataset it stands in for,
driven through an operation stream of uniform single-type batches as in
Section 5.2.

Everything is drawn from ``numpy.random.Generator(PCG64)`` seeded by
``SeedSequence([seed, purpose, index])`` so that every batch can be
regenerated independently of the others.  Id bookkeeping (which ids are
active, which are free) follows only the operation stream: fresh ids are the
smallest free ids in ascending order, and deleted ids become free again
(the pool of Section 4 reuses deleted ids).

This module contains no distance computation, search or pruning.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Iterator, List, Optional, Tuple

import numpy as np

INVALID = 0xFFFFFFFF

# purpose codes for SeedSequence entropy
_P_MODEL, _P_BASE, _P_INS, _P_DEL, _P_QRY = 1, 2, 3, 4, 5


def _rng(seed: int, purpose: int, index: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, purpose, index])))


@dataclass(frozen=True)
class IndexConfig:
    """Index parameters (Section 5.4 names l, alpha, P, k, c; R per workload)."""
    algo: str            # "vamana" | "cagra"
    dtype: str           # "f32" | "u8"
    metric: str          # "l2" | "ip" | "mips" (inner product through the L2 augmentation)
    dim: int
    capacity: int
    R: int
    L_build: int         # beam width of insert/delete searches (CAGRA: internal top-k)
    alpha: float = 1.2
    P: int = 64          # scratch capacity per node
    c: int = 2           # replacement edges per repaired neighbour
    k_repair: int = 50   # top-k of the delete search used for repair
    max_iters: int = 0   # expansion cap of build searches; 0 means 2 * L_build
    prune_rule: str = "alpha_on_sq"   # or "alpha_on_l2"
    cas_mode: str = "grouped"         # or "racing" (CAGRA insert only)
    mips_norm: float = 0.0            # metric "mips": the bound M on every vector norm

    @property
    def iters(self) -> int:
        return self.max_iters if self.max_iters > 0 else 2 * self.L_build

    def replace(self, **kw) -> "IndexConfig":
        return dataclasses.replace(self, **kw)


@dataclass(frozen=True)
class StreamSpec:
    base_n: int
    build_batch: int
    n_rounds: int
    n_insert: int
    n_delete: int
    n_query: int
    k: int
    beam: int
    order: Tuple[str, ...] = ("insert", "delete", "search")
    delete_policy: str = "uniform"    # "uniform" | "oldest"
    # growing base build: with build_frac > 0 each base batch holds
    # build_frac x (points already built) points, at least build_min and at
    # most build_batch (the first batch, into the empty index, is build_min)
    build_frac: float = 0.0
    build_min: int = 0
    # untimed refresh passes after the base build: every base batch is
    # deleted and re-inserted, so each list is rebuilt against the whole base
    refresh: int = 1

    def build_sizes(self):
        if self.build_frac <= 0.0:
            n_b = (self.base_n + self.build_batch - 1) // self.build_batch
            return [min(self.build_batch, self.base_n - b * self.build_batch) for b in range(n_b)]
        sizes, done = [], 0
        while done < self.base_n:
            n = min(self.build_batch, max(self.build_min, int(self.build_frac * done)), self.base_n - done)
            sizes.append(n)
            done += n
        return sizes


@dataclass(frozen=True)
class WorkloadDef:
    name: str
    description: str
    index: IndexConfig
    stream: StreamSpec
    sampler: str
    sampler_args: Tuple = ()


CONFIGS = {
    # 10,000 x 32 fp32 N(0,1), built by 10 batches of 1,000, then one round of
    # +1,000 inserts, -500 uniform deletes, 100 queries (k=10, beam 64).
    "tiny": WorkloadDef(
        "tiny", "10K x 32 fp32 N(0,1), Vamana R=32 L=64",
        IndexConfig("vamana", "f32", "l2", 32, 11_000, 32, 64, max_iters=128),
        StreamSpec(10_000, 1_000, 1, 1_000, 500, 100, 10, 64),
        "gauss"),
    # 1M x 128 uint8 from a 256-component Gaussian mixture, centres U[0,255],
    # sigma 20, rounded and clipped; 20 rounds of +10K / -10K / 10K queries.
    "sift1m_u8": WorkloadDef(
        "sift1m_u8", "1M x 128 uint8 256-component mixture, Vamana R=64 L=128",
        IndexConfig("vamana", "u8", "l2", 128, 1_010_000, 64, 128),
        StreamSpec(1_000_000, 10_000, 20, 10_000, 10_000, 10_000, 10, 64),
        "mix_u8", (256, 20.0)),
    # 1M x 96 fp32 sliding window, 512-component mixture, L2-normalised,
    # drifting mixture weights; 50 steps of +10K / -10K oldest / 10K queries.
    "deep1m_window": WorkloadDef(
        "deep1m_window", "1M x 96 fp32 sliding window, Vamana R=64 L=128",
        IndexConfig("vamana", "f32", "l2", 96, 1_010_000, 64, 128),
        StreamSpec(1_000_000, 10_000, 50, 10_000, 10_000, 10_000, 10, 64,
                   delete_policy="oldest"),
        "mix_norm_drift", (512, 0.5, 50)),
    # 1M x 100 fp32 unit vectors, inner product, Student-t(3) mixture of 1,000
    # components; CAGRA fixed degree 64; 10 batches of -30K / +10K.
    "glove1m_cagra": WorkloadDef(
        "glove1m_cagra", "1M x 100 fp32 IP, CAGRA fixed degree 64",
        IndexConfig("cagra", "f32", "ip", 100, 1_000_000, 64, 64),
        StreamSpec(1_000_000, 10_000, 10, 10_000, 30_000, 10_000, 10, 64,
                   order=("delete", "insert", "search"), refresh=0),
        "mix_t_norm", (1000, 0.3, 3.0)),
    # 500K x 768 fp32 inner-product data with varying norms (a Gaussian
    # mixture, norms clipped at 40), searched through the L2 augmentation
    # with M = 40; 10 rounds of +5K / -5K / 5K queries (beam 128).
    "ip768_mips": WorkloadDef(
        "ip768_mips", "500K x 768 fp32 inner product (MIPS via L2 augmentation), Vamana R=64 L=128",
        IndexConfig("vamana", "f32", "mips", 768, 505_000, 64, 128, mips_norm=40.0),
        StreamSpec(500_000, 5_000, 10, 5_000, 5_000, 5_000, 10, 128, refresh=3),
        "mix_ip", (128, 0.35, 40.0)),
    # 500K x 960 fp32, 128-component mixture, per-dimension scale U[0.1,1],
    # clipped at zero; 10 rounds of +5K / -5K / 5K queries (beam 128).
    "gist500k": WorkloadDef(
        "gist500k", "500K x 960 fp32 scaled clipped mixture, Vamana R=64 L=128",
        IndexConfig("vamana", "f32", "l2", 960, 505_000, 64, 128),
        StreamSpec(500_000, 5_000, 10, 5_000, 5_000, 5_000, 10, 128, refresh=3),
        "mix_relu_scaled", (128, 0.5)),
}


class _Sampler:
    """Draws vectors; also returns the mixture component of each vector."""

    def __init__(self, kind: str, args: Tuple, dim: int, seed: int):
        self.kind, self.args, self.dim = kind, args, dim
        g = _rng(seed, _P_MODEL)
        d = dim
        if kind == "gauss":
            self.n_comp = 1
        elif kind == "mix_u8":
            self.n_comp, self.sigma = args
            self.centres = g.uniform(0.0, 255.0, size=(self.n_comp, d))
        elif kind == "mix_norm_drift":
            self.n_comp, self.sigma, self.horizon = args
            self.centres = g.standard_normal((self.n_comp, d))
            self.w0 = g.dirichlet(np.ones(self.n_comp))
            self.w1 = g.dirichlet(np.ones(self.n_comp))
        elif kind == "mix_t_norm":
            self.n_comp, self.scale, self.nu = args
            self.centres = g.standard_normal((self.n_comp, d))
        elif kind == "mix_relu_scaled":
            self.n_comp, self.sigma = args
            self.dim_scale = g.uniform(0.1, 1.0, size=d)
            self.centres = g.standard_normal((self.n_comp, d))
        elif kind == "mix_ip":
            self.n_comp, self.sigma, self.max_norm = args
            # centres of different lengths, so that norms vary across components
            self.centres = g.standard_normal((self.n_comp, d)) * g.uniform(0.5, 1.5, size=(self.n_comp, 1))
        else:
            raise ValueError(kind)

    def weights(self, t: float) -> np.ndarray:
        if self.kind == "mix_norm_drift":
            a = min(max(t / float(self.horizon), 0.0), 1.0)
            w = (1.0 - a) * self.w0 + a * self.w1
            return w / w.sum()
        return np.full(self.n_comp, 1.0 / self.n_comp)

    def draw(self, g: np.random.Generator, n: int, t: float = 0.0,
             comps: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
        d = self.dim
        if self.kind == "gauss":
            return g.standard_normal((n, d)).astype(np.float32), np.zeros(n, np.int32)
        if comps is None:
            comps = g.choice(self.n_comp, size=n, p=self.weights(t)).astype(np.int32)
        mu = self.centres[comps]
        if self.kind == "mix_u8":
            x = np.rint(mu + self.sigma * g.standard_normal((n, d)))
            return np.clip(x, 0, 255).astype(np.uint8), comps
        if self.kind == "mix_ip":
            x = mu + self.sigma * g.standard_normal((n, d))
            nrm = np.linalg.norm(x, axis=1, keepdims=True)
            x = x * np.minimum(1.0, (0.999 * self.max_norm) / np.maximum(nrm, 1e-30))
            return x.astype(np.float32), comps
        if self.kind == "mix_norm_drift":
            x = mu + self.sigma * g.standard_normal((n, d))
        elif self.kind == "mix_t_norm":
            x = mu + self.scale * g.standard_t(self.nu, size=(n, d))
        else:  # mix_relu_scaled
            x = np.maximum(0.0, self.dim_scale * (mu + self.sigma * g.standard_normal((n, d))))
            return x.astype(np.float32), comps
        nrm = np.linalg.norm(x, axis=1, keepdims=True)
        nrm[nrm == 0] = 1.0
        return (x / nrm).astype(np.float32), comps


@dataclass
class Op:
    kind: str                        # "insert" | "delete" | "search"
    ids: Optional[np.ndarray] = None  # uint32
    vecs: Optional[np.ndarray] = None  # n x dim (insert vectors or queries)


class Workload:
    """Operation stream: base build batches, then rounds of single-type batches.

    Fresh ids are the smallest free ids (ascending); deletes are uniform
    without replacement over the currently active ids, or the oldest ids for
    the sliding window.  The stream depends only on the seed, never on the
    index state.
    """

    def __init__(self, wdef: WorkloadDef, seed: int = 0):
        self.wdef = wdef
        self.cfg = wdef.index
        self.spec = wdef.stream
        self.seed = seed
        self.sampler = _Sampler(wdef.sampler, wdef.sampler_args, self.cfg.dim, seed)
        cap = self.cfg.capacity
        self.active = np.zeros(cap, dtype=bool)
        self.birth = np.full(cap, -1, dtype=np.int64)    # insertion counter
        self.comp = np.full(cap, -1, dtype=np.int32)
        self._clock = 0
        self.vectors = None  # optional host copy of every inserted vector
        self._np_dtype = np.uint8 if self.cfg.dtype == "u8" else np.float32

    # -- bookkeeping -------------------------------------------------------
    def keep_vectors(self) -> "Workload":
        """Keep a host copy of the vector pool (for ground truth)."""
        self.vectors = np.zeros((self.cfg.capacity, self.cfg.dim), self._np_dtype)
        return self

    def active_ids(self) -> np.ndarray:
        return np.flatnonzero(self.active).astype(np.uint32)

    def _alloc(self, n: int) -> np.ndarray:
        free = np.flatnonzero(~self.active)
        if free.size < n:
            raise RuntimeError("workload exceeds index capacity")
        return free[:n].astype(np.uint32)

    def _apply_insert(self, ids, vecs, comps):
        self.active[ids] = True
        self.birth[ids] = self._clock + np.arange(ids.size)
        self._clock += ids.size
        self.comp[ids] = comps
        if self.vectors is not None:
            self.vectors[ids] = vecs

    def _apply_delete(self, ids):
        self.active[ids] = False
        self.birth[ids] = -1
        self.comp[ids] = -1

    # -- stream ------------------------------------------------------------
    def base_batches(self) -> Iterator[Op]:
        s = self.spec
        for b, n in enumerate(s.build_sizes()):
            g = _rng(self.seed, _P_BASE, b)
            vecs, comps = self.sampler.draw(g, n, t=0.0)
            ids = self._alloc(n)
            self._apply_insert(ids, vecs, comps)
            yield Op("insert", ids, vecs)

    def _queries(self, r: int, t: float) -> np.ndarray:
        s = self.spec
        g = _rng(self.seed, _P_QRY, r)
        if self.sampler.kind == "mix_norm_drift":
            act = np.flatnonzero(self.active)
            comps = self.comp[act[g.integers(0, act.size, size=s.n_query)]]
            return self.sampler.draw(g, s.n_query, t, comps=comps)[0]
        return self.sampler.draw(g, s.n_query, t)[0]

    def round_ops(self, r: int) -> Iterator[Op]:
        """Operations of round r (0-based), in the stream's order."""
        s = self.spec
        t = float(r + 1)
        for kind in s.order:
            if kind == "insert" and s.n_insert > 0:
                g = _rng(self.seed, _P_INS, r)
                vecs, comps = self.sampler.draw(g, s.n_insert, t)
                ids = self._alloc(s.n_insert)
                self._apply_insert(ids, vecs, comps)
                yield Op("insert", ids, vecs)
            elif kind == "delete" and s.n_delete > 0:
                act = np.flatnonzero(self.active)
                n = min(s.n_delete, act.size)
                if s.delete_policy == "oldest":
                    order = np.argsort(self.birth[act], kind="stable")
                    ids = np.sort(act[order[:n]]).astype(np.uint32)
                else:
                    g = _rng(self.seed, _P_DEL, r)
                    ids = np.sort(g.choice(act, size=n, replace=False)).astype(np.uint32)
                    ids = g.permutation(ids).astype(np.uint32)
                self._apply_delete(ids)
                yield Op("delete", ids)
            elif kind == "search" and s.n_query > 0:
                yield Op("search", None, self._queries(r, t))

    def rounds(self, n_rounds: Optional[int] = None) -> Iterator[Tuple[int, List[Op]]]:
        n = self.spec.n_rounds if n_rounds is None else n_rounds
        for r in range(n):
            yield r, list(self.round_ops(r))


def make_workload(name: str, seed: int = 0, index: Optional[dict] = None,
                  stream: Optional[dict] = None, sampler_args: Optional[Tuple] = None) -> Workload:
    """Build a workload by name, optionally overriding index or stream fields
    or the sampler's arguments (used to make small variants of the large
    workloads for tests)."""
    w = CONFIGS[name]
    idx = dataclasses.replace(w.index, **(index or {}))
    st = dataclasses.replace(w.stream, **(stream or {}))
    sa = w.sampler_args if sampler_args is None else tuple(sampler_args)
    return Workload(WorkloadDef(w.name, w.description, idx, st, w.sampler, sa), seed)


# ---------------------------------------------------------------------------
# Streaming patterns of the paper's workload generator (Section 5.2), over a
# fixed synthetic dataset of `n_total` points drawn from a workload's
# sampler.  Batches are uniform and of a single operation type; searches use
# fresh queries from the same distribution.  Ids are the smallest free ids at
# insert time.  The k-means of the clustered pattern is workload generation
# (it orders the data), not part of the index method.
PATTERNS = ("sliding_window", "interleaved", "expiration", "clustered", "insert_heavy")
_P_PAT, _P_PATQ, _P_KM = 6, 7, 8


def _kmeans(x: np.ndarray, k: int, seed: int, iters: int = 10, sample: int = 50_000) -> np.ndarray:
    """Lloyd's k-means on a sample (float32), then every point assigned to
    its nearest centre; returns the cluster of each point."""
    g = _rng(seed, _P_KM)
    xs = x[g.choice(len(x), min(sample, len(x)), replace=False)].astype(np.float32)
    c = xs[g.choice(len(xs), k, replace=False)].copy()

    def assign(pts):
        out = np.empty(len(pts), np.int64)
        cn = (c * c).sum(1)
        for s in range(0, len(pts), 65536):
            p = pts[s:s + 65536].astype(np.float32)
            out[s:s + len(p)] = np.argmin(cn[None, :] - 2.0 * p @ c.T, axis=1)
        return out

    for _ in range(iters):
        a = assign(xs)
        for j in range(k):
            m = a == j
            if m.any():
                c[j] = xs[m].mean(0)
    return assign(x)


class PatternStream:
    """One streaming pattern over `n_total` points of workload `w`'s
    distribution.  `base_ops()` builds the starting index; `ops()` yields
    the operation stream (Op with kind insert / delete / search)."""

    def __init__(self, w: "Workload", pattern: str, n_total: int, n_query: int = 1000, seed: int = 0,
                 batch_frac: float = 0.01, build_batch: int = 10_000):
        if pattern not in PATTERNS:
            raise ValueError(pattern)
        self.w, self.pattern, self.n, self.nq, self.seed = w, pattern, n_total, n_query, seed
        self.batch = max(1, int(round(batch_frac * n_total)))
        self.build_batch = build_batch
        g = _rng(seed, _P_PAT)
        self.x = w.sampler.draw(g, n_total, 0.0)[0]
        self.ids = np.full(n_total, INVALID, np.uint64)   # pool id of each dataset point while active
        self._q = 0
        if pattern == "clustered":
            cl = _kmeans(self.x.astype(np.float32), 64, seed)
            self.order = np.argsort(cl, kind="stable")
            self.cluster_bounds = np.searchsorted(cl[self.order], np.arange(65))
        elif pattern == "expiration":
            half = n_total // 2
            life = _rng(seed, _P_PAT, 1).choice(np.array([10, 100, -1]), size=n_total - half,
                                                  p=np.array([10, 2, 1]) / 13.0)
            self.lifetime = np.concatenate([np.full(half, -1), life])   # -1: permanent

    # -- helpers
    def _insert(self, pts: np.ndarray) -> Op:
        ids = self.w._alloc(len(pts))
        self.w._apply_insert(ids, self.x[pts], np.zeros(len(pts), np.int32))
        self.ids[pts] = ids
        return Op("insert", ids, self.x[pts])

    def _delete(self, pts: np.ndarray) -> Op:
        ids = self.ids[pts].astype(np.uint32)
        assert (self.ids[pts] != INVALID).all()
        self.w._apply_delete(ids)
        self.ids[pts] = INVALID
        return Op("delete", ids)

    def _search(self) -> Op:
        g = _rng(self.seed, _P_PATQ, self._q)
        self._q += 1
        return Op("search", None, self.w.sampler.draw(g, self.nq, 0.0)[0])

    def _batches(self, pts):
        for s in range(0, len(pts), self.batch):
            yield pts[s:s + self.batch]

    def _base_points(self) -> np.ndarray:
        n = self.n
        if self.pattern == "sliding_window":
            return np.arange(n // 2)                       # the first 50 of 100 segments
        if self.pattern == "expiration":
            return np.arange(n // 2)                       # the first half
        if self.pattern == "clustered":
            return self.order[:self.cluster_bounds[32]]    # the first 32 clusters
        return np.arange(n // 10)                          # interleaved, insert-heavy: 10%

    def base_ops(self) -> Iterator[Op]:
        pts = self._base_points()
        for s in range(0, len(pts), self.build_batch):
            yield self._insert(pts[s:s + self.build_batch])

    def ops(self) -> Iterator[Op]:
        n, p = self.n, self.pattern
        if p == "sliding_window":
            seg = n // 100
            for t in range(50):
                for b in self._batches(np.arange((t + 50) * seg, (t + 51) * seg)):
                    yield self._insert(b)
                for b in self._batches(np.arange(t * seg, (t + 1) * seg)):
                    yield self._delete(b)
                yield self._search()
        elif p == "expiration":
            half = n // 2
            seg = (n - half) // 50
            born = np.full(n, -1)
            for c in range(50):
                pts = np.arange(half + c * seg, half + (c + 1) * seg)
                for b in self._batches(pts):
                    yield self._insert(b)
                born[pts] = c
                exp = np.flatnonzero((born >= 0) & (self.lifetime > 0) & (born + self.lifetime == c) &
                                     (self.ids != INVALID))
                for b in self._batches(exp):
                    yield self._delete(b)
                yield self._search()
        elif p == "clustered":
            for t in range(32):
                for b in self._batches(self.order[self.cluster_bounds[t + 32]:self.cluster_bounds[t + 33]]):
                    yield self._insert(b)
                    yield self._search()
                for b in self._batches(self.order[self.cluster_bounds[t]:self.cluster_bounds[t + 1]]):
                    yield self._delete(b)
                    yield self._search()
        elif p == "interleaved":
            g = _rng(self.seed, _P_PAT, 2)
            nxt = n // 10
            while nxt < n:
                kind = g.choice(3, p=[0.5, 0.3, 0.2])
                if kind == 0:
                    pts = np.arange(nxt, min(n, nxt + self.batch))
                    nxt += len(pts)
                    yield self._insert(pts)
                elif kind == 1:
                    yield self._search()
                else:
                    act = np.flatnonzero(self.ids != INVALID)
                    if len(act) > self.batch:
                        yield self._delete(np.sort(g.choice(act, self.batch, replace=False)))
        else:  # insert_heavy
            g = _rng(self.seed, _P_PAT, 3)
            nxt = n // 10
            while nxt < n:
                if g.random() < 0.9:
                    pts = np.arange(nxt, min(n, nxt + self.batch))
                    nxt += len(pts)
                    yield self._insert(pts)
                else:
                    yield self._search()


_P_INIT = 9


def cagra_init_lists(n: int, knn: int, seed: int = 0) -> np.ndarray:
    """Random initial neighbour lists for the CAGRA graph construction's
    NN-Descent: row u holds ``knn`` distinct positions in [0, n) other than u,
    drawn uniformly.  These are the random numbers the construction starts
    from; both the GPU library and the oracle take them as input."""
    if not 0 < knn < n:
        raise ValueError("need 0 < knn < n")
    g = _rng(seed, _P_INIT)
    off = np.sort(g.integers(0, n - 1, size=(n, knn), dtype=np.int64), axis=1)
    while True:  # redraw repeated offsets until every row is distinct
        dup = np.zeros_like(off, dtype=bool)
        dup[:, 1:] = off[:, 1:] == off[:, :-1]
        k = int(dup.sum())
        if k == 0:
            break
        off[dup] = g.integers(0, n - 1, size=k, dtype=np.int64)
        off.sort(axis=1)
    u = np.arange(n, dtype=np.int64)[:, None]
    return ((u + 1 + off) % n).astype(np.uint32)
