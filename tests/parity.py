"""Helpers of the GPU-vs-oracle parity tests.  The oracle's state is the
reference; GPU results are compared with it by the acceptance rules:
integer structures bit-exact, distances within 1e-5 relative, adjacency
lists identical (as sets for Vamana, as slot sequences for CAGRA) except
for rare rows explained by distance ties."""
import sys

import numpy as np

from helpers import INVALID, canonical_rows

DIST_RTOL = 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def pool_vectors(w):
    """The full vector pool (capacity rows) of a workload that keeps vectors."""
    assert w.vectors is not None
    return w.vectors


def to_gpu(o, g, w):
    """Copies the oracle's current state (and the workload's vectors) into
    the GPU index."""
    st = o.export()
    g.import_graph(pool_vectors(w), st["adj"], st["deg"], st["active"], st["medoid"])
    return st


def _row_sets(st, algo):
    adj = st["adj"]
    return adj if algo == "cagra" else canonical_rows(adj)


def differing_rows(gst, ost, algo):
    a, b = _row_sets(gst, algo), _row_sets(ost, algo)
    return np.flatnonzero(np.any(a != b, axis=1) | (gst["deg"] != ost["deg"]))


def _near(x, y, tol=DIST_RTOL):
    return abs(x - y) <= tol * max(abs(x), abs(y), 1e-30)


def _search_has_tie(o_pre, vec, start, ell, iters):
    """True when the oracle's search from `vec` on the pre-batch state meets
    two keys whose distances agree within the tolerance (a tie that can
    order the keys differently on the two sides)."""
    C_ids, C_d, V_ids, V_d = o_pre.beam_search(vec, start, ell, iters)
    d = np.sort(np.concatenate([C_d, V_d]).astype(np.float64))
    d = np.unique(d)
    if len(d) < 2:
        return False
    gap = np.abs(np.diff(d)) <= DIST_RTOL * np.maximum(np.abs(d[1:]), 1e-30)
    return bool(gap.any())


def explain_differences(gst, ost, rows, ctx):
    """Traces every differing list to a distance tie within DIST_RTOL of the
    oracle's own distances (the acceptance rule: each mismatch is explained
    by a tie).  A list u is explained when
      (1) two ids of either side's list have Dist(u, .) within the tolerance,
      (2) an alpha-test of u's prune sits within the tolerance of its
          boundary: coef * Dist(s, x) ~ Dist(u, x) for s, x in the lists,
      (3) it differs by an id x whose own list differs and holds u on one
          side only (the reverse edge x -> u exists on one side only), or
      (4) u is a point of the batch whose search on the pre-batch state meets
          a tie (its forward list, or the repair candidates C_u, follow).
    Returns the rows left unexplained."""
    algo, dist, coef = ctx["algo"], ctx["dist"], ctx["coef"]
    rows_set = set(int(r) for r in rows)
    G, O = _row_sets(gst, algo), _row_sets(ost, algo)

    def ids(row):
        return set(int(v) for v in row if v != INVALID)

    batch_tie = {}
    left = []
    for u in rows_set:
        g, o = ids(G[u]), ids(O[u])
        X = g ^ o
        every = g | o
        D = {x: dist(u, x) for x in every}
        ok = False
        for x in X:                                              # (1)
            if any(y != x and _near(D[x], D[y]) for y in every):
                ok = True
                break
        if not ok and coef is not None:                          # (2)
            ok = any(s != x and _near(coef * dist(s, x), D[x]) for x in X for s in every)
        if not ok:                                               # (3)
            for x in X:
                if x in rows_set and u in (ids(G[x]) ^ ids(O[x])):
                    ok = True
                    break
        if not ok and ctx.get("batch") is not None and u in ctx["batch"]:   # (4)
            if u not in batch_tie:
                if ctx["start"] == INVALID:
                    # empty index: the candidates are the batch points by brute force
                    d = np.unique(np.array([dist(u, x) for x in ctx["batch"] if x != u], np.float64))
                    batch_tie[u] = bool(len(d) > 1 and (np.diff(d) <= DIST_RTOL * np.abs(d[1:])).any())
                else:
                    batch_tie[u] = _search_has_tie(ctx["pre"], ctx["vecs"][u], ctx["start"], ctx["ell"],
                                                   ctx["iters"])
            ok = batch_tie[u]
        if not ok and algo == "cagra" and not X and g == o:
            ok = True                                            # same set, slot order only: (4) of a neighbour
        if not ok:
            left.append(u)
    return left


def compare_states(gst, ost, algo, allow_frac=0.0, ctx=None):
    """Returns the number of differing rows.  The integer state (active map,
    medoid) must be identical; at most allow_frac of the active lists may
    differ, and with a context (fp32 data) every differing list must be
    traced to a distance tie within DIST_RTOL (explain_differences)."""
    assert np.array_equal(gst["active"], ost["active"]), "active maps differ"
    assert gst["medoid"] == ost["medoid"], (gst["medoid"], ost["medoid"])
    rows = differing_rows(gst, ost, algo)
    n_act = max(int(ost["active"].sum()), 1)
    frac = len(rows) / n_act
    assert frac <= allow_frac, f"{len(rows)} of {n_act} lists differ (allowed {allow_frac:.4%}): {rows[:10]}"
    if len(rows) and ctx is not None:
        left = explain_differences(gst, ost, rows, ctx)
        assert not left, f"lists without a distance tie: {left[:10]}"
    return len(rows)


def tie_context(o_pre, w, algo, batch_ids, coef):
    """Context for explain_differences: the oracle of the pre-batch state,
    the pool vectors, the batch ids and the search parameters."""
    vecs = w.vectors
    stored = {}

    def row(i):
        # the stored form of a point (the MIPS augmentation appends a coordinate)
        if i not in stored:
            stored[i] = o_pre.store_row(vecs[i])[0]
        return stored[i]

    def dist(a, b):
        return o_pre.dist(row(a), row(b))

    cfg = w.cfg
    return dict(algo=algo, dist=dist, coef=coef, pre=o_pre, vecs=vecs,
                batch=set(int(x) for x in batch_ids), start=o_pre.export()["medoid"],
                ell=cfg.L_build, iters=cfg.iters)


def compare_search(gi, gd, oi, od, allow_frac=0.0):
    """Search results: distances within DIST_RTOL; ids identical except rows
    whose differences are explained by distance ties within DIST_RTOL."""
    assert gi.shape == oi.shape
    valid = oi != INVALID
    assert np.array_equal(valid, gi != INVALID), "different number of results"
    scale = np.maximum(np.abs(od), 1e-30)
    dd = np.where(valid, np.abs(gd.astype(np.float64) - od.astype(np.float64)) / scale, 0.0)
    assert dd.max(initial=0.0) <= DIST_RTOL, f"distance mismatch {dd.max()}"
    bad = np.flatnonzero(np.any(gi != oi, axis=1))
    for r in bad:
        # a tie-explained row holds the same distances; differing ids sit at
        # positions whose distance has a near-equal neighbour
        for j in np.flatnonzero(gi[r] != oi[r]):
            near = np.abs(od[r] - od[r, j]) <= DIST_RTOL * max(abs(float(od[r, j])), 1e-30)
            assert near.sum() >= 2 or j == gi.shape[1] - 1, f"row {r}: id mismatch without a tie"
    assert len(bad) <= allow_frac * len(gi) + 1e-9, f"{len(bad)} rows differ"
    return len(bad)


def recall(ids, gt):
    k = gt.shape[1]
    hits = [len(set(a[:k].tolist()) & set(b.tolist())) for a, b in zip(ids, gt)]
    return float(np.mean(hits)) / k
