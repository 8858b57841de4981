"""Small helpers shared by the tests (no method arithmetic beyond plain
numpy re-statements of definitions used as independent checks)."""
import numpy as np

INVALID = 0xFFFFFFFF


def line_config(n, R, ell=8, algo="vamana", **kw):
    from workloads import IndexConfig
    return IndexConfig(algo, "f32", "l2", 1, n, R, ell, **kw)


def rows_to_adj(rows, R, cap=None):
    cap = len(rows) if cap is None else cap
    adj = np.full((cap, R), INVALID, np.uint32)
    for i, r in enumerate(rows):
        adj[i, :len(r)] = r
    deg = (adj != INVALID).sum(1).astype(np.uint32)
    return adj, deg


def np_l2(a, b):
    """Squared L2 in float64 (numpy), one row against many."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return ((b - a) ** 2).sum(-1)


def brute_knn(base, active, queries, k, metric="l2"):
    """Exact k-NN over active rows by (distance, id), numpy float64."""
    ids = np.flatnonzero(active)
    X = base[ids].astype(np.float64)
    out = np.zeros((len(queries), k), np.int64)
    for i, q in enumerate(np.asarray(queries, np.float64)):
        if metric == "l2":
            d = ((X - q) ** 2).sum(1)
        else:
            d = -(X @ q)
        order = np.lexsort((ids, d.astype(np.float32)))
        out[i] = ids[order[:k]]
    return out


def canonical_rows(adj):
    """Vamana lists are sets: sort each row ascending, INVALID last."""
    return np.sort(adj, axis=1)


def check_graph_invariants(st, R, check_deg=True):
    """Out-degree <= R, no self loops, no duplicates, no edges to inactive
    ids, deleted rows empty, degree equals the valid count, medoid active."""
    adj, deg, act = st["adj"], st["deg"], st["active"].astype(bool)
    cap = adj.shape[0]
    valid = adj != INVALID
    assert adj.shape[1] == R
    if check_deg:
        assert np.array_equal(valid.sum(1), deg)
    assert not valid[~act].any(), "inactive rows must be empty"
    tgt = np.where(valid, adj, 0).astype(np.int64)
    assert (tgt < cap).all()
    assert act[tgt[valid]].all(), "edge to an inactive id"
    self_loop = valid & (adj == np.arange(cap, dtype=np.uint32)[:, None])
    assert not self_loop.any(), "self loop"
    s = np.sort(np.where(valid, adj, INVALID), axis=1)
    dup = (s[:, 1:] == s[:, :-1]) & (s[:, 1:] != INVALID)
    assert not dup.any(), "repeated neighbour"
    if act.any():
        assert st["medoid"] != INVALID and act[st["medoid"]], "medoid must be active"
    else:
        assert st["medoid"] == INVALID
