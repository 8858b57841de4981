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


def compare_states(gst, ost, algo, allow_frac=0.0):
    """Returns the number of differing rows; asserts the integer state
    (active map, medoid) is identical and the differing fraction small."""
    assert np.array_equal(gst["active"], ost["active"]), "active maps differ"
    assert gst["medoid"] == ost["medoid"], (gst["medoid"], ost["medoid"])
    if algo == "vamana":
        a, b = canonical_rows(gst["adj"]), canonical_rows(ost["adj"])
    else:
        a, b = gst["adj"], ost["adj"]
    rows = np.flatnonzero(np.any(a != b, axis=1) | (gst["deg"] != ost["deg"]))
    n_act = max(int(ost["active"].sum()), 1)
    frac = len(rows) / n_act
    assert frac <= allow_frac, f"{len(rows)} of {n_act} lists differ (allowed {allow_frac:.4%}): {rows[:10]}"
    return len(rows)


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
