"""The fp32 acceptance rule of the GPU parity tests, checked on the CPU:
a list that differs from the oracle's passes only when a distance tie
within 1e-5 (relative) explains it."""
import numpy as np

from helpers import INVALID, line_config, rows_to_adj
from oracle.oracle import Oracle
from parity import compare_states, explain_differences


class _W:
    def __init__(self, cfg, vecs):
        self.cfg, self.vectors = cfg, vecs


def _ctx(o, vecs):
    return dict(algo="vamana", dist=lambda a, b: o.dist(vecs[a], vecs[b]), coef=1.2, pre=o, vecs=vecs,
                batch=None, start=0, ell=8, iters=16)


def _state(rows, R, n):
    adj, deg = rows_to_adj(rows, R)
    return dict(adj=adj, deg=deg, active=np.ones(n, np.uint8), medoid=0)


def test_tie_explains_a_swapped_neighbour_and_nothing_else_does():
    # u = 0 at 0; ids 1 and 2 at +1 and -1 tie at distance 1; id 3 at 5
    vecs = np.array([[0.0], [1.0], [-1.0], [5.0], [9.0]], np.float32)
    n, R = 5, 2
    o = Oracle(line_config(n, R))
    o.import_graph(vecs, *rows_to_adj([[1, 3], [0], [0], [0], [3]], R), np.ones(n, np.uint8), 0)
    ost = _state([[1, 3], [0], [0], [0], [3]], R, n)
    tied = _state([[2, 3], [0], [0], [0], [3]], R, n)      # 1 <-> 2: a tie at distance 1
    untied = _state([[4, 3], [0], [0], [0], [3]], R, n)    # 1 -> 4: distance 1 against 81
    assert explain_differences(tied, ost, [0], _ctx(o, vecs)) == []
    assert explain_differences(untied, ost, [0], _ctx(o, vecs)) == [0]
    assert compare_states(tied, ost, "vamana", allow_frac=0.5, ctx=_ctx(o, vecs)) == 1
    try:
        compare_states(untied, ost, "vamana", allow_frac=0.5, ctx=_ctx(o, vecs))
    except AssertionError:
        pass
    else:
        raise AssertionError("an untied difference was accepted")


def test_fraction_bar_applies_before_tracing():
    vecs = np.arange(10, dtype=np.float32)[:, None]
    ost = _state([[1]] * 10, 1, 10)
    gst = _state([[1]] * 9 + [[2]], 1, 10)
    try:
        compare_states(gst, ost, "vamana", allow_frac=0.001)
    except AssertionError:
        return
    raise AssertionError("10% differing lists passed a 0.1% bar")
