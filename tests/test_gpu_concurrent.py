"""Searches concurrent with updates (readers): a reader on its own stream
returns exactly grand_search's results when no update overlaps it, and
while another host thread inserts and deletes it returns only pool ids that
were active at some point of the run (the consistency model of
include/grand.h); the updates themselves are unaffected: the final graph
equals the oracle's after the same batches."""
import threading

import numpy as np
import pytest

from helpers import INVALID, check_graph_invariants, canonical_rows
from oracle.oracle import Oracle
from parity import say
from workloads import make_workload

pytestmark = pytest.mark.gpu

CASES = {
    "u8_d128": ("sift1m_u8", dict(capacity=14_000),
                dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=400)),
    "f32_d96": ("deep1m_window", dict(capacity=11_000),
                dict(base_n=6_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=400)),
    "cagra_ip_d100": ("glove1m_cagra", dict(capacity=11_000),
                      dict(base_n=6_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=400)),
}


def _setup(case):
    from paper_2608_21163_amd import GrandIndex
    name, idx, st = CASES[case]
    w = make_workload(name, seed=9, index=idx, stream=st).keep_vectors()
    g = GrandIndex.from_config(w.cfg, max_batch=2_000)
    o = Oracle(w.cfg)
    for op in w.base_batches():
        g.insert(op.ids, op.vecs)
        assert o.insert(op.ids, op.vecs) == 0
    return w, g, o


@pytest.mark.parametrize("case", list(CASES))
def test_reader_matches_search_when_quiescent(case):
    from paper_2608_21163_amd import Reader
    say(f"[reader quiescent] {case}")
    w, g, o = _setup(case)
    r = Reader(g)
    q = next(op for _, ops in w.rounds(1) for op in ops if op.kind == "search").vecs
    gi, gd = g.search(q, w.spec.k, w.spec.beam)
    ri, rd = r.search(q, w.spec.k, w.spec.beam)
    assert np.array_equal(gi, ri) and np.array_equal(gd.view(np.uint32), rd.view(np.uint32))
    r.close()
    g.close()


@pytest.mark.parametrize("case", list(CASES))
def test_reader_during_updates(case):
    from paper_2608_21163_amd import Reader
    say(f"[reader during updates] {case}")
    w, g, o = _setup(case)
    r = Reader(g)
    ever_active = w.active.copy()
    rounds = list(w.rounds(3))
    for _, ops in rounds:
        for op in ops:
            if op.kind == "insert":
                ever_active[op.ids] = True
    queries = [op.vecs for _, ops in rounds for op in ops if op.kind == "search"]
    results, errors = [], []
    stop = threading.Event()

    def reader():
        try:
            i = 0
            while not stop.is_set() or i < 2:
                ids, d = r.search(queries[i % len(queries)], w.spec.k, w.spec.beam)
                results.append((ids.copy(), d.copy()))
                i += 1
        except Exception as e:  # reported below
            errors.append(e)

    t = threading.Thread(target=reader)
    t.start()
    try:
        for _, ops in rounds:
            for op in ops:
                if op.kind == "insert":
                    g.insert(op.ids, op.vecs)
                    assert o.insert(op.ids, op.vecs) == 0
                elif op.kind == "delete":
                    g.delete(op.ids)
                    assert o.delete(op.ids) == 0
    finally:
        stop.set()
        t.join()
    assert not errors, errors
    say(f"  {len(results)} reader searches ran beside {sum(len(ops) for _, ops in rounds)} batches")
    assert len(results) >= 2
    for ids, d in results:
        valid = ids != INVALID
        assert (ids[valid] < w.cfg.capacity).all()
        assert ever_active[ids[valid].astype(np.int64)].all(), "a search returned an id that was never active"
        assert np.isfinite(d[valid]).all() and np.isinf(d[~valid]).all()
        if w.cfg.metric == "l2":
            assert (d[valid] >= 0).all()
    gst, ost = g.export(), o.export()
    check_graph_invariants(gst, w.cfg.R)
    assert np.array_equal(gst["active"], ost["active"]) and gst["medoid"] == ost["medoid"]
    a, b = (canonical_rows(gst["adj"]), canonical_rows(ost["adj"])) if w.cfg.algo == "vamana" else \
        (gst["adj"], ost["adj"])
    frac = np.any(a != b, axis=1).sum() / max(int(ost["active"].sum()), 1)
    say(f"  differing lists after the concurrent run: {frac:.5f}")
    assert frac <= (0.0 if w.cfg.dtype == "u8" else 0.001)
    r.close()
    g.close()
