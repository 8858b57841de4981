"""The five streaming patterns of Section 5.2, free-running on the GPU and
on the oracle from the same seeded stream (uint8 rows: distances are exact
integers on both sides, so every query result and the final graph must be
identical)."""
import numpy as np
import pytest

from helpers import canonical_rows, check_graph_invariants
from oracle.oracle import Oracle
from parity import say
from workloads import PATTERNS, PatternStream, make_workload

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("pattern", PATTERNS)
def test_pattern_stream_matches_oracle(pattern):
    from paper_2608_21163_amd import GrandIndex
    say(f"[pattern] {pattern}")
    w = make_workload("sift1m_u8", seed=6, index=dict(capacity=14_000, dim=32, R=32, L_build=64)).keep_vectors()
    ps = PatternStream(w, pattern, 12_000, n_query=100, seed=3, batch_frac=0.02, build_batch=2_000)
    g = GrandIndex.from_config(w.cfg, max_batch=2_000)
    o = Oracle(w.cfg)
    for op in ps.base_ops():
        g.insert(op.ids, op.vecs)
        assert o.insert(op.ids, op.vecs) == 0
    n = {"insert": 0, "delete": 0, "search": 0}
    for op in ps.ops():
        n[op.kind] += 1
        if op.kind == "insert":
            g.insert(op.ids, op.vecs)
            assert o.insert(op.ids, op.vecs) == 0
        elif op.kind == "delete":
            g.delete(op.ids)
            assert o.delete(op.ids) == 0
        else:
            gi, gd = g.search(op.vecs, 10, 64)
            oi, od = o.search(op.vecs, 10, 64)
            assert np.array_equal(gi, oi) and np.array_equal(gd, od), f"search {n['search']}"
    gst, ost = g.export(), o.export()
    check_graph_invariants(gst, w.cfg.R)
    assert np.array_equal(gst["active"], ost["active"]) and gst["medoid"] == ost["medoid"]
    assert np.array_equal(canonical_rows(gst["adj"]), canonical_rows(ost["adj"]))
    say(f"  {n} operations, identical throughout")
    g.close()
