"""The streaming patterns of the workload generator (Section 5.2) follow
their definitions: sliding window, interleaved, expiration time, clustered
(k-means) and insert heavy.  Generator only; no index arithmetic."""
import numpy as np
import pytest

from workloads import PATTERNS, PatternStream, make_workload


def _stream(pattern, n=10_000):
    w = make_workload("sift1m_u8", seed=4, index=dict(capacity=n + 2_000, dim=16)).keep_vectors()
    ps = PatternStream(w, pattern, n, n_query=20, seed=2, batch_frac=0.01, build_batch=2_000)
    base = list(ps.base_ops())
    return w, ps, base, list(ps.ops())


def test_sliding_window_keeps_half_the_segments_active():
    w, ps, base, ops = _stream("sliding_window")
    assert sum(len(o.ids) for o in base) == 5_000
    act = 5_000
    steps = 0
    for o in ops:
        if o.kind == "insert":
            act += len(o.ids)
        elif o.kind == "delete":
            act -= len(o.ids)
        else:
            steps += 1
            assert act == 5_000          # insert of segment t+50, then delete of segment t
    assert steps == 50


def test_expiration_deletes_exactly_the_expired_points():
    w, ps, base, ops = _stream("expiration")
    life = ps.lifetime
    assert (life[:5_000] == -1).all()    # the first half is permanent
    frac = np.bincount(np.searchsorted([-1, 10, 100], life[5_000:]), minlength=3) / 5_000.0
    assert abs(frac[1] - 10 / 13) < 0.03 and abs(frac[2] - 2 / 13) < 0.03 and abs(frac[0] - 1 / 13) < 0.03
    cycle, inserted_at, n_del = 0, {}, 0
    for o in ops:
        if o.kind == "insert":
            for i in o.ids.tolist():
                inserted_at[i] = cycle
        elif o.kind == "delete":
            # ids are reused after deletion: check at the time of deletion
            assert all(inserted_at[i] == cycle - 10 for i in o.ids.tolist())
            n_del += len(o.ids)
        else:
            cycle += 1
    assert n_del > 0, "short-lived points expire within 50 cycles"


def test_clustered_processes_whole_kmeans_clusters():
    w, ps, base, ops = _stream("clustered")
    assert sum(len(o.ids) for o in base) == ps.cluster_bounds[32]
    assert (np.diff(ps.cluster_bounds) > 0).sum() >= 48   # k-means gives non-empty clusters
    kinds = [o.kind for o in ops]
    # a search follows every insert or delete batch (every 1% of the dataset)
    assert all(kinds[i + 1] == "search" for i, k in enumerate(kinds) if k != "search")
    n_ins = sum(len(o.ids) for o in ops if o.kind == "insert")
    assert n_ins == ps.cluster_bounds[64] - ps.cluster_bounds[32]


@pytest.mark.parametrize("pattern", ["interleaved", "insert_heavy"])
def test_growth_patterns_insert_every_point(pattern):
    w, ps, base, ops = _stream(pattern)
    n_ins = sum(len(o.ids) for o in base) + sum(len(o.ids) for o in ops if o.kind == "insert")
    assert n_ins == 10_000
    kinds = np.array([o.kind for o in ops])
    if pattern == "insert_heavy":
        assert not (kinds == "delete").any()
        assert 0.8 < (kinds == "insert").mean() < 0.97
    else:
        assert (kinds == "delete").any() and (kinds == "search").any()
    assert w.active.sum() == 10_000 - sum(len(o.ids) for o in ops if o.kind == "delete")


@pytest.mark.parametrize("pattern", PATTERNS)
def test_patterns_are_deterministic(pattern):
    a = _stream(pattern)[3]
    b = _stream(pattern)[3]
    assert len(a) == len(b)
    for x, y in zip(a, b):
        assert x.kind == y.kind
        if x.ids is not None:
            assert np.array_equal(x.ids, y.ids)
        if x.vecs is not None:
            assert np.array_equal(x.vecs, y.vecs)
