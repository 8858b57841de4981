"""Pins of the oracle's Dist and BeamSearch (Alg. 1) against definitions
computed independently (exact integers, math.fsum, numpy brute force) and a
hand-traced example."""
import math

import numpy as np
import pytest

from helpers import INVALID, brute_knn, line_config, rows_to_adj
from oracle.oracle import Oracle
from workloads import IndexConfig


def _oracle(dtype, metric, dim, cap=4, R=4):
    return Oracle(IndexConfig("vamana" if metric == "l2" else "cagra", dtype, metric, dim, cap, R, 8))


def test_dist_uint8_is_exact_integer_l2():
    g = np.random.default_rng(1)
    o = _oracle("u8", "l2", 128)
    for _ in range(200):
        a = g.integers(0, 256, 128, dtype=np.uint8)
        b = g.integers(0, 256, 128, dtype=np.uint8)
        exact = int(((a.astype(np.int64) - b.astype(np.int64)) ** 2).sum())
        assert o.dist(a, b) == float(exact)
    # the largest possible value is still exact in fp32 (< 2^24)
    a = np.zeros(128, np.uint8)
    b = np.full(128, 255, np.uint8)
    assert o.dist(a, b) == 128 * 255 * 255


@pytest.mark.parametrize("metric", ["l2", "ip"])
def test_dist_fp32_matches_exactly_rounded_sum(metric):
    """fp32 Dist is the fp64 sum rounded once; compare with math.fsum (the
    correctly rounded sum of exact terms) rounded to fp32: equal, or at most
    one fp32 ulp apart when the fp64 chain lands next to a rounding edge."""
    g = np.random.default_rng(2)
    o = _oracle("f32", metric, 96)
    n_equal = 0
    for _ in range(500):
        a = g.standard_normal(96).astype(np.float32)
        b = g.standard_normal(96).astype(np.float32)
        if metric == "l2":
            terms = [(float(x) - float(y)) ** 2 for x, y in zip(a, b)]
            ref = np.float32(math.fsum(terms))
        else:
            terms = [float(x) * float(y) for x, y in zip(a, b)]
            ref = np.float32(-math.fsum(terms))
        got = np.float32(o.dist(a, b))
        assert abs(int(got.view(np.int32)) - int(ref.view(np.int32))) <= 1
        n_equal += got == ref
    assert n_equal >= 495


@pytest.mark.parametrize("dtype,metric", [("f32", "l2"), ("f32", "ip"), ("u8", "l2")])
def test_dist_is_symmetric_and_zero_is_positive(dtype, metric):
    g = np.random.default_rng(3)
    o = _oracle(dtype, metric, 33)
    for _ in range(50):
        if dtype == "u8":
            a, b = g.integers(0, 256, (2, 33), dtype=np.uint8)
        else:
            a, b = g.standard_normal((2, 33)).astype(np.float32)
        assert o.dist(a, b) == o.dist(b, a)
    z = np.zeros(33, np.uint8 if dtype == "u8" else np.float32)
    d = np.float32(o.dist(z, z))
    assert d == 0 and not np.signbit(d)


def _line_graph(golden):
    cfg = line_config(6, 2, ell=8)
    o = Oracle(cfg)
    rows = [[1], [0, 2], [1, 3], [2, 4], [3, 5], [4]]
    adj, deg = rows_to_adj(rows, 2)
    vecs = np.arange(6, dtype=np.float32)[:, None]
    o.import_graph(vecs, adj, deg, np.ones(6, np.uint8), 0)
    return o


def test_beam_search_hand_trace(golden):
    fx = golden("beam_search_trace.json")
    o = _line_graph(golden)
    for case in fx["cases"]:
        q = np.array([case["query"]], np.float32)
        C, Cd, V, Vd = o.beam_search(q, 0, case["ell"], case["max_iters"])
        assert C.tolist() == case["expected_C"], case["name"]
        assert V.tolist() == case["expected_V"], case["name"]
        for i, d in zip(C, Cd):
            assert d == np.float32((np.float64(q[0]) - float(i)) ** 2)


@pytest.mark.parametrize("dtype", ["f32", "u8"])
def test_beam_search_complete_graph_is_exact_knn(dtype):
    """With l >= N and max_iters >= N on a complete graph, BeamSearch expands
    every node and returns the exact nearest neighbours (Alg. 1)."""
    g = np.random.default_rng(4)
    n, d = 40, 8
    cfg = IndexConfig("vamana", dtype, "l2", d, n, n - 1, n, max_iters=2 * n)
    o = Oracle(cfg)
    if dtype == "u8":
        X = g.integers(0, 256, (n, d), dtype=np.uint8)
        Q = g.integers(0, 256, (10, d), dtype=np.uint8)
    else:
        X = g.standard_normal((n, d)).astype(np.float32)
        Q = g.standard_normal((10, d)).astype(np.float32)
    rows = [[j for j in range(n) if j != i] for i in range(n)]
    adj, deg = rows_to_adj(rows, n - 1)
    o.import_graph(X, adj, deg, np.ones(n, np.uint8), 0)
    gt = brute_knn(X, np.ones(n, bool), Q, n)
    for qi, q in enumerate(Q):
        C, Cd, V, Vd = o.beam_search(q, 0, n, 2 * n)
        assert sorted(V.tolist()) == list(range(n))
        assert C.tolist() == gt[qi].tolist()
    ids, _ = o.search(Q, 10, n)
    assert np.array_equal(ids, gt[:, :10].astype(np.uint32))


def test_beam_search_result_properties():
    """C sorted by (dist, id), no repeats, |C| <= l, every distance equal to
    Dist recomputed, V expanded in nondecreasing order of first appearance."""
    g = np.random.default_rng(5)
    n, d, R = 300, 16, 8
    cfg = IndexConfig("vamana", "u8", "l2", d, n, R, 16)
    o = Oracle(cfg)
    X = g.integers(0, 256, (n, d), dtype=np.uint8)
    adj = np.stack([g.choice(np.delete(np.arange(n), i), R, replace=False) for i in range(n)]).astype(np.uint32)
    o.import_graph(X, adj, np.full(n, R, np.uint32), np.ones(n, np.uint8), 0)
    for _ in range(20):
        q = g.integers(0, 256, d, dtype=np.uint8)
        C, Cd, V, Vd = o.beam_search(q, 0, 16, 32)
        assert len(C) <= 16 and len(set(C.tolist())) == len(C)
        keys = list(zip(Cd.tolist(), C.tolist()))
        assert keys == sorted(keys)
        exact = ((X[C].astype(np.int64) - q.astype(np.int64)) ** 2).sum(1)
        assert np.array_equal(Cd, exact.astype(np.float32))
        assert len(V) <= 32 and len(set(V.tolist())) == len(V)
        exact_v = ((X[V].astype(np.int64) - q.astype(np.int64)) ** 2).sum(1)
        assert np.array_equal(Vd, exact_v.astype(np.float32))


def test_search_api_pads_and_handles_empty_index():
    cfg = line_config(8, 2)
    o = Oracle(cfg)
    ids, d = o.search(np.zeros((3, 1), np.float32), 4, 4)
    assert (ids == INVALID).all() and np.isinf(d).all()
    o.insert(np.array([0, 1], np.uint32), np.array([[0.0], [1.0]], np.float32))
    ids, d = o.search(np.array([[0.2]], np.float32), 4, 4)
    assert ids[0, :2].tolist() == [0, 1] and (ids[0, 2:] == INVALID).all()
    assert np.isinf(d[0, 2:]).all()
