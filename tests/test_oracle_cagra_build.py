"""Pins of the oracle's CAGRA graph construction (Section 2.2 on CAGRA;
Section 4.2, CAGRA graph construction): hand-traced NN-Descent rounds,
convergence to the exact k-NN graph on small inputs, hand examples of the
rank-based pruning and the reverse-edge merge, and the properties of the
built graph."""
import numpy as np
import pytest

from helpers import INVALID
from oracle.oracle import Oracle, rank_prune, reverse_merge
from workloads import IndexConfig, make_workload
from workloads.generators import cagra_init_lists


def _cfg(dim, dtype="f32", metric="l2", R=2, capacity=4096):
    return IndexConfig(algo="cagra", dtype=dtype, metric=metric, dim=dim, capacity=capacity, R=R, L_build=16)


def _exact_lists(x, k, metric="l2"):
    """k nearest other points by (distance, id), distances as the method
    defines them (exact for uint8; fp64 sums rounded once for fp32)."""
    xd = x.astype(np.float64)
    if metric == "l2":
        D = ((xd[:, None, :] - xd[None, :, :]) ** 2).sum(-1)
    else:
        D = -(xd @ xd.T)
    D = D.astype(np.float32) if x.dtype != np.uint8 else D.astype(np.float32)
    n = len(x)
    out = np.empty((n, k), np.int64)
    for u in range(n):
        order = sorted((float(D[u, v]), v) for v in range(n) if v != u)
        out[u] = [v for _, v in order[:k]]
    return out


# ---------------------------------------------------------------- NN-Descent
def test_nn_descent_hand_rounds(golden):
    fx = golden("cagra_build_examples.json")["nn_descent"]
    x = np.array(fx["x"], np.float32)[:, None]
    init = np.array(fx["init"], np.uint32)
    for rounds, exp in fx["rounds"].items():
        o = Oracle(_cfg(1))
        ids, d = o.nn_descent(x, init, fx["knn"], int(rounds), fx["sample"])
        assert ids.tolist() == exp["ids"], rounds
        assert d.tolist() == exp["d"], rounds


@pytest.mark.parametrize("dtype,metric,seed", [("f32", "l2", 0), ("f32", "l2", 1), ("u8", "l2", 2),
                                               ("f32", "ip", 3)])
def test_nn_descent_finds_nearly_all_of_the_exact_knn_graph(dtype, metric, seed):
    """NN-Descent is approximate (it stops once no sampled join improves a
    list), but on small inputs it recovers nearly every true neighbour."""
    g = np.random.default_rng(seed)
    n, dim, K = 160, 6, 8
    if dtype == "u8":
        x = g.integers(0, 256, size=(n, dim)).astype(np.uint8)
    else:
        x = g.standard_normal((n, dim)).astype(np.float32)
        if metric == "ip":
            x /= np.linalg.norm(x, axis=1, keepdims=True)
    o = Oracle(_cfg(dim, dtype, metric))
    ids, _ = o.nn_descent(x, cagra_init_lists(n, K, seed), K, 30, K)
    ex = _exact_lists(x, K, metric)
    found = np.mean([len(set(ids[u].tolist()) & set(ex[u].tolist())) / K for u in range(n)])
    assert found >= 0.97
    # and far more than the random start
    init = cagra_init_lists(n, K, seed)
    assert np.mean([len(set(init[u].tolist()) & set(ex[u].tolist())) / K for u in range(n)]) < 0.2


def test_nn_descent_lists_are_valid_and_never_get_worse():
    g = np.random.default_rng(7)
    n, dim, K, S = 300, 8, 12, 4
    x = g.standard_normal((n, dim)).astype(np.float32)
    init = cagra_init_lists(n, K, 7)
    xd = x.astype(np.float64)
    prev = None
    for it in range(0, 5):
        ids, d = Oracle(_cfg(dim)).nn_descent(x, init, K, it, S)
        for u in range(n):
            row = ids[u].astype(np.int64)
            assert len(set(row.tolist())) == K and u not in row
            dd = ((xd[u] - xd[row]) ** 2).sum(1).astype(np.float32)
            assert (dd == d[u]).all()
            keys = list(zip(d[u].tolist(), row.tolist()))
            assert keys == sorted(keys)
        if prev is not None:  # the K-th key of every list never increases
            assert all((d[u, -1], ids[u, -1]) <= (prev[1][u, -1], prev[0][u, -1]) for u in range(n))
        prev = (ids, d)


# ---------------------------------------------------------------- rank-based pruning, reverse edges
def test_rank_prune_hand_example(golden):
    fx = golden("cagra_build_examples.json")["rank_prune"]
    P = rank_prune(np.array(fx["lists"], np.uint32), fx["R"])
    assert P.tolist() == fx["pruned"]


def test_reverse_merge_hand_example(golden):
    fx = golden("cagra_build_examples.json")["reverse_merge"]
    out, nout = reverse_merge(np.array(fx["pruned"], np.uint32))
    assert out.tolist() == fx["out"]
    assert nout.tolist() == [len(r) for r in fx["out"]]


def _random_lists(n, K, seed):
    return cagra_init_lists(n, K, seed)


def test_rank_prune_properties():
    n, K = 200, 10
    L = _random_lists(n, K, 5)
    P = rank_prune(L, K)  # R = K: a reordering of each list
    for u in range(n):
        assert sorted(P[u].tolist()) == sorted(L[u].tolist())
        assert P[u, 0] == L[u, 0]  # the nearest neighbour has no detourable route
    P4 = rank_prune(L, 4)
    assert (P4 == P[:, :4]).all()  # pruning keeps a prefix of the (routes, rank) order


def test_reverse_merge_properties():
    n, R = 300, 8
    P = rank_prune(_random_lists(n, 16, 9), R)
    out, nout = reverse_merge(P)
    rev = [set() for _ in range(n)]
    for u in range(n):
        for v in P[u]:
            rev[int(v)].add(u)
    for y in range(n):
        row = out[y, :nout[y]].tolist()
        assert len(set(row)) == len(row) and y not in row
        assert row[:R // 2] == P[y, :R // 2].tolist()
        assert set(row) <= set(P[y].tolist()) | rev[y]
        assert nout[y] == min(R, len(set(P[y].tolist()) | rev[y]))


# ---------------------------------------------------------------- the whole construction
def _small_cagra(n=600, R=8):
    return make_workload("glove1m_cagra", seed=4, index=dict(capacity=n + 200, R=R, L_build=32),
                         stream=dict(base_n=n, build_batch=n, n_insert=50, n_delete=50, n_query=50))


def test_build_is_the_composition_of_the_three_steps():
    w = _small_cagra()
    op = next(iter(w.base_batches()))
    K, S, iters = 16, 8, 3
    init = cagra_init_lists(op.ids.size, K, 2)
    o = Oracle(w.cfg)
    assert o.build_cagra(op.ids, op.vecs, init, K, iters, S) == 0
    st = o.export()
    lists, _ = Oracle(w.cfg).nn_descent(op.vecs, init, K, iters, S)
    out, nout = reverse_merge(rank_prune(lists, w.cfg.R))
    for p, i in enumerate(op.ids):
        assert st["deg"][i] == nout[p] == w.cfg.R
        assert st["adj"][i].tolist() == op.ids[out[p]].tolist()
    assert st["active"][op.ids].all() and st["active"].sum() == op.ids.size
    assert st["medoid"] in set(op.ids.tolist())


def test_build_rejects_bad_input_and_leaves_the_index_empty():
    w = _small_cagra(n=100)
    op = next(iter(w.base_batches()))
    K = 16
    good = cagra_init_lists(op.ids.size, K, 1)
    o = Oracle(w.cfg)
    bad = good.copy(); bad[3, 0] = 3                      # itself
    assert o.build_cagra(op.ids, op.vecs, bad, K, 2, 4) != 0
    bad = good.copy(); bad[5, 1] = bad[5, 0]              # repeated
    assert o.build_cagra(op.ids, op.vecs, bad, K, 2, 4) != 0
    bad = good.copy(); bad[7, 2] = op.ids.size            # out of range
    assert o.build_cagra(op.ids, op.vecs, bad, K, 2, 4) != 0
    small = cagra_init_lists(op.ids.size, w.cfg.R - 1, 1)
    assert o.build_cagra(op.ids, op.vecs, small, w.cfg.R - 1, 2, 4) != 0   # K < R
    assert o.export()["active"].sum() == 0
    assert o.build_cagra(op.ids, op.vecs, good, K, 2, 4) == 0
    assert o.build_cagra(op.ids, op.vecs, good, K, 2, 4) != 0    # no longer empty
