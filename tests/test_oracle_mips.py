"""Pins of the oracle's MIPS-to-L2 augmentation (Section 5.4): the stored
row is [x, sqrt(M^2 - |x|^2)] and the query [q, 0]; the squared L2
distance of the two is M^2 + |q|^2 - 2<x, q>, so L2 order on stored rows is
inner-product order.  Checked against exact rational arithmetic, numpy
inner products, and exhaustive search."""
import math
from fractions import Fraction

import numpy as np

from helpers import INVALID, rows_to_adj
from oracle.oracle import Oracle
from workloads import IndexConfig


def _cfg(n, d=8, M=5.0, R=None, ell=16):
    return IndexConfig("vamana", "f32", "mips", d, n, R or n - 1, ell, max_iters=4 * n, mips_norm=M)


def test_augmented_coordinate_is_the_rounded_exact_root():
    g = np.random.default_rng(1)
    o = Oracle(_cfg(4, d=24, M=7.5))
    for _ in range(300):
        x = g.standard_normal(24) * g.uniform(0.1, 1.4)
        x = (x * min(1.0, 7.4 / np.linalg.norm(x))).astype(np.float32)
        row, rc = o.store_row(x)
        assert rc == 0 and np.array_equal(row[:24], x)
        t = Fraction(7.5) ** 2 - sum(Fraction(float(v)) ** 2 for v in x)
        exact = math.sqrt(t.numerator / t.denominator) if t > 0 else 0.0
        ref = np.float32(exact)
        # fp64 sum and fp64 root, rounded once to fp32: equal, or one fp32 ulp
        assert abs(int(row[24].view(np.int32)) - int(ref.view(np.int32))) <= 1
        q, rc = o.store_row(x, is_query=True)
        assert rc == 0 and q[24] == 0.0 and np.array_equal(q[:24], x)


def test_norm_above_the_bound_is_rejected_before_any_change():
    o = Oracle(_cfg(6, d=4, M=2.0))
    x = np.array([[1.0, 1.0, 1.0, 1.0], [0.5, 0.0, 0.0, 0.0]], np.float32)   # norms 2.0 and 0.5
    assert o.store_row(x[0])[1] == 0
    assert o.store_row(np.array([1.5, 1.5, 0, 0], np.float32))[1] == -1      # norm 2.12 > 2
    assert o.insert(np.array([0, 1], np.uint32), x) == 0
    st0 = o.export()
    assert o.insert(np.array([2], np.uint32), np.array([[1.5, 1.5, 0, 0]], np.float32)) == -1
    st1 = o.export()
    assert np.array_equal(st0["active"], st1["active"])


def test_l2_on_stored_rows_is_the_inner_product_identity():
    g = np.random.default_rng(2)
    M = 6.0
    o = Oracle(_cfg(4, d=16, M=M))
    for _ in range(200):
        x = (g.standard_normal(16) * 0.9).astype(np.float32)
        q = g.standard_normal(16).astype(np.float32)
        xs, _ = o.store_row(x)
        qs, _ = o.store_row(q, is_query=True)
        d = o.dist(xs, qs)
        want = M * M + float(np.dot(q.astype(np.float64), q)) - 2.0 * float(np.dot(x.astype(np.float64), q))
        assert abs(d - want) <= 1e-5 * max(abs(want), 1.0)


def test_bruteforce_and_exhaustive_search_return_the_largest_inner_products():
    g = np.random.default_rng(3)
    n, d, M = 60, 8, 5.0
    X = g.standard_normal((n, d)).astype(np.float32)
    X *= np.minimum(1.0, 0.99 * M / np.linalg.norm(X, axis=1, keepdims=True)).astype(np.float32)
    o = Oracle(_cfg(n, d=d, M=M, ell=n))
    adj, deg = rows_to_adj([[j for j in range(n) if j != i] for i in range(n)], n - 1)
    o.import_graph(X, adj, deg, np.ones(n, np.uint8), 0)
    Q = g.standard_normal((12, d)).astype(np.float32)
    ids, _ = o.bruteforce_knn(Q, 5)
    sids, _ = o.search(Q, 5, n)
    ip = Q.astype(np.float64) @ X.astype(np.float64).T
    want = np.argsort(-ip, axis=1, kind="stable")[:, :5]
    assert np.array_equal(ids.astype(np.int64), want)
    assert np.array_equal(sids.astype(np.int64), want)
