"""Pins of the oracle's GrANDRobustPrune (Alg. 4): hand-checked examples,
special cases that reduce to k-NN selection, and an independent property
checker that fixes the greedy output uniquely."""
import numpy as np
import pytest

from helpers import INVALID, line_config
from oracle.oracle import Oracle
from workloads import IndexConfig


def _line_oracle(coords, R, rule, alpha):
    ids = [int(k) for k in coords]
    cap = max(ids) + 1
    cfg = line_config(cap, R, alpha=alpha, prune_rule=rule)
    o = Oracle(cfg)
    vecs = np.zeros((cap, 1), np.float32)
    for k, x in coords.items():
        vecs[int(k), 0] = x
    adj = np.full((cap, R), INVALID, np.uint32)
    o.import_graph(vecs, adj, np.zeros(cap, np.uint32), np.ones(cap, np.uint8), 0)
    return o, vecs


@pytest.mark.parametrize("rule", ["alpha_on_sq", "alpha_on_l2"])
def test_prune_hand_examples(golden, rule):
    fx = golden("robust_prune_examples.json")
    for ex in fx["examples"]:
        o, vecs = _line_oracle(ex["coords"], ex["R"], rule, ex["alpha"])
        p = ex["p"]
        cand = np.array(ex["candidates"], np.uint32)
        D = np.array([o.dist(vecs[p], vecs[c]) for c in cand], np.float32)
        L = o.robust_prune(p, cand, D)
        assert L.tolist() == ex["expected"][rule], ex["name"]


def _random_set(g, dtype, n, d):
    if dtype == "u8":
        return g.integers(0, 256, (n, d), dtype=np.uint8)
    # small integers stored as fp32: distances are exact, so the checker's
    # numpy arithmetic agrees with the oracle bit for bit
    return g.integers(-8, 9, (n, d)).astype(np.float32)


def _exact_dist(X, i, j):
    a = X[i].astype(np.int64)
    b = X[j].astype(np.int64)
    return float(((a - b) ** 2).sum())


@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_prune_large_alpha_is_knn_selection(dtype):
    """alpha -> infinity invalidates only exact duplicates of a selected
    point, so on distinct points the output is the R nearest by (D, id)."""
    g = np.random.default_rng(7)
    n, d, R = 60, 6, 10
    cfg = IndexConfig("vamana", dtype, "l2", d, n, R, 8, alpha=1e30)
    o = Oracle(cfg)
    X = _random_set(g, dtype, n, d)
    X = np.unique(X, axis=0)[: n]
    while len(X) < n:
        X = np.vstack([X, _random_set(g, dtype, 1, d)])
        X = np.unique(X, axis=0)
    X = g.permutation(X)
    o.import_graph(X, np.full((n, R), INVALID, np.uint32), np.zeros(n, np.uint32), np.ones(n, np.uint8), 0)
    cand = np.arange(1, n, dtype=np.uint32)
    D = np.array([_exact_dist(X, 0, j) for j in cand], np.float32)
    L = o.robust_prune(0, cand, D)
    order = np.lexsort((cand, D))
    assert L.tolist() == cand[order[:R]].tolist()


def test_prune_zero_alpha_keeps_only_the_nearest():
    """alpha = 0 makes every later candidate redundant: L = [nearest]."""
    g = np.random.default_rng(8)
    n, d = 30, 4
    cfg = IndexConfig("vamana", "u8", "l2", d, n, 8, 8, alpha=0.0)
    o = Oracle(cfg)
    X = _random_set(g, "u8", n, d)
    o.import_graph(X, np.full((n, 8), INVALID, np.uint32), np.zeros(n, np.uint32), np.ones(n, np.uint8), 0)
    cand = np.arange(1, n, dtype=np.uint32)
    D = np.array([_exact_dist(X, 0, j) for j in cand], np.float32)
    L = o.robust_prune(0, cand, D)
    assert L.tolist() == [int(cand[np.lexsort((cand, D))[0]])]


def test_prune_drops_self_invalid_and_repeats():
    o, vecs = _line_oracle({"0": 0.0, "1": 1.0, "2": -3.0}, 3, "alpha_on_sq", 1.2)
    cand = np.array([0, 1, INVALID, 1, 2], np.uint32)
    D = np.array([0.0, 1.0, 5.0, 1.0, 9.0], np.float32)
    assert o.robust_prune(0, cand, D).tolist() == [1, 2]


def check_prune_properties(X, p, cand, D, L, alpha, R, coef):
    """Independent checker of the greedy alpha-pruning output:
    (i) L is ascending in (D, id); (ii) no selected s dominates a later
    selected t (coef * Dist(s,t) > D_t); (iii) every rejected candidate
    ranked before the last selected one (all of them when |L| < R) is
    dominated by an earlier selected s."""
    key = {int(c): (float(dv), int(c)) for c, dv in zip(cand, D)}
    Ls = [int(x) for x in L]
    assert len(Ls) <= R and len(set(Ls)) == len(Ls)
    assert [key[x] for x in Ls] == sorted(key[x] for x in Ls)
    for a in range(len(Ls)):
        for b in range(a + 1, len(Ls)):
            assert coef * _exact_dist(X, Ls[a], Ls[b]) > key[Ls[b]][0]
    rejected = [c for c in key if c not in Ls and c != p]
    last = key[Ls[-1]] if Ls else None
    for c in rejected:
        if len(Ls) == R and key[c] > last:
            continue
        dominated = any(key[s] < key[c] and coef * _exact_dist(X, s, c) <= key[c][0] for s in Ls)
        assert dominated, f"candidate {c} was neither selected nor dominated"


@pytest.mark.parametrize("rule", ["alpha_on_sq", "alpha_on_l2"])
@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_prune_property_checker_random(dtype, rule):
    g = np.random.default_rng(9)
    n, d, R, alpha = 120, 5, 12, 1.2
    cfg = IndexConfig("vamana", dtype, "l2", d, n, R, 8, alpha=alpha, prune_rule=rule)
    o = Oracle(cfg)
    coef = float(np.float32(alpha)) ** (2 if rule == "alpha_on_l2" else 1)
    for trial in range(15):
        X = _random_set(g, dtype, n, d)
        o.import_graph(X, np.full((n, R), INVALID, np.uint32), np.zeros(n, np.uint32),
                       np.ones(n, np.uint8), 0)
        p = int(g.integers(0, n))
        cand = g.choice(np.delete(np.arange(n), p), size=80, replace=False).astype(np.uint32)
        D = np.array([_exact_dist(X, p, j) for j in cand], np.float32)
        L = o.robust_prune(p, cand, D)
        assert len(L) >= 1
        check_prune_properties(X, p, cand, D, L, alpha, R, coef)
