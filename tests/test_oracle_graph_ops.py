"""Pins of the oracle's reverse CSR (Alg. 8), medoid, batch insert (Alg. 5,
Alg. 7) and batch delete (Alg. 6, Alg. 8): a hand example, library
transposes, brute-force definitions, hand-computed CAGRA rewiring, and
graph invariants after every batch."""
import numpy as np
import pytest
import scipy.sparse as sp

from helpers import INVALID, brute_knn, canonical_rows, check_graph_invariants, line_config, rows_to_adj
from oracle.oracle import Oracle, reverse_csr
from workloads import IndexConfig, make_workload


# ---------------------------------------------------------------- reverse CSR
def test_reverse_csr_hand_example(golden):
    fx = golden("reverse_csr_example.json")
    adj, _ = rows_to_adj(fx["rows"], fx["R"])
    offs, srcs = reverse_csr(adj, np.ones(len(fx["rows"]), np.uint8))
    assert offs.tolist() == fx["expected_offsets"]
    assert srcs.tolist() == fx["expected_srcs"]


def test_reverse_csr_matches_scipy_transpose():
    g = np.random.default_rng(11)
    cap, R = 500, 7
    adj = np.full((cap, R), INVALID, np.uint32)
    active = g.random(cap) < 0.8
    for u in np.flatnonzero(active):
        k = int(g.integers(0, R + 1))
        adj[u, :k] = g.choice(np.flatnonzero(active), k, replace=False)
    offs, srcs = reverse_csr(adj, active.astype(np.uint8))
    r, c = np.nonzero(adj != INVALID)
    A = sp.csr_matrix((np.ones(len(r)), (r, adj[r, c].astype(np.int64))), shape=(cap, cap))
    T = A.T.tocsr()
    T.sort_indices()
    assert offs.tolist() == T.indptr.tolist()
    assert srcs.tolist() == T.indices.tolist()


def test_reverse_csr_ignores_inactive_rows():
    adj, _ = rows_to_adj([[1], [0], [0, 1]], 2)
    offs, srcs = reverse_csr(adj, np.array([1, 1, 0], np.uint8))
    assert offs.tolist() == [0, 1, 2, 2] and srcs.tolist() == [1, 0]


# ---------------------------------------------------------------- medoid
def _exact_u8_medoid(X, active):
    """argmin over active ids of (|x - S/n|^2, id), compared exactly as
    |n x - S|^2 with Python integers (reading Q13 for uint8)."""
    ids = np.flatnonzero(active)
    n = len(ids)
    S = [int(v) for v in X[ids].astype(np.int64).sum(0)]
    best = None
    for i in ids:
        key = sum((n * int(x) - s) ** 2 for x, s in zip(X[i], S))
        if best is None or key < best[0]:
            best = (key, int(i))
    return best[1]


def test_medoid_hand_examples(golden):
    for case in golden("medoid_examples.json")["cases"]:
        X = np.array(case["vectors"], np.uint8 if case["dtype"] == "u8" else np.float32)
        n, d = X.shape
        o = Oracle(IndexConfig("vamana", case["dtype"], "l2", d, n, 2, 4))
        o.import_graph(X, np.full((n, 2), INVALID, np.uint32), np.zeros(n, np.uint32), np.ones(n, np.uint8), INVALID)
        assert o.medoid() == case["expected"], case["name"]


@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_medoid_matches_brute_force(dtype):
    g = np.random.default_rng(12)
    cap, d = 3000, 9
    cfg = IndexConfig("vamana", dtype, "l2", d, cap, 4, 8)
    o = Oracle(cfg)
    X = g.integers(0, 256, (cap, d), dtype=np.uint8) if dtype == "u8" else \
        g.standard_normal((cap, d)).astype(np.float32)
    act = (g.random(cap) < 0.7).astype(np.uint8)
    o.import_graph(X, np.full((cap, 4), INVALID, np.uint32), np.zeros(cap, np.uint32), act, INVALID)
    ids = np.flatnonzero(act)
    if dtype == "u8":
        assert o.medoid() == _exact_u8_medoid(X, act)
    else:
        c = X[ids].astype(np.float64).mean(0)
        dd = ((X[ids].astype(np.float64) - c) ** 2).sum(1)
        assert o.medoid() == ids[np.argmin(dd)]


# ---------------------------------------------------------------- insert
def _small_u8(seed=0):
    return make_workload("sift1m_u8", seed=seed, index=dict(capacity=4000, R=16, L_build=32, dim=16),
                         stream=dict(base_n=3000, build_batch=500, n_insert=300, n_delete=300,
                                     n_query=50)).keep_vectors()


def test_insert_invariants_and_reverse_edges():
    w = _small_u8()
    o = Oracle(w.cfg)
    R, P = w.cfg.R, w.cfg.P
    before = o.export()
    for op in w.base_batches():
        assert o.insert(op.ids, op.vecs) == 0
        after = o.export()
        check_graph_invariants(after, R)
        new = set(op.ids.tolist())
        # every new node has at least one out-edge once the index has >1 point
        assert (after["deg"][op.ids] >= 1).all()
        # reverse edges: if u gained fewer edges than its free room and the
        # cap, nothing was pruned, so u keeps its old list and gains every
        # new in-neighbour
        incoming = {}
        for p in op.ids:
            for u in after["adj"][p][: after["deg"][p]]:
                incoming.setdefault(int(u), []).append(int(p))
        for u, srcs in incoming.items():
            if u in new:
                continue
            old = set(before["adj"][u][: before["deg"][u]].tolist())
            if len(old) + len(srcs) <= R and len(srcs) <= P:
                got = set(after["adj"][u][: after["deg"][u]].tolist())
                assert got == old | set(srcs), u
        before = after


def test_insert_dirty_bound():
    w = _small_u8()
    o = Oracle(w.cfg)
    batches = list(w.base_batches())
    o.insert(batches[0].ids, batches[0].vecs)
    s0 = o.stats()
    o.insert(batches[1].ids, batches[1].vecs)
    s1 = o.stats()
    assert s1["dirty"] - s0["dirty"] <= len(batches[1].ids) * w.cfg.R   # Alg. 5: |Dirty| <= B * R


def test_single_insert_into_complete_graph_prunes_all_points():
    """l >= N on a complete graph: V is every active point, so the new list
    is RobustPrune over all of them (Alg. 5 with Alg. 1 exhaustive)."""
    g = np.random.default_rng(13)
    n, d, R = 30, 4, 29
    cfg = IndexConfig("vamana", "u8", "l2", d, n + 1, R, 64, max_iters=128)
    o = Oracle(cfg)
    X = np.zeros((n + 1, d), np.uint8)
    X[:n] = g.integers(0, 256, (n, d), dtype=np.uint8)
    rows = [[j for j in range(n) if j != i] for i in range(n)] + [[]]
    adj, deg = rows_to_adj(rows, R)
    act = np.ones(n + 1, np.uint8)
    act[n] = 0
    o.import_graph(X, adj, deg, act, 0)
    x = g.integers(0, 256, (1, d), dtype=np.uint8)
    assert o.insert(np.array([n], np.uint32), x) == 0
    st = o.export()
    ref = Oracle(cfg)
    X2 = X.copy()
    X2[n] = x[0]
    ref.import_graph(X2, adj, deg, np.ones(n + 1, np.uint8), 0)
    D = np.array([ref.dist(X2[n], X2[j]) for j in range(n)], np.float32)
    expect = ref.robust_prune(n, np.arange(n, dtype=np.uint32), D)
    assert st["adj"][n][: st["deg"][n]].tolist() == sorted(expect.tolist())


def _knn_sets_u8(X, k):
    """Exact k nearest other points of every row, by (distance, id), with
    int64 arithmetic (numpy brute force)."""
    Xi = X.astype(np.int64)
    out = []
    for i in range(len(X)):
        d = ((Xi - Xi[i]) ** 2).sum(1)
        d[i] = np.iinfo(np.int64).max
        order = np.lexsort((np.arange(len(X)), d))
        out.append(set(order[:k].tolist()))
    return out


@pytest.mark.parametrize("ell", [3, 5])
def test_bootstrap_lists_are_the_batch_knn(ell):
    """Empty index (reading Q14): each new point's candidates are its
    min(B-1, l) nearest other batch points.  With alpha -> infinity (no
    pruning between distinct points) and R = l, the forward list is exactly
    those l nearest; a reverse-edge rebuild keeps the R nearest of a union
    that contains them, so every final list is the point's exact l-NN in
    the batch, whatever P is.  Checked against numpy brute force."""
    g = np.random.default_rng(14)
    n, d = 60, 6
    X = np.unique(g.integers(0, 256, (n + 10, d), dtype=np.uint8), axis=0)[:n]
    X = g.permutation(X)
    for P in (1, 64):
        cfg = IndexConfig("vamana", "u8", "l2", d, n, ell, ell, alpha=1e30, P=P)
        o = Oracle(cfg)
        assert o.insert(np.arange(n, dtype=np.uint32), X) == 0
        st = o.export()
        check_graph_invariants(st, ell)
        want = _knn_sets_u8(X, ell)
        for i in range(n):
            assert set(st["adj"][i][: st["deg"][i]].tolist()) == want[i], (P, i)


def test_bootstrap_medoid_is_the_brute_force_medoid():
    g = np.random.default_rng(14)
    n, d = 200, 6
    cfg = IndexConfig("vamana", "u8", "l2", d, n, 8, 20)
    o = Oracle(cfg)
    X = g.integers(0, 256, (n, d), dtype=np.uint8)
    o.insert(np.arange(n, dtype=np.uint32), X)
    st = o.export()
    check_graph_invariants(st, 8)
    assert st["medoid"] == _exact_u8_medoid(X, np.ones(n, bool))


# ---------------------------------------------------------------- hand examples of Alg. 5 / Alg. 6
def _line_index(coords, rows, R, medoid, extra=0, **kw):
    """A 1-D fp32 index holding `coords` (ids 0..n-1) with the given lists,
    and `extra` inactive slots after them."""
    n = len(coords)
    cfg = line_config(n + extra, R, **kw)
    o = Oracle(cfg)
    X = np.zeros((n + extra, 1), np.float32)
    X[:n, 0] = coords
    adj, deg = rows_to_adj(list(rows) + [[]] * extra, R)
    act = np.zeros(n + extra, np.uint8)
    act[:n] = 1
    o.import_graph(X, adj, deg, act, medoid)
    return o, X


def _delete_cases():
    from conftest import load_golden
    return [c["name"] for c in load_golden("delete_repair_examples.json")["cases"]]


@pytest.mark.parametrize("name", _delete_cases())
def test_delete_repair_hand_examples(golden, name):
    """Alg. 6 on a hand-derived 1-D graph: C_i without the batch, the c
    closest of C_i for every in-neighbour z, the out-neighbour direction (w
    enters the lists of its c closest points of C_i), the P cap keeping the
    smallest (Dist, src) records, the dirty rebuild with and without prune,
    and a deleted node without in-edges."""
    fx = golden("delete_repair_examples.json")
    case = next(c for c in fx["cases"] if c["name"] == name)
    coords, rows = list(fx["coords"]), [list(r) for r in fx["rows"]]
    if "extra_node" in case:
        coords.append(case["extra_node"]["coord"])
        rows.append(case["extra_node"]["row"])
    o, _ = _line_index(coords, rows, case["R"], fx["medoid"], ell=fx["ell"], P=case["P"],
                       k_repair=case["k_repair"], c=case["c"], max_iters=fx["max_iters"], alpha=fx["alpha"])
    assert o.delete(np.array(case["delete"], np.uint32)) == 0
    st = o.export()
    got = [sorted(st["adj"][u][st["adj"][u] != INVALID].tolist()) for u in range(len(coords))]
    assert got == [sorted(r) for r in case["expected_rows"]]
    assert st["medoid"] == case["expected_medoid"]
    assert not st["active"][case["delete"]].any()
    check_graph_invariants(st, case["R"])


@pytest.mark.parametrize("P", [1, 2])
def test_scratch_cap_hand_examples(golden, P):
    """Alg. 5 with the scratch capacity P (reading Q6): a target keeps the P
    records with the smallest (Dist, src); the two new points search the
    batch-start graph only."""
    fx = golden("scratch_cap_examples.json")
    case = next(c for c in fx["cases"] if c["P"] == P)
    o, _ = _line_index(fx["coords"], fx["rows"], fx["R"], fx["medoid"], extra=2, ell=fx["ell"], P=P,
                       alpha=fx["alpha"])
    ids = np.array(fx["insert_ids"], np.uint32)
    assert o.insert(ids, np.array(fx["insert_coords"], np.float32)[:, None]) == 0
    st = o.export()
    got = [sorted(st["adj"][u][st["adj"][u] != INVALID].tolist()) for u in range(4)]
    assert got == [sorted(r) for r in case["expected_rows"]]


def test_delete_without_in_edges_changes_only_out_repair_targets():
    """Special case of Alg. 6: a deleted node that no list points to has no
    in-neighbour repair, so the only lists that change are those of the
    points that receive out-neighbour repair edges: for every surviving
    out-neighbour w, the c points of C_x (the search's first k_repair
    results) closest to w.  C_x comes from the pinned BeamSearch; the c
    closest are picked with numpy."""
    w = _small_u8(seed=6)
    o = Oracle(w.cfg)
    for op in w.base_batches():
        o.insert(op.ids, op.vecs)
    st0 = o.export()
    act = np.flatnonzero(st0["active"])
    g = np.random.default_rng(7)
    x = int(np.flatnonzero(st0["active"] == 0)[0])
    outs = g.choice(act, w.cfg.R // 2, replace=False).astype(np.uint32)
    adj = st0["adj"].copy()
    adj[x] = INVALID
    adj[x, : outs.size] = outs
    deg = st0["deg"].copy()
    deg[x] = outs.size
    active = st0["active"].copy()
    active[x] = 1
    vecs = w.vectors.copy()
    vecs[x] = vecs[int(outs[0])] // 2 + 40
    o.import_graph(vecs, adj, deg, active, st0["medoid"])
    C, _, _, _ = o.beam_search(vecs[x], st0["medoid"], w.cfg.L_build, w.cfg.iters)
    Cx = [int(v) for v in C if v != x][: w.cfg.k_repair]
    V = vecs.astype(np.int64)
    targets = set()
    for wv in outs.tolist():
        cand = [y for y in Cx if y != wv]
        d = ((V[cand] - V[wv]) ** 2).sum(1)
        targets.update(np.array(cand)[np.lexsort((cand, d))][: w.cfg.c].tolist())
    assert o.delete(np.array([x], np.uint32)) == 0
    st1 = o.export()
    changed = set(np.flatnonzero(np.any(canonical_rows(st1["adj"]) != canonical_rows(adj), axis=1)).tolist())
    assert x in changed
    assert changed - {x} <= targets
    assert changed - {x}, "some target gained an edge"


@pytest.mark.parametrize("algo", ["vamana", "cagra"])
def test_oracle_determinism_threads_and_batch_order(algo):
    """Batch semantics read a snapshot and write owner-private state, so the
    result does not depend on thread count or on the order of the batch."""
    idx = dict(capacity=3000, R=12, L_build=24, dim=12)
    st = dict(base_n=2000, build_batch=500, n_insert=300, n_delete=300, n_query=20)
    name = "sift1m_u8"
    if algo == "cagra":
        idx.update(algo="cagra", metric="l2")
    outs = []
    for threads, permute in [(1, False), (8, False), (8, True)]:
        w = make_workload(name, seed=3, index=idx, stream=st)
        o = Oracle(w.cfg, threads=threads)
        g = np.random.default_rng(99)
        ops = list(w.base_batches()) + [op for _, ops in w.rounds(2) for op in ops]
        for op in ops:
            if op.kind == "insert":
                perm = g.permutation(len(op.ids)) if permute else np.arange(len(op.ids))
                assert o.insert(op.ids[perm], op.vecs[perm]) == 0
            elif op.kind == "delete":
                perm = g.permutation(len(op.ids)) if permute else np.arange(len(op.ids))
                assert o.delete(op.ids[perm]) == 0
        outs.append(o.export())
    for s in outs[1:]:
        if algo == "vamana":
            assert np.array_equal(canonical_rows(s["adj"]), canonical_rows(outs[0]["adj"]))
        else:
            assert np.array_equal(s["adj"], outs[0]["adj"])
        assert np.array_equal(s["active"], outs[0]["active"]) and s["medoid"] == outs[0]["medoid"]


# ---------------------------------------------------------------- delete
def test_delete_invariants_medoid_and_recall():
    w = _small_u8(seed=1)
    o = Oracle(w.cfg)
    for op in w.base_batches():
        o.insert(op.ids, op.vecs)
    for r, ops in w.rounds(3):
        for op in ops:
            if op.kind == "insert":
                assert o.insert(op.ids, op.vecs) == 0
            elif op.kind == "delete":
                med0 = o.export()["medoid"]
                assert o.delete(op.ids) == 0
                st = o.export()
                check_graph_invariants(st, w.cfg.R)
                assert not st["active"][op.ids].any()
                assert (st["adj"][op.ids] == INVALID).all() and (st["deg"][op.ids] == 0).all()
                if med0 in set(op.ids.tolist()):
                    assert st["medoid"] == o.medoid()
                else:
                    assert st["medoid"] == med0
            else:
                ids, _ = o.search(op.vecs, 10, 64)
                gt = brute_knn(w.vectors, w.active, op.vecs, 10)
                rec = np.mean([len(set(a) & set(b)) for a, b in zip(ids.tolist(), gt.tolist())]) / 10
                assert rec >= 0.9


def test_delete_medoid_reinstalls_brute_force_medoid():
    w = _small_u8(seed=2)
    o = Oracle(w.cfg)
    for op in w.base_batches():
        o.insert(op.ids, op.vecs)
    med = o.export()["medoid"]
    assert o.delete(np.array([med], np.uint32)) == 0
    st = o.export()
    assert st["medoid"] == _exact_u8_medoid(w.vectors, st["active"].astype(bool))
    check_graph_invariants(st, w.cfg.R)


def test_delete_everything_empties_the_index():
    cfg = line_config(20, 4)
    o = Oracle(cfg)
    X = np.arange(20, dtype=np.float32)[:, None]
    o.insert(np.arange(20, dtype=np.uint32), X)
    assert o.delete(np.arange(20, dtype=np.uint32)[::-1].copy()) == 0
    st = o.export()
    check_graph_invariants(st, 4)
    assert not st["active"].any() and st["medoid"] == INVALID
    ids, d = o.search(X[:2], 3, 4)
    assert (ids == INVALID).all()


def test_delete_in_neighbours_are_all_repaired():
    """Every node that pointed at a deleted node loses that edge (exact
    in-neighbours from the reverse graph), whatever the search visited."""
    w = _small_u8(seed=4)
    o = Oracle(w.cfg)
    for op in w.base_batches():
        o.insert(op.ids, op.vecs)
    st0 = o.export()
    act = np.flatnonzero(st0["active"])
    dele = np.random.default_rng(5).choice(act, 400, replace=False).astype(np.uint32)
    o.delete(dele)
    st1 = o.export()
    check_graph_invariants(st1, w.cfg.R)
    # every in-neighbour of the batch was repaired: it lost its edges into
    # the batch and received replacements, so its list is not empty
    offs, srcs = reverse_csr(st0["adj"], st0["active"])
    B = set(dele.tolist())
    touched = set()
    for p in dele:
        touched.update(x for x in srcs[offs[p]:offs[p + 1]].tolist() if x not in B)
    assert touched
    for u in touched:
        assert st1["deg"][u] >= 1
        assert not np.isin(st1["adj"][u], dele).any()


# ---------------------------------------------------------------- CAGRA
def test_cagra_insert_hand_example(golden):
    fx = golden("cagra_examples.json")["insert"]
    n = len(fx["coords"])
    cfg = line_config(n + 1, 3, ell=fx["ell"], algo="cagra")
    o = Oracle(cfg)
    X = np.zeros((n + 1, 1), np.float32)
    X[:n, 0] = fx["coords"]
    adj, deg = rows_to_adj(fx["rows"] + [[]], 3)
    act = np.ones(n + 1, np.uint8)
    act[n] = 0
    o.import_graph(X, adj, deg, act, fx["medoid"])
    assert o.insert(np.array([fx["new_id"]], np.uint32), np.array([[fx["new_coord"]]], np.float32)) == 0
    st = o.export()
    for k, row in fx["expected_rows"].items():
        assert st["adj"][int(k)].tolist() == row, k


def test_cagra_insert_fills_an_empty_slot_first(golden):
    """Reading Q16b: a CAGRA list below the fixed degree takes the new point
    into its first empty slot; full lists follow the detour rule."""
    fx = golden("cagra_examples.json")["insert_free_slot"]
    n = len(fx["coords"])
    cfg = line_config(n + 1, 3, ell=fx["ell"], algo="cagra")
    o = Oracle(cfg)
    X = np.zeros((n + 1, 1), np.float32)
    X[:n, 0] = fx["coords"]
    adj, deg = rows_to_adj(fx["rows"] + [[]], 3)
    act = np.ones(n + 1, np.uint8)
    act[n] = 0
    o.import_graph(X, adj, deg, act, fx["medoid"])
    assert o.insert(np.array([fx["new_id"]], np.uint32), np.array([[fx["new_coord"]]], np.float32)) == 0
    st = o.export()
    for k, row in fx["expected_rows"].items():
        assert st["adj"][int(k)].tolist() == row, k
    assert st["deg"][0] == 3


def test_cagra_delete_hand_example(golden):
    fx = golden("cagra_examples.json")["delete"]
    n = len(fx["coords"])
    cfg = line_config(n, 3, algo="cagra")
    o = Oracle(cfg)
    X = np.array(fx["coords"], np.float32)[:, None]
    adj, deg = rows_to_adj(fx["rows"], 3)
    o.import_graph(X, adj, deg, np.ones(n, np.uint8), fx["medoid"])
    assert o.delete(np.array(fx["delete"], np.uint32)) == 0
    st = o.export()
    for k, row in fx["expected_rows"].items():
        assert st["adj"][int(k)].tolist() == row, k


def _small_cagra(seed=0):
    return make_workload("glove1m_cagra", seed=seed, index=dict(capacity=4000, R=16, L_build=32, dim=16),
                         stream=dict(base_n=3000, build_batch=500, n_insert=300, n_delete=600,
                                     n_query=50)).keep_vectors()


def test_cagra_detour_invariant_and_delete_rules():
    """Insert: whenever p replaced r in q's list, r is in N_out(p) (the path
    q -> p -> r exists).  Delete: no edge into the batch survives, and every
    replacement r comes from the deleted node's list, is outside the batch,
    differs from u and was not already in u's list."""
    w = _small_cagra()
    o = Oracle(w.cfg)
    for op in w.base_batches():
        o.insert(op.ids, op.vecs)
    for r, ops in w.rounds(2):
        for op in ops:
            st0 = o.export()
            if op.kind == "insert":
                assert o.insert(op.ids, op.vecs) == 0
                st1 = o.export()
                new = set(op.ids.tolist())
                changed = (st0["adj"] != st1["adj"]) & (st0["adj"] != INVALID)
                for u, s in zip(*np.nonzero(changed)):
                    p, r_old = int(st1["adj"][u, s]), int(st0["adj"][u, s])
                    assert p in new
                    assert r_old in set(st1["adj"][p].tolist())
            elif op.kind == "delete":
                assert o.delete(op.ids) == 0
                st1 = o.export()
                check_graph_invariants(st1, w.cfg.R)
                B = set(op.ids.tolist())
                changed = (st0["adj"] != st1["adj"])
                for u, s in zip(*np.nonzero(changed)):
                    if u in B:
                        continue
                    p, r_new = int(st0["adj"][u, s]), int(st1["adj"][u, s])
                    assert p in B
                    if r_new != INVALID:
                        assert r_new in set(st0["adj"][p].tolist()) and r_new not in B and r_new != u
                        assert r_new not in set(st0["adj"][u].tolist())


# ---------------------------------------------------------------- validation
def test_validation_leaves_state_untouched():
    cfg = line_config(10, 3)
    o = Oracle(cfg)
    X = np.arange(6, dtype=np.float32)[:, None]
    assert o.insert(np.arange(6, dtype=np.uint32), X) == 0
    st0 = o.export()
    assert o.insert(np.array([6, 6], np.uint32), X[:2]) == -2          # repeated id
    assert o.insert(np.array([3], np.uint32), X[:1]) == -2             # already active
    assert o.insert(np.array([10], np.uint32), X[:1]) == -2            # out of range
    assert o.insert(np.array([7], np.uint32), np.array([[np.nan]], np.float32)) == -1
    assert o.delete(np.array([8], np.uint32)) == -2                    # not active
    assert o.delete(np.array([1, 1], np.uint32)) == -2
    assert o.insert(np.zeros(0, np.uint32), X[:0]) == 0 and o.delete(np.zeros(0, np.uint32)) == 0
    st1 = o.export()
    for k in ("adj", "deg", "active"):
        assert np.array_equal(st0[k], st1[k])
    with pytest.raises(ValueError):
        o.search(X[:1], 5, 4)                                          # k > beam
