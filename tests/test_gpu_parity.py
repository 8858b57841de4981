"""GPU parity: the HIP path (through the C ABI) against the oracle on the
same seeded inputs.  Lockstep tests import the oracle's state into the GPU,
apply one batch on both and compare the resulting states; free-running
tests run whole workloads on both independently."""
import numpy as np
import pytest

from helpers import INVALID, brute_knn, check_graph_invariants
from oracle.oracle import Oracle, reverse_csr
from parity import compare_search, compare_states, recall, say, tie_context, to_gpu
from workloads import make_workload

pytestmark = pytest.mark.gpu

# (workload, index overrides, stream overrides, allowed fraction of differing lists)
CASES = {
    "tiny_f32_d32": ("tiny", dict(capacity=12_000), {}, 0.001),
    "u8_d128": ("sift1m_u8", dict(capacity=12_000),
                dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    # uint8 variants that take the other matrix-core paths: 64-byte rows with
    # c = 4 (one K step per tile, 4-key repair lists), and P = 100 (R + P >
    # 128 candidates: the LDS-staged prune)
    "u8_d64_c4": ("sift1m_u8", dict(capacity=12_000, dim=64, c=4, k_repair=40),
                  dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    "u8_d128_p100": ("sift1m_u8", dict(capacity=12_000, P=100, c=3),
                     dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    # the Euclidean reading of the alpha test (alpha^2 on squared distances)
    "u8_d128_l2": ("sift1m_u8", dict(capacity=12_000, prune_rule="alpha_on_l2"),
                   dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    "f32_d96": ("deep1m_window", dict(capacity=9_000),
                dict(base_n=6_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.001),
    "cagra_ip_d100": ("glove1m_cagra", dict(capacity=9_000),
                      dict(base_n=6_000, build_batch=2_000, n_insert=1_000, n_delete=2_000, n_query=200), 0.001),
    "f32_d960": ("gist500k", dict(capacity=3_500),
                 dict(base_n=2_500, build_batch=1_250, n_insert=500, n_delete=500, n_query=100), 0.001),
    # dispatch branches of their own: c = 5 (one wave per deleted node in the
    # repair), uint8 rows of 96 bytes (no matrix-core path), CAGRA R = 30
    # (lists not 16-byte aligned), and the edge parameters P = 1 (every
    # target over the scratch cap), c = 0 (no replacement edges) and R = 1
    "u8_d128_c5": ("sift1m_u8", dict(capacity=12_000, c=5),
                   dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    "u8_d96": ("sift1m_u8", dict(capacity=12_000, dim=96),
               dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    "cagra_ip_r30": ("glove1m_cagra", dict(capacity=9_000, R=30),
                     dict(base_n=6_000, build_batch=2_000, n_insert=1_000, n_delete=2_000, n_query=200), 0.001),
    "u8_d128_p1": ("sift1m_u8", dict(capacity=12_000, P=1),
                   dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    "u8_d128_c0": ("sift1m_u8", dict(capacity=12_000, c=0),
                   dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    "u8_d128_r1": ("sift1m_u8", dict(capacity=12_000, R=1),
                   dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    # uint8 points within about one unit of their component's centre: the
    # distances among a node's candidates repeat often, so ties broken by id
    # decide searches, prunes, repairs and the rebuild's key order; with
    # alpha = 1.25 (exact in binary) alpha * Dist also equals D_p often, the
    # boundary of the prune test
    "u8_d128_ties": ("sift1m_u8", dict(capacity=12_000, alpha=1.25),
                     dict(base_n=8_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.0),
    # inner-product data through the L2 augmentation (Section 5.4)
    "mips_f32_d64": ("ip768_mips", dict(capacity=9_000, dim=64),
                     dict(base_n=6_000, build_batch=2_000, n_insert=1_000, n_delete=1_000, n_query=200), 0.001),
}


def _ctx(case, w, pre_state, batch_ids):
    """Tie-tracing context of a batch for fp32 cases (None for uint8, whose
    distances are exact integers on both sides: no mismatch is allowed)."""
    if w.cfg.dtype != "f32":
        return None
    pre = Oracle(w.cfg)
    pre.import_graph(w.vectors, pre_state["adj"], pre_state["deg"], pre_state["active"], pre_state["medoid"])
    coef = None
    if w.cfg.algo == "vamana":
        a = float(np.float32(w.cfg.alpha))
        coef = a * a if w.cfg.prune_rule == "alpha_on_l2" else a
    return tie_context(pre, w, w.cfg.algo, batch_ids, coef)

_BASE = {}


# sampler arguments of the cases that change them (mixture components, sigma)
SAMPLER = {"u8_d128_ties": (16, 0.7)}


def _workload(case):
    name, idx, st, _ = CASES[case]
    return make_workload(name, seed=7, index=idx or None, stream=st or None,
                         sampler_args=SAMPLER.get(case)).keep_vectors()


def base_state(case):
    """(workload positioned after its base batches, oracle with the base
    graph).  The oracle's base graph is built once per case and re-imported."""
    w = _workload(case)
    ops = list(w.base_batches())
    if case not in _BASE:
        o = Oracle(w.cfg)
        for op in ops:
            assert o.insert(op.ids, op.vecs) == 0
        _BASE[case] = o.export()
    st = _BASE[case]
    o = Oracle(w.cfg)
    o.import_graph(w.vectors, st["adj"], st["deg"], st["active"], st["medoid"])
    return w, o


def gpu_index(cfg, **kw):
    from paper_2608_21163_amd import GrandIndex
    return GrandIndex.from_config(cfg, max_batch=2_000, **kw)


@pytest.mark.parametrize("case", list(CASES))
def test_bootstrap_batch_matches_oracle(case):
    say(f"[bootstrap] {case}")
    w = _workload(case)
    op = next(w.base_batches())
    o = Oracle(w.cfg)
    g = gpu_index(w.cfg)
    pre = o.export()
    assert o.insert(op.ids, op.vecs) == 0
    g.insert(op.ids, op.vecs)
    gst, ost = g.export(), o.export()
    check_graph_invariants(gst, w.cfg.R)
    n = compare_states(gst, ost, w.cfg.algo, CASES[case][3], ctx=_ctx(case, w, pre, op.ids))
    say(f"  {n} differing lists")


@pytest.mark.parametrize("case", list(CASES))
def test_search_matches_oracle(case):
    say(f"[search] {case}")
    w, o = base_state(case)
    g = gpu_index(w.cfg)
    to_gpu(o, g, w)
    q = next(op for _, ops in w.rounds(1) for op in ops if op.kind == "search").vecs
    k, beam = w.spec.k, w.spec.beam
    gi, gd = g.search(q, k, beam)
    oi, od = o.search(q, k, beam)
    n = compare_search(gi, gd, oi, od, allow_frac=0.01 if w.cfg.dtype == "f32" else 0.0)
    # the k = beam edge and a small beam
    gi, gd = g.search(q[:20], 16, 16)
    oi, od = o.search(q[:20], 16, 16)
    n += compare_search(gi, gd, oi, od, allow_frac=0.05 if w.cfg.dtype == "f32" else 0.0)
    say(f"  {n} query rows differ (each by a distance tie)")


@pytest.mark.parametrize("case", list(CASES))
def test_reverse_graph_is_bit_exact(case):
    say(f"[reverse csr] {case}")
    w, o = base_state(case)
    g = gpu_index(w.cfg)
    ost = to_gpu(o, g, w)
    gst = g.export(with_reverse=True)
    offs, srcs = reverse_csr(ost["adj"], ost["active"])
    assert np.array_equal(gst["rev_offsets"], offs)
    assert np.array_equal(gst["rev_srcs"], srcs)


@pytest.mark.parametrize("case", list(CASES))
def test_insert_lockstep(case):
    say(f"[insert lockstep] {case}")
    w, o = base_state(case)
    g = gpu_index(w.cfg)
    for r, ops in w.rounds(2):
        for op in ops:
            if op.kind != "insert":
                if op.kind == "delete":
                    assert o.delete(op.ids) == 0
                continue
            pre = to_gpu(o, g, w)
            assert o.insert(op.ids, op.vecs) == 0
            g.insert(op.ids, op.vecs)
            gst, ost = g.export(), o.export()
            check_graph_invariants(gst, w.cfg.R)
            n = compare_states(gst, ost, w.cfg.algo, CASES[case][3], ctx=_ctx(case, w, pre, op.ids))
            say(f"  round {r}: {n} differing lists")


@pytest.mark.parametrize("rev_mode", [0, 1])
@pytest.mark.parametrize("case", list(CASES))
def test_delete_lockstep(case, rev_mode):
    say(f"[delete lockstep] {case} rev_mode={rev_mode}")
    w, o = base_state(case)
    g = gpu_index(w.cfg, rev_mode=rev_mode)
    for r, ops in w.rounds(2):
        for op in ops:
            if op.kind == "insert":
                assert o.insert(op.ids, op.vecs) == 0
            elif op.kind == "delete":
                pre = to_gpu(o, g, w)
                assert o.delete(op.ids) == 0
                g.delete(op.ids)
                gst, ost = g.export(), o.export()
                check_graph_invariants(gst, w.cfg.R)
                n = compare_states(gst, ost, w.cfg.algo, CASES[case][3], ctx=_ctx(case, w, pre, op.ids))
                say(f"  round {r}: {n} differing lists")


@pytest.mark.parametrize("case", ["u8_d128", "cagra_ip_r30", "u8_d128_r1"])
def test_in_edge_counts_agree_with_the_transpose(case):
    """grand_count_in_edges: the per-id linear scan, the batch-rows reverse
    build and the full reverse graph all count, for each given id, exactly
    the in-degree of the oracle's transpose."""
    from paper_2608_21163_amd import grand
    say(f"[in-edge counts] {case}")
    w, o = base_state(case)
    g = gpu_index(w.cfg)
    st = to_gpu(o, g, w)
    offs, _ = reverse_csr(st["adj"], st["active"])
    act = np.flatnonzero(st["active"])
    ids = np.random.default_rng(2).choice(act, 300, replace=False).astype(np.uint32)
    want = (offs[ids.astype(np.int64) + 1] - offs[ids]).astype(np.uint32)
    for method in (grand.INDEG_SCAN, grand.INDEG_REV_BATCH, grand.INDEG_REV_FULL):
        got, ms = g.count_in_edges(ids, method)
        assert np.array_equal(got, want), method
        say(f"  method {method}: {ms:.3f} ms")
    assert np.array_equal(g.export()["adj"], o.export()["adj"]) if w.cfg.algo == "cagra" else True
    inactive = np.flatnonzero(st["active"] == 0)[:1].astype(np.uint32)
    with pytest.raises(grand.GrandError):
        g.count_in_edges(inactive, grand.INDEG_SCAN)


def test_delete_medoid_installs_the_same_medoid():
    say("[medoid delete] u8_d128")
    w, o = base_state("u8_d128")
    g = gpu_index(w.cfg)
    st = to_gpu(o, g, w)
    med = np.array([st["medoid"]], np.uint32)
    assert o.delete(med) == 0
    g.delete(med)
    gst, ost = g.export(), o.export()
    assert gst["medoid"] == ost["medoid"] != st["medoid"]
    compare_states(gst, ost, "vamana", 0.0)


def test_free_running_tiny_workload():
    """The whole tiny workload on both sides independently: 10 bootstrap and
    insert batches, one round of inserts and deletes, 100 queries."""
    say("[free running] tiny")
    w = make_workload("tiny").keep_vectors()
    o = Oracle(w.cfg)
    g = gpu_index(w.cfg)
    for op in w.base_batches():
        assert o.insert(op.ids, op.vecs) == 0
        g.insert(op.ids, op.vecs)
    for r, ops in w.rounds():
        for op in ops:
            if op.kind == "insert":
                assert o.insert(op.ids, op.vecs) == 0
                g.insert(op.ids, op.vecs)
            elif op.kind == "delete":
                assert o.delete(op.ids) == 0
                g.delete(op.ids)
            else:
                gi, gd = g.search(op.vecs, 10, 64)
                oi, od = o.search(op.vecs, 10, 64)
                gt = brute_knn(w.vectors, w.active, op.vecs, 10)
                rg, ro = recall(gi, gt), recall(oi, gt)
                say(f"  recall@10 gpu {rg:.4f} oracle {ro:.4f}")
                assert abs(rg - ro) <= 0.005
                assert rg >= 0.9
    gst, ost = g.export(), o.export()
    check_graph_invariants(gst, w.cfg.R)
    assert np.array_equal(gst["active"], ost["active"])
    from helpers import canonical_rows
    same = np.all(canonical_rows(gst["adj"]) == canonical_rows(ost["adj"]), axis=1)
    frac = 1.0 - same[ost["active"] > 0].mean()
    say(f"  differing lists after the whole workload: {frac:.5f}")
    assert frac <= 0.001


def test_validation_errors_leave_the_gpu_state_untouched():
    say("[validation]")
    from paper_2608_21163_amd import grand
    w, o = base_state("tiny_f32_d32")
    g = gpu_index(w.cfg)
    to_gpu(o, g, w)
    st0 = g.export()
    act = np.flatnonzero(st0["active"]).astype(np.uint32)
    free = np.flatnonzero(st0["active"] == 0).astype(np.uint32)
    x = np.zeros((2, w.cfg.dim), np.float32)
    assert g.insert(np.array([free[0], free[0]], np.uint32), x, check=False) == grand.E_ID
    assert g.insert(act[:1], x[:1], check=False) == grand.E_ID
    assert g.insert(np.array([w.cfg.capacity], np.uint32), x[:1], check=False) == grand.E_ID
    bad = x[:1].copy()
    bad[0, 3] = np.inf
    assert g.insert(free[:1], bad, check=False) == grand.E_ARG
    assert g.delete(free[:1], check=False) == grand.E_ID
    assert g.delete(np.array([act[0], act[0]], np.uint32), check=False) == grand.E_ID
    assert g.search_rc(x[:1], 5, 4) == grand.E_ARG
    assert g.insert(np.zeros(0, np.uint32), x[:0], check=False) == 0
    st1 = g.export()
    for k in ("adj", "deg", "active"):
        assert np.array_equal(st0[k], st1[k])
    assert st0["medoid"] == st1["medoid"]


def test_capacity_overflow_is_rejected_before_any_change():
    """An insert batch larger than the free capacity returns
    GRAND_E_CAPACITY and leaves the index as it was; a batch that fills the
    pool exactly is accepted."""
    say("[capacity]")
    from paper_2608_21163_amd import grand
    w = make_workload("tiny", index=dict(capacity=1_200), stream=dict(base_n=1_000, build_batch=1_000)).keep_vectors()
    g = gpu_index(w.cfg)
    op = next(w.base_batches())
    g.insert(op.ids, op.vecs)
    st0 = g.export()
    free = np.flatnonzero(st0["active"] == 0).astype(np.uint32)
    x = np.random.default_rng(3).standard_normal((free.size + 1, w.cfg.dim)).astype(np.float32)
    ids = np.concatenate([free, np.array([0], np.uint32)])
    assert g.insert(ids, x, check=False) == grand.E_CAPACITY
    st1 = g.export()
    for k in ("adj", "deg", "active"):
        assert np.array_equal(st0[k], st1[k])
    g.insert(free, x[: free.size])
    st2 = g.export()
    assert st2["active"].all()
    check_graph_invariants(st2, w.cfg.R)


def test_empty_index_search_and_delete_everything():
    say("[empty index]")
    w = make_workload("tiny", index=dict(capacity=300), stream=dict(base_n=200, build_batch=200)).keep_vectors()
    g = gpu_index(w.cfg)
    q = np.zeros((3, w.cfg.dim), np.float32)
    ids, d = g.search(q, 5, 8)
    assert (ids == INVALID).all() and np.isinf(d).all()
    op = next(w.base_batches())
    g.insert(op.ids, op.vecs)
    g.delete(op.ids[::-1].copy())
    st = g.export()
    check_graph_invariants(st, w.cfg.R)
    assert not st["active"].any() and st["medoid"] == INVALID
    ids, d = g.search(q, 5, 8)
    assert (ids == INVALID).all()


def test_cagra_racing_mode_keeps_invariants():
    """The racing (paper-literal, last writer wins) compare-and-swap mode is
    order dependent; it is checked by invariants only: valid lists, and every
    replaced entry was reachable through the new node (detour)."""
    say("[cagra racing]")
    w, o = base_state("cagra_ip_d100")
    cfg = w.cfg.replace(cas_mode="racing")
    g = gpu_index(cfg)
    to_gpu(o, g, w)
    for op in next(w.rounds(1))[1]:
        if op.kind == "delete":
            g.delete(op.ids)           # this stream deletes first, then inserts
        elif op.kind == "insert":
            break
    st0 = g.export()
    g.insert(op.ids, op.vecs)
    st1 = g.export()
    check_graph_invariants(st1, cfg.R)
    new = set(op.ids.tolist())
    changed = (st0["adj"] != st1["adj"]) & (st0["adj"] != INVALID)
    assert changed.any()
    for u, s in zip(*np.nonzero(changed)):
        if u in new:
            continue
        p, r_old = int(st1["adj"][u, s]), int(st0["adj"][u, s])
        assert p in new and r_old in set(st1["adj"][p].tolist())

def test_reverse_graph_large_random_graph_is_exact_transpose():
    """The reverse CSR of an imported 300,000-node random graph (64 distinct
    out-neighbours per row, a few inactive rows) against the transpose
    computed with numpy."""
    from paper_2608_21163_amd import GrandIndex
    from workloads.generators import IndexConfig
    say("[reverse large]")
    cap, R, dim = 300_000, 64, 64
    rng = np.random.default_rng(11)
    active = np.ones(cap, np.uint8)
    active[rng.choice(cap, 3_000, replace=False)] = 0
    act_ids = np.flatnonzero(active)
    adj = np.full((cap, R), INVALID, np.uint32)
    deg = np.zeros(cap, np.uint32)
    # rows: distinct random active targets other than u, random degree 0..R
    d = rng.integers(0, R + 1, size=cap)
    d[active == 0] = 0
    cand = act_ids[rng.integers(0, act_ids.size, size=(cap, R + 8))]
    for u in np.flatnonzero(d):
        row = cand[u][cand[u] != u]
        row = np.unique(row)[: d[u]]
        rng.shuffle(row)
        adj[u, : row.size] = row
        deg[u] = row.size
    vecs = rng.integers(0, 256, size=(cap, dim), dtype=np.uint8)
    cfg = IndexConfig("vamana", "u8", "l2", dim, cap, R, 64)
    g = GrandIndex.from_config(cfg, max_batch=1_000)
    g.import_graph(vecs, adj, deg, active, int(act_ids[0]))
    e = g.export(with_reverse=True)
    src = np.repeat(np.arange(cap, dtype=np.int64), R)
    tgt = adj.reshape(-1).astype(np.int64)
    keep = tgt != INVALID
    src, tgt = src[keep], tgt[keep]
    order = np.lexsort((src, tgt))
    want_off = np.zeros(cap + 1, np.int64)
    np.add.at(want_off, tgt + 1, 1)
    want_off = np.cumsum(want_off)
    assert np.array_equal(e["rev_offsets"].astype(np.int64), want_off)
    assert np.array_equal(e["rev_srcs"].astype(np.int64), src[order])


def test_large_capacity_forms_match_the_small_index():
    """A capacity just above 2^24 ids takes the one-level forms of the
    record grouping (global atomics) and of the search's visited hash
    (16-bit tags); a 12,000-slot index takes the two-level grouping and the
    8-bit hash.  Both receive the same batches, with ids below 12,000 only,
    so the graphs, the reverse graphs and the query results must be
    identical (uint8 distances are exact on both)."""
    import dataclasses

    from helpers import canonical_rows
    from paper_2608_21163_amd import GrandIndex
    say("[large capacity forms] u8_d128")
    w = _workload("u8_d128")
    small = w.cfg
    big = dataclasses.replace(small, capacity=(1 << 24) + 1)
    gs = GrandIndex.from_config(small, max_batch=2_000)
    gb = GrandIndex.from_config(big, max_batch=2_000)
    for op in w.base_batches():
        gs.insert(op.ids, op.vecs)
        gb.insert(op.ids, op.vecs)
    n = small.capacity

    def same(tag):
        a, b = gs.export(with_reverse=True), gb.export(with_reverse=True)
        assert np.array_equal(a["active"], b["active"][:n]) and not b["active"][n:].any(), tag
        assert a["medoid"] == b["medoid"], tag
        assert np.array_equal(a["deg"], b["deg"][:n]), tag
        assert np.array_equal(canonical_rows(a["adj"]), canonical_rows(b["adj"][:n])), tag
        assert np.array_equal(a["rev_offsets"], b["rev_offsets"][: n + 1]), tag
        assert (b["rev_offsets"][n:] == a["rev_offsets"][n]).all(), tag
        assert np.array_equal(a["rev_srcs"], b["rev_srcs"]), tag

    same("base")
    for r, ops in w.rounds(1):
        for op in ops:
            if op.kind == "insert":
                gs.insert(op.ids, op.vecs)
                gb.insert(op.ids, op.vecs)
                same(f"round {r} insert")
            elif op.kind == "delete":
                gs.delete(op.ids)
                gb.delete(op.ids)
                same(f"round {r} delete")
            else:
                si, sd = gs.search(op.vecs, 10, 64)
                bi, bd = gb.search(op.vecs, 10, 64)
                assert np.array_equal(si, bi) and np.array_equal(sd, bd)
    gs.close()
    gb.close()
