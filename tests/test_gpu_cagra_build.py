"""GPU parity of the CAGRA graph construction (grand_build_cagra; Section 2.2
on CAGRA, Section 4.2 CAGRA graph construction) against the oracle on the
same points and the same random initial lists.  Both sides evaluate every
distance the same way (exact integers; fp64 sums in dimension order rounded
once), so the built graphs must be identical slot for slot."""
import numpy as np
import pytest

from helpers import INVALID
from oracle.oracle import Oracle
from parity import say
from workloads import IndexConfig
from workloads.generators import cagra_init_lists

pytestmark = pytest.mark.gpu

# (dtype, metric, dim, n, knn, R, sample, iters)
CASES = {
    "f32_ip_d100": ("f32", "ip", 100, 3000, 32, 16, 8, 4),
    "f32_l2_d24": ("f32", "l2", 24, 2500, 40, 20, 10, 3),
    "u8_l2_d128": ("u8", "l2", 128, 3000, 32, 16, 8, 4),
    "u8_l2_d64_r30": ("u8", "l2", 64, 2000, 48, 30, 12, 2),
    # large samples: a round's proposals (tens of millions) exceed the record
    # buffers (n * 2 * sample), so the joins are written and merged in chunks
    "f32_l2_d16_chunked": ("f32", "l2", 16, 8000, 64, 32, 32, 2),
}


def _points(dtype, metric, dim, n, seed):
    g = np.random.default_rng(seed)
    if dtype == "u8":
        c = g.integers(0, 256, size=(16, dim))
        x = np.clip(c[g.integers(0, 16, n)] + g.normal(0, 20, (n, dim)), 0, 255)
        return np.rint(x).astype(np.uint8)
    x = (g.standard_normal((16, dim))[g.integers(0, 16, n)] + 0.4 * g.standard_normal((n, dim))).astype(np.float32)
    if metric == "ip":
        x /= np.linalg.norm(x, axis=1, keepdims=True)
    return x


@pytest.mark.parametrize("case", list(CASES))
def test_construction_matches_the_oracle(case):
    from paper_2608_21163_amd import GrandIndex
    dtype, metric, dim, n, K, R, S, iters = CASES[case]
    cap = n + 500
    cfg = IndexConfig(algo="cagra", dtype=dtype, metric=metric, dim=dim, capacity=cap, R=R, L_build=64)
    x = _points(dtype, metric, dim, n, 3)
    ids = np.random.default_rng(4).permutation(cap)[:n].astype(np.uint32)  # scattered ids
    init = cagra_init_lists(n, K, 5)
    say(f"[{case}] n {n} knn {K} R {R} sample {S} rounds {iters}")
    o = Oracle(cfg)
    assert o.build_cagra(ids, x, init, K, iters, S) == 0, o.last_error()
    ost = o.export()
    say(f"[{case}] oracle built")
    g = GrandIndex.from_config(cfg, max_batch=1_000)
    g.build_cagra(ids, x, init, K, iters, S)
    gst = g.export()
    say(f"[{case}] GPU built")
    assert (gst["active"] == ost["active"]).all()
    assert (gst["deg"] == ost["deg"]).all()
    diff = np.flatnonzero((gst["adj"][ids] != ost["adj"][ids]).any(1))
    say(f"[{case}] differing lists: {diff.size} of {n}")
    assert diff.size == 0, (diff[:5], gst["adj"][ids[diff[:1]]], ost["adj"][ids[diff[:1]]])
    assert gst["medoid"] == ost["medoid"]
    # a built index serves searches and updates like a grown one
    q = _points(dtype, metric, dim, 50, 9)
    gi, _ = g.search(q, 10, 64)
    oi, _ = o.search(q, 10, 64)
    same = (np.asarray(gi) == np.asarray(oi)).all(1).mean()
    assert same == 1.0 if dtype == "u8" else same >= 0.96
    # ... and updates: one insert and one delete batch on both sides
    free = np.setdiff1d(np.arange(cap, dtype=np.uint32), ids)[:200]
    xn = _points(dtype, metric, dim, free.size, 11)
    dele = np.random.default_rng(12).choice(ids, 300, replace=False).astype(np.uint32)
    for side in (o, g):
        assert side.insert(free, xn) in (0, None)
        assert side.delete(dele) in (0, None)
    gst, ost = g.export(), o.export()
    assert (gst["active"] == ost["active"]).all()
    live = np.flatnonzero(ost["active"])
    diff = np.flatnonzero((gst["adj"][live] != ost["adj"][live]).any(1) | (gst["deg"][live] != ost["deg"][live]))
    say(f"[{case}] after an insert and a delete batch: {diff.size} differing lists")
    assert diff.size <= (0 if dtype == "u8" else 0.001 * live.size)
    g.close()


def test_construction_rejects_bad_input_and_changes_nothing():
    from paper_2608_21163_amd import GrandIndex
    from paper_2608_21163_amd.grand import GrandError
    n, K, R = 600, 16, 8
    cfg = IndexConfig(algo="cagra", dtype="f32", metric="l2", dim=8, capacity=1000, R=R, L_build=32)
    x = _points("f32", "l2", 8, n, 1)
    ids = np.arange(n, dtype=np.uint32)
    good = cagra_init_lists(n, K, 1)
    g = GrandIndex.from_config(cfg, max_batch=1_000)
    for bad_row, bad_val in ((3, 3), (5, None), (7, n)):
        bad = good.copy()
        bad[bad_row, 1] = bad[bad_row, 0] if bad_val is None else bad_val
        with pytest.raises(GrandError):
            g.build_cagra(ids, x, bad, K, 2, 4)
        assert g.export()["active"].sum() == 0
    with pytest.raises(GrandError):
        g.build_cagra(ids, x, cagra_init_lists(n, R - 1, 1), R - 1, 2, 4)   # knn < R
    vcfg = IndexConfig(algo="vamana", dtype="f32", metric="l2", dim=8, capacity=1000, R=R, L_build=32)
    gv = GrandIndex.from_config(vcfg, max_batch=1_000)
    with pytest.raises(GrandError):
        gv.build_cagra(ids, x, good, K, 2, 4)   # the Vamana variant
    g.build_cagra(ids, x, good, K, 2, 4)
    st = g.export()
    assert st["active"].sum() == n and (st["deg"][ids] == R).all()
    with pytest.raises(GrandError):
        g.build_cagra(ids, x, good, K, 2, 4)    # not empty any more
    g.close()
    gv.close()
