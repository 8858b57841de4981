"""grand_search_static (the search entry point that allocates nothing)
against grand_search, through the C ABI: identical ids and distances on two
calls in a row, the second with fewer queries (the fixed device array keeps
the first call's contents), for uint8 rows and for fp32 rows with padding;
a request larger than the array is refused with GRAND_E_CAPACITY."""
import numpy as np
import pytest

from parity import say
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _index(name, index, stream):
    from paper_2608_21163_amd import GrandIndex
    w = make_workload(name, seed=5, index=index, stream=stream).keep_vectors()
    g = GrandIndex.from_config(w.cfg, max_batch=2_000)
    for op in w.base_batches():
        g.insert(op.ids, op.vecs)
    return w, g


def _queries(w, n, seed):
    return w.sampler.draw(np.random.default_rng(seed), n)[0]


@pytest.mark.parametrize("name,index", [
    ("sift1m_u8", dict(capacity=5_000, R=32, L_build=64)),
    ("deep1m_window", dict(capacity=5_000, R=32, L_build=64, dim=30)),   # 120-byte rows padded to 128
])
def test_static_search_matches_search_twice(name, index):
    say(f"[no-alloc search] {name}")
    w, g = _index(name, index, dict(base_n=4_000, build_batch=2_000))
    for call, (nq, k, beam) in enumerate([(700, 10, 64), (230, 8, 32)]):
        q = _queries(w, nq, 100 + call)
        ref_i, ref_d = g.search(q, k, beam)
        got_i, got_d = g.search_static(q, k, beam)
        assert np.array_equal(got_i, ref_i), call
        assert np.array_equal(got_d.view(np.uint32), ref_d.view(np.uint32)), call
        say(f"  call {call}: {nq} queries identical")
    g.close()


def test_static_search_with_device_buffers_and_limit():
    import torch

    from paper_2608_21163_amd import grand
    say("[no-alloc search] device buffers, size limit")
    w, g = _index("sift1m_u8", dict(capacity=5_000, R=32, L_build=64), dict(base_n=4_000, build_batch=2_000))
    q = _queries(w, 500, 7)
    ref_i, ref_d = g.search(q, 10, 64)
    dq = torch.from_numpy(q).cuda()
    oi = torch.empty((500, 10), dtype=torch.int32, device="cuda")
    od = torch.empty((500, 10), dtype=torch.float32, device="cuda")
    g.set_stream(torch.cuda.current_stream().cuda_stream)
    g.search_static(dq, 10, 64, out_ids=oi, out_dists=od)
    assert np.array_equal(oi.cpu().numpy().view(np.uint32), ref_i)
    assert np.array_equal(od.cpu().numpy(), ref_d)
    big = np.zeros(((grand.STATIC_SCRATCH_BYTES // 128) + 1, 128), np.uint8)
    assert g.search_static(big, 10, 64, check=False) == grand.E_CAPACITY
    again_i, _ = g.search_static(q, 10, 64)
    assert np.array_equal(again_i, ref_i)
    g.close()
