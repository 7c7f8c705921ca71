"""gnnav_gather_noalloc: the gather for callers that cannot allocate device
memory, with its workspace in a static device array.  Checked against
gnnav_gather on the same requests -- rows bit-exact, counts equal -- on two
calls in a row, the second with fewer ids (the array keeps the first call's
contents), with the library's allocation hook armed so that any allocation
on the path would fail the call; a FIFO and an LRU cache are checked against a twin
cache updated by gnnav_gather; sizes above the maximum are refused.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W
from test_gpu_parity import G, dev, graph_case, host, say  # noqa: F401  (G is a fixture)

pytestmark = pytest.mark.gpu

MAX_IDS = 1 << 20


def noalloc(G, cache, ids_d, n, out, counts):
    """Status of one gnnav_gather_noalloc call through the C ABI."""
    f = G._lib.gnnav_gather_noalloc
    G.debug_fail_allocations(0)        # any allocation on this path would now fail
    try:
        st = f(cache._h, ids_d.data_ptr() if ids_d is not None else None, n, out.data_ptr(), out.stride(0),
               counts.data_ptr(), G._stream(None))
    finally:
        G.debug_fail_allocations(-1)
    return st


@pytest.mark.parametrize("d,dtype,r,on_device", [(100, "f32", 0.3, False), (128, "bf16", 0.25, True),
                                                 (602, "f32", 0.5, False)])
def test_noalloc_matches_gather(G, d, dtype, r, on_device):
    import torch
    n, u, v = graph_case("random-200000-800000-11")
    g = G.Graph(n, u, v)
    feats = W.features(n, d, dtype, seed=d + 1)
    c = G.Cache(g, feats, dtype, r, store_on_device=on_device)
    tdt = torch.int16 if dtype == "bf16" else torch.float32
    rng = np.random.default_rng(d)
    for m in (MAX_IDS if d < 600 else 300_000, 5_003, 0):
        say("noalloc", d, dtype, r, on_device, m)
        ids = rng.integers(0, n, max(m, 1)).astype(np.int32)[:m]
        if m > 10:
            ids[::997] = -1              # invalid ids: zero rows, counted apart
            ids[5::1009] = n + 3
        ids_d = dev(ids) if m else None
        a = torch.full((max(m, 1), c.ld), 7, dtype=tdt, device="cuda")
        b = torch.full((max(m, 1), c.ld), 9, dtype=tdt, device="cuda")
        ca = torch.full((3,), -1, dtype=torch.int64, device="cuda")
        cb = torch.full((3,), -2, dtype=torch.int64, device="cuda")
        assert noalloc(G, c, ids_d, m, a, ca) == 0, G._lib.gnnav_last_error()
        G.gather(c, ids_d.data_ptr() if m else 0, m, b, cb)
        G.sync()
        assert np.array_equal(host(ca), host(cb))
        assert np.array_equal(host(a, dtype)[:m].view(np.uint8), host(b, dtype)[:m].view(np.uint8))
        if m:
            _, slot, _ = O.rank_cache(O.build_csr(n, u, v), r) if m == 5_003 else (None, None, None)
            if slot is not None:
                ref_rows, ref_counts = O.gather(feats, slot, ids)
                assert np.array_equal(host(ca), ref_counts)
                assert np.array_equal(host(a, dtype)[:, :d].view(np.uint8), ref_rows.view(np.uint8))
    c.close()


@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_noalloc_dynamic_matches_gather_on_a_twin_cache(G, policy):
    import torch
    from test_gpu_cache_update import POLICY, check_cache
    n, u, v = graph_case("random-6000-40000-12")
    g = G.Graph(n, u, v)
    feats = W.features(n, 48, "f32", seed=12)
    ca_, cb_ = (G.Cache(g, feats, "f32", 0.3) for _ in range(2))
    for c in (ca_, cb_):
        c.set_policy(policy, 400)
    ref = POLICY[policy](O.build_csr(n, u, v), 0.3, 400)
    rng = np.random.default_rng(4)
    for m in (3000, 700):
        ids = rng.integers(0, n, m).astype(np.int32)
        ids_d = dev(ids)
        a = torch.zeros((m, ca_.ld), device="cuda")
        b = torch.zeros((m, cb_.ld), device="cuda")
        ka = torch.zeros(3, dtype=torch.int64, device="cuda")
        kb = torch.zeros(3, dtype=torch.int64, device="cuda")
        assert noalloc(G, ca_, ids_d, m, a, ka) == 0, G._lib.gnnav_last_error()
        G.gather(cb_, ids_d.data_ptr(), m, b, kb)
        G.sync()
        ref.gather(feats, ids)
        assert np.array_equal(host(ka), host(kb))
        assert np.array_equal(host(a), host(b))
        check_cache(ca_, ref, feats)
        check_cache(cb_, ref, feats)


def test_noalloc_refuses_more_than_its_maximum(G):
    import torch
    n, u, v = graph_case("random-3000-9000-13")
    g = G.Graph(n, u, v)
    c = G.Cache(g, W.features(n, 8, "f32", seed=1), "f32", 0.5)
    out = torch.zeros((1, c.ld), device="cuda")
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    ids = dev(np.zeros(1, np.int32))
    assert noalloc(G, c, ids, MAX_IDS + 1, out, counts) == 4          # E_CAPACITY, before any work
    assert b"at most" in G._lib.gnnav_last_error()
    assert noalloc(G, c, ids, -1, out, counts) == 1                   # E_INVALID
    G.sync()
