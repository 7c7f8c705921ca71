"""Failure paths of the C ABI, forced from the host so every kernel still
ends normally: a device-wide scan whose look-back wait gives up (reported by
the next synchronisation point), the Eq. 12 capacity bound (checked on the
host before any work), allocation failure (a test hook makes the library's
allocations fail), and that a failed call leaves its output handle and the
previous results unchanged; an LRU update whose partition scan gave up is
skipped whole.  Also FIFO and LRU caches with repeated ids in one request
list, against the oracle's one-at-a-time admission.
"""
import ctypes as C

import numpy as np
import pytest

import oracle as O
import workloads as W
from test_gpu_parity import G, dev, graph_case, host, say  # noqa: F401  (G is a fixture)

pytestmark = pytest.mark.gpu

E_INVALID, E_NOMEM, E_CAPACITY, E_DEVICE = 1, 3, 4, 5
DEFAULT_SPIN_LIMIT = 1 << 20


@pytest.fixture
def hooks(G):
    yield G
    G.debug_set_spin_limit(DEFAULT_SPIN_LIMIT)
    G.debug_fail_allocations(-1)


def _status(fn):
    try:
        fn()
    except Exception as e:  # GnnavError
        return getattr(e, "status", None)
    return 0


def test_gather_scan_timeout_reported_by_sync(hooks):
    """Spin limit 0: every classification tile after the first gives up at
    once; gnnav_sync reports it (once), and with the limit restored the same
    gather is exact again."""
    import torch
    G = hooks
    n, u, v = graph_case("random-20000-100000-3")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, 40, "f32", seed=5)
    c = G.Cache(g, feats, "f32", 0.3)
    ids = np.random.default_rng(0).integers(0, n, 9000).astype(np.int32)   # five scan tiles
    ids_d = dev(ids)
    out = torch.zeros((ids.size, c.ld), device="cuda")
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    G.sync()
    say("errors", "gather with spin limit 0")
    G.debug_set_spin_limit(0)
    G.gather(c, ids_d.data_ptr(), ids.size, out, counts)       # enqueues fine
    assert _status(G.sync) == E_DEVICE
    assert "gave up" in G._lib.gnnav_last_error().decode()
    assert _status(G.sync) == 0                                  # reported once
    G.debug_set_spin_limit(DEFAULT_SPIN_LIMIT)
    G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
    G.sync()
    _, slot, _ = O.rank_cache(csr, 0.3)
    ref_rows, ref_counts = O.gather(feats, slot, ids)
    assert np.array_equal(host(counts), ref_counts)
    assert np.array_equal(host(out)[:, :40], ref_rows)


def test_sample_scan_timeout_reported_by_blocks_sync(hooks):
    """The sampler's scans under spin limit 0: gnnav_blocks_sync (after the
    asynchronous sample) and gnnav_sample itself return E_DEVICE; with the
    limit restored the blocks equal the oracle's."""
    G = hooks
    n, u, v = graph_case("random-20000-100000-4")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    seeds = np.random.default_rng(1).permutation(n)[:6000].astype(np.int32)   # three dedup tiles
    seeds_d = dev(seeds)
    fan = [5, 5]
    blk = G.Blocks()
    G.sync()
    say("errors", "sample with spin limit 0")
    G.debug_set_spin_limit(0)
    G.sample_async(g, seeds_d, fan, 77, blk)
    assert _status(lambda: blk.sync()) == E_DEVICE
    assert _status(lambda: G.sample(g, seeds_d, fan, 78, blk)) == E_DEVICE
    G.debug_set_spin_limit(DEFAULT_SPIN_LIMIT)
    G.sample(g, seeds_d, fan, 77, blk)
    nodes, sizes, ip, nb, ix = blk.to_host()
    ref = O.sample_blocks(csr, seeds, fan, 77)
    assert sizes == ref.sizes and np.array_equal(nodes, ref.nodes)
    for h in range(2):
        assert np.array_equal(ip[h], ref.indptr[h]) and np.array_equal(ix[h], ref.indices[h])


def test_lru_partition_timeout_skips_the_update(hooks):
    """An LRU ring of 5,000 slots (three partition tiles) under spin limit 0,
    gathering 1,500 ids (one classification tile, so the gather itself is
    exact): the partition's waits give up, the update is skipped as a whole
    -- slot map, slot owners and cached rows stay as they were -- and
    gnnav_sync reports E_DEVICE.  With the limit restored the cache goes on
    exactly as the oracle's LRU without that batch."""
    import torch
    from test_gpu_cache_update import check_cache
    G = hooks
    n, u, v = graph_case("random-20000-100000-5")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, 24, "f32", seed=6)
    c = G.Cache(g, feats, "f32", 0.3)
    ring = 5000
    c.set_policy("lru", ring)
    ref = O.LruCache(csr, 0.3, ring)
    rng = np.random.default_rng(2)
    hot = rng.permutation(n)[:3000].astype(np.int32)
    out = torch.zeros((1500, c.ld), device="cuda")
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")

    def gather(ids):
        ids_d = dev(ids)
        G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
        return ids_d

    for b in range(2):
        ids = rng.choice(hot, 1500, replace=False).astype(np.int32)
        ids_d = gather(ids)
        G.sync()
        ref_rows, ref_counts = ref.gather(feats, ids)
        assert np.array_equal(host(counts), ref_counts) and np.array_equal(host(out)[:, :24], ref_rows)
        check_cache(c, ref, feats)
    ids = rng.choice(hot, 1500, replace=False).astype(np.int32)
    say("errors", "LRU gather with spin limit 0")
    G.debug_set_spin_limit(0)
    ids_d = gather(ids)
    assert _status(G.sync) == E_DEVICE
    G.debug_set_spin_limit(DEFAULT_SPIN_LIMIT)
    ref_rows, ref_counts = O.gather(feats, ref.slot_map, ids)
    assert np.array_equal(host(counts), ref_counts) and np.array_equal(host(out)[:, :24], ref_rows)
    check_cache(c, ref, feats)          # unchanged: the update was skipped
    for b in range(2):
        ids = rng.choice(hot, 1500, replace=False).astype(np.int32)
        ids_d = gather(ids)
        G.sync()
        ref.gather(feats, ids)
        check_cache(c, ref, feats)
    del ids_d


@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_set_policy_allocation_failure_leaves_cache_static(hooks, policy):
    """Each device allocation of gnnav_cache_set_policy made to fail in
    turn: the call returns E_NOMEM and the cache stays static (a gather
    after it leaves the slot map as the degree ranking made it); the first
    attempt that succeeds gives a cache that follows the oracle's policy."""
    import torch
    from test_gpu_cache_update import POLICY, check_cache
    G = hooks
    n, u, v = graph_case("random-8000-60000-6")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, 16, "f32", seed=8)
    c = G.Cache(g, feats, "f32", 0.3)
    ring = c.n_cached // 2
    _, slot, _ = O.rank_cache(csr, 0.3)
    rng = np.random.default_rng(5)
    out = torch.zeros((3000, c.ld), device="cuda")
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    code = {"fifo": 1, "lru": 2}[policy]
    done = False
    for k in range(12):
        say("errors", policy, "set_policy allocation failure after", k)
        G.debug_fail_allocations(k)
        st = G._lib.gnnav_cache_set_policy(c._h, code, ring)
        G.debug_fail_allocations(-1)
        if st == 0:
            done = True
            break
        assert st == E_NOMEM, (k, st)
        ids = rng.integers(0, n, 3000).astype(np.int32)
        ids_d = dev(ids)
        G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
        G.sync()
        ref_rows, ref_counts = O.gather(feats, slot, ids)
        assert np.array_equal(host(counts), ref_counts)
        assert np.array_equal(host(out)[:, :16], ref_rows)
        assert np.array_equal(c.slot_map(), slot), "a failed set_policy must leave the cache static"
    assert done and k >= 1
    ref = POLICY[policy](csr, 0.3, ring)
    for b in range(3):
        ids = rng.integers(0, n, 3000).astype(np.int32)
        ids_d = dev(ids)
        G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
        G.sync()
        ref.gather(feats, ids)
        check_cache(c, ref, feats)


def test_failed_node_table_growth_leaves_blocks_usable(hooks):
    """Blocks reused across graphs: growing the node table for a larger
    graph fails (E_NOMEM; the old table is gone, and the blocks read as
    unsampled), and a later sample of a graph the old table would have
    fitted builds a new table and equals the oracle's."""
    G = hooks
    graphs = {}
    for n in (5000, 30000, 60000):
        n_, u, v = graph_case(f"random-{n}-{4 * n}-7")
        graphs[n] = (O.build_csr(n_, u, v), G.Graph(n_, u, v))
    blk = G.Blocks()
    fan = [5, 5]
    for n in (5000, 30000):
        seeds = np.random.default_rng(n).permutation(n)[:400].astype(np.int32)
        G.sample(graphs[n][1], dev(seeds), fan, 3, blk)
    seeds = np.random.default_rng(1).permutation(60000)[:400].astype(np.int32)
    say("errors", "node table growth fails")
    assert blk.hop(1).n_dst > 0
    G.debug_fail_allocations(0)
    assert _status(lambda: G.sample(graphs[60000][1], dev(seeds), fan, 3, blk)) == E_NOMEM
    G.debug_fail_allocations(-1)
    # the failed growth freed the previous sample's node table: the blocks
    # read as unsampled rather than describing buffers that may be gone
    assert _status(lambda: blk.hop(1)) == E_INVALID
    for n in (30000, 5000):
        seeds = np.random.default_rng(n + 1).permutation(n)[:400].astype(np.int32)
        G.sample(graphs[n][1], dev(seeds), fan, 4, blk)
        nodes, sizes, ip, nb, ix = blk.to_host()
        ref = O.sample_blocks(graphs[n][0], seeds, fan, 4)
        assert sizes == ref.sizes and np.array_equal(nodes, ref.nodes)
        for h in range(2):
            assert np.array_equal(ix[h], ref.indices[h])
    blk.close()


def test_capacity_bound_checked_before_any_work(hooks):
    """A star with 50,000 leaves sampled with fanout -1 (every neighbour) from
    all of its vertices: the Eq. 12 bound 50,001 x 50,000 exceeds INT32_MAX,
    so gnnav_sample fails with E_CAPACITY before enqueuing anything and the
    blocks still hold the previous sample."""
    import torch
    G = hooks
    n = 50_001
    u = np.zeros(n - 1, np.int32)
    v = np.arange(1, n, dtype=np.int32)
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    assert g.max_degree == n - 1
    blk = G.Blocks()
    small = dev(np.array([3, 0, 9], np.int32))
    G.sample(g, small, [4, 2], 5, blk)
    before = blk.to_host()
    everyone = dev(np.arange(n, dtype=np.int32))
    for fan in ([-1], [3, -1]):
        say("errors", "capacity", fan)
        for fn in (G.sample, G.sample_async):
            with pytest.raises(G.GnnavError) as e:
                fn(g, everyone, fan, 5, blk)
            assert e.value.status == E_CAPACITY
    torch.cuda.synchronize()
    after = blk.to_host()
    assert before[1] == after[1]
    for a, b in zip([before[0]] + before[2] + before[3] + before[4], [after[0]] + after[2] + after[3] + after[4]):
        assert np.array_equal(a, b)
    ref = O.sample_blocks(csr, np.array([3, 0, 9], np.int32), [4, 2], 5)
    assert after[1] == ref.sizes and np.array_equal(after[0], ref.nodes)


def test_allocation_failure_leaves_handles_unwritten(hooks):
    """With the allocation hook armed, every set-up call fails with E_NOMEM
    after 0, 1, 2, ... successful allocations and leaves *out as it was; the
    library then works normally once the hook is off."""
    import torch
    G = hooks
    lib = G._lib
    n, u, v = graph_case("random-3000-20000-6")
    csr = O.build_csr(n, u, v)
    feats = W.features(n, 24, "f32", seed=6)
    sentinel = 0x5EED
    for k in range(4):
        say("errors", "alloc failure after", k)
        h = C.c_void_p(sentinel)
        G.debug_fail_allocations(k)
        st = lib.gnnav_build_csr(n, u.size, u.ctypes.data, v.ctypes.data, 1, C.byref(h))
        G.debug_fail_allocations(-1)
        if st == 0:
            lib.gnnav_graph_free(h)
            assert k >= 2          # row offsets and columns: two allocations
            continue
        assert st == E_NOMEM and h.value == sentinel
    g = G.Graph(n, u, v)
    made = False
    for k in range(8):
        h = C.c_void_p(sentinel)
        G.debug_fail_allocations(k)
        st = lib.gnnav_build_cache(g._h, feats.ctypes.data, 24, 0, 0.4, 0, C.byref(h))
        G.debug_fail_allocations(-1)
        if st == 0:
            lib.gnnav_cache_free(h)
            made = True
            break
        assert st == E_NOMEM and h.value == sentinel, (k, st)
    assert made
    h = C.c_void_p(sentinel)
    G.debug_fail_allocations(0)
    st = lib.gnnav_blocks_create(C.byref(h))
    G.debug_fail_allocations(-1)
    assert st == E_NOMEM and h.value == sentinel
    # a sample whose workspace cannot grow fails; the blocks stay usable
    blk = G.Blocks()
    seeds = np.random.default_rng(2).permutation(n)[:300].astype(np.int32)
    seeds_d = dev(seeds)
    G.debug_fail_allocations(1)
    with pytest.raises(G.GnnavError) as e:
        G.sample(g, seeds_d, [5, 5], 9, blk)
    assert e.value.status == E_NOMEM
    G.debug_fail_allocations(-1)
    assert _status(lambda: blk.hop(1)) == E_INVALID   # nothing sampled
    torch.cuda.synchronize()
    G.sample(g, seeds_d, [5, 5], 9, blk)
    nodes, sizes, _, _, ix = blk.to_host()
    ref = O.sample_blocks(csr, seeds, [5, 5], 9)
    assert sizes == ref.sizes and np.array_equal(nodes, ref.nodes)
    assert all(np.array_equal(a, b) for a, b in zip(ix, ref.indices))
    # a gather whose workspace cannot be allocated fails before enqueuing
    c = G.Cache(g, feats, "f32", 0.4)
    out = torch.zeros((seeds.size, c.ld), device="cuda")
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    G.debug_fail_allocations(0)
    with pytest.raises(G.GnnavError) as e:
        G.gather(c, seeds_d.data_ptr(), seeds.size, out, counts, None)
    assert e.value.status == E_NOMEM
    G.debug_fail_allocations(-1)
    G.gather(c, seeds_d.data_ptr(), seeds.size, out, counts, None)
    G.sync()
    _, slot, _ = O.rank_cache(csr, 0.4)
    rows, cnt = O.gather(feats, slot, seeds)
    assert np.array_equal(host(counts), cnt) and np.array_equal(host(out)[:, :24], rows)


@pytest.mark.parametrize("d,dtype,r,ring", [(32, "f32", 0.3, None), (64, "f32", 0.2, 50), (128, "bf16", 0.25, 7)])
@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_dynamic_repeated_ids_match_oracle(G, policy, d, dtype, r, ring):
    """Request lists with repeated ids through a FIFO or LRU cache: counts,
    rows, slot map, owners and cached rows after every gather equal the
    oracle's one-at-a-time admission."""
    import torch
    from test_gpu_cache_update import POLICY, check_cache
    n, u, v = graph_case("random-4000-30000-9")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, d, dtype, seed=d)
    c = G.Cache(g, feats, dtype, r)
    ring = c.n_cached if ring is None else ring
    c.set_policy(policy, ring)
    ref = POLICY[policy](csr, r, ring)
    rng = np.random.default_rng(d + 1)
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    for b in range(6):
        m = [700, 1, 40, 2500, 300, 64][b]
        ids = rng.integers(0, n, m).astype(np.int32)
        k = max(1, m // 4)
        ids[rng.integers(0, m, k)] = ids[rng.integers(0, m, k)]       # repeats
        say(policy, "repeats", d, dtype, r, ring, b, m)
        out = torch.zeros((m, c.ld), dtype=torch.int16 if dtype == "bf16" else torch.float32, device="cuda")
        ids_d = dev(ids)
        G.gather(c, ids_d.data_ptr(), m, out, counts)
        ref_rows, ref_counts = ref.gather(feats, ids)
        assert np.array_equal(host(counts), ref_counts)
        assert np.array_equal(host(out, dtype)[:, :d].view(np.uint8), ref_rows.view(np.uint8))
        check_cache(c, ref, feats)
