"""GPU parity of the dynamic (FIFO and LRU) cache updates against the oracle.

After every gather the cache must hold exactly what the oracle's sequential
policy holds: the slot map, the vertex in every slot, and that vertex's row;
the hit/miss counts and the gathered rows must match batch by batch.  The
frontiers gathered here are duplicate-free, as the sampler's are.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W
from parity_util import BF16_TOL, FP32_TOL, assert_rows_close
from test_gpu_parity import G, dev, graph_case, host, say  # noqa: F401  (G is a fixture)

pytestmark = pytest.mark.gpu

POLICY = {"fifo": O.FifoCache, "lru": O.LruCache}


def check_cache(c, ref: "O.FifoCache", feats):
    assert np.array_equal(c.slot_map(), ref.slot_map)
    owners, rows = c.contents()
    assert np.array_equal(owners, ref.owner)
    d = feats.shape[1]
    assert np.array_equal(rows[:, :d].view(np.uint8), feats[owners].view(np.uint8))


FIFO_CASES = [  # (d, dtype, r, ring): ring None = the whole cache
    (64, "f32", 0.3, None), (64, "f32", 0.3, 100), (602, "f32", 0.25, 7),
    (3, "f32", 0.5, 1), (128, "bf16", 0.2, 333), (100, "bf16", 1.0, None), (16, "f32", 0.3, 0)]


@pytest.mark.parametrize("store_on_device", [False, True])
@pytest.mark.parametrize("d,dtype,r,ring", FIFO_CASES)
@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_dynamic_gather_sequence(G, policy, d, dtype, r, ring, store_on_device):
    import torch
    n, u, v = graph_case("random-5000-30000-7")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, d, dtype, seed=d + 3)
    c = G.Cache(g, feats, dtype, r, store_on_device=store_on_device)
    ring = c.n_cached if ring is None else min(ring, c.n_cached)
    c.set_policy(policy, ring)
    ref = POLICY[policy](csr, r, ring)
    check_cache(c, ref, feats)
    rng = np.random.default_rng(d)
    pool = rng.permutation(n).astype(np.int32)
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    for b in range(6):
        # consecutive batches overlap, so rows admitted by one are hit by the next
        m = [1500, 1, 0, 2200, 900, 1500][b]
        ids = np.ascontiguousarray(pool[(b * 700) % 3000:][:m])
        say(policy, d, dtype, r, ring, store_on_device, b, m)
        out = torch.full((max(m, 1), c.ld), -7, dtype=torch.int16 if dtype == "bf16" else torch.float32,
                         device="cuda")
        ids_d = dev(ids if m else np.zeros(1, np.int32))
        G.gather(c, ids_d.data_ptr(), m, out, counts)
        ref_rows, ref_counts = ref.gather(feats, ids)
        assert np.array_equal(host(counts), ref_counts)
        assert np.array_equal(host(out, dtype)[:m, :d].view(np.uint8), ref_rows.view(np.uint8))
        check_cache(c, ref, feats)


def test_policy_errors_and_static_default(G):
    import torch
    n, u, v = graph_case("random-3000-40000-1")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, 8, "f32", seed=1)
    c = G.Cache(g, feats, "f32", 0.1)
    for pol, k in [(7, 1), (3, 1), (1, c.n_cached + 1), (1, -1), (2, c.n_cached + 1), (2, -1)]:
        with pytest.raises(G.GnnavError) as e:
            G._check(G._lib.gnnav_cache_set_policy(c._h, pol, k))
        assert e.value.status == 1
    _, slot, _ = O.rank_cache(csr, 0.1)
    ids = np.arange(0, n, 3, dtype=np.int32)
    out = torch.zeros((ids.size, c.ld), device="cuda")
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    ids_d = dev(ids)
    G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
    assert np.array_equal(c.slot_map(), slot), "the default policy must leave the cache unchanged"
    # FIFO, then back to static: the admitted vertices stay, nothing more moves
    c.set_policy("fifo", c.n_cached // 2)
    ref = O.FifoCache(csr, 0.1, c.n_cached // 2)
    G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
    ref.gather(feats, ids)
    check_cache(c, ref, feats)
    c.set_policy("static")
    G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
    check_cache(c, ref, feats)
    # then LRU from the current contents (recency restarts in slot order)
    c.set_policy("lru", c.n_cached // 3)
    lru = O.LruCache(csr, 0.1, c.n_cached // 3)
    lru.slot_map[:], lru.owner[:] = ref.slot_map, ref.owner
    for ids2 in (ids, ids[::2], np.arange(1, n, 7, dtype=np.int32)):
        ids2 = np.ascontiguousarray(ids2)
        ids2_d = dev(ids2)
        G.gather(c, ids2_d.data_ptr(), ids2.size, out, counts)
        lru.gather(feats, ids2)
        check_cache(c, lru, feats)


def _dynamic_workload():
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], wl.dtype, seed=11 + l) for l in range(wl.L)]
    return wl, s, d, wl.features(), ws


def _oracle_dynamic_batches(policy, wl, s, d, feats, ws, r, ring, nb):
    csr = O.build_csr(wl.n, s, d)
    ref = POLICY[policy](csr, r, ring)
    out = []
    for b in range(nb):
        blocks = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b))
        h0, counts = ref.gather(feats, blocks.nodes)
        logits = O.sage_forward(blocks, O.to_f64(h0, wl.dtype), [O.to_f64(w, wl.dtype) for w in ws],
                                bf16=wl.dtype == "bf16")
        out.append((h0, counts, logits, ref.slot_map.copy(), ref.owner.copy()))
    return out


def _check_dynamic_step(step, want, dtype, d):
    h0, counts, logits = want[:3]
    assert np.array_equal(host(step.counts), counts)
    assert np.array_equal(host(step.h0_view(), dtype)[:, :d].view(np.uint8), h0.view(np.uint8))
    assert_rows_close(host(step.logits[:step.sizes[0]]), logits, BF16_TOL if dtype == "bf16" else FP32_TOL,
                      "logits")


@pytest.mark.parametrize("ring_frac", [1.0, 0.1])
@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_dynamic_async_steps(G, policy, ring_frac):
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl, s, d, feats, ws = _dynamic_workload()
    r = 0.2
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, feats, wl.dtype, r)
    ring = int(c.n_cached * ring_frac)
    c.set_policy(policy, ring)
    want = _oracle_dynamic_batches(policy, wl, s, d, feats, ws, r, ring, 4)
    step = MiniBatchStep(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype)
    for b in range(4):
        say(policy, "async", ring_frac, b)
        step.enqueue(dev(wl.seeds(b)), wl.rng_seed(b))
        step.finish()
        _check_dynamic_step(step, want[b], wl.dtype, wl.d)
        assert np.array_equal(c.slot_map(), want[b][3])
        assert np.array_equal(c.contents()[0], want[b][4])


@pytest.mark.parametrize("depth", [2, 3])
@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_dynamic_pipeline(G, policy, depth):
    """Batches in flight on several streams update the cache in call order."""
    from paper_2404_09544_amd.step import Pipeline, to_device_weights
    wl, s, d, feats, ws = _dynamic_workload()
    r = 0.2
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, feats, wl.dtype, r)
    ring = c.n_cached // 2
    c.set_policy(policy, ring)
    nb = 2 * depth
    want = _oracle_dynamic_batches(policy, wl, s, d, feats, ws, r, ring, nb)
    pipe = Pipeline(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype, depth=depth)
    seeds_dev = [dev(wl.seeds(b)) for b in range(nb)]
    for rnd in range(2):
        slots = []
        for k in range(depth):
            b = rnd * depth + k
            say(policy, "pipeline", depth, b)
            slots.append((b, pipe.enqueue(seeds_dev[b], wl.rng_seed(b))))
        for b, slot in slots:
            slot.finish()
            _check_dynamic_step(slot, want[b], wl.dtype, wl.d)
    pipe.synchronize()
    assert np.array_equal(c.slot_map(), want[-1][3])
    owners, rows = c.contents()
    assert np.array_equal(owners, want[-1][4])
    assert np.array_equal(rows[:, :wl.d].view(np.uint8), feats[owners].view(np.uint8))
