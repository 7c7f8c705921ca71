"""GPU parity of the locality-biased sampler (cached neighbours weigh eta).

Frontiers, blocks and local ids must equal the oracle's bit for bit, for
static and self-updating (FIFO, LRU) caches, alone and inside the full step.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W
from parity_util import FP32_TOL, assert_rows_close
from test_gpu_parity import G, compare_blocks, dev, graph_case, host, say  # noqa: F401  (G is a fixture)

pytestmark = pytest.mark.gpu

BIASED_CASES = [
    ("star", 0.3, [5, 5], 8),
    ("star", 0.5, [64, 3], 2),
    ("clique", 0.4, [3, 2], 65536),
    ("deg_k", 0.5, [5, 6], 3),
    ("random-3000-40000-1", 0.3, [25, 10], 1),
    ("random-3000-40000-2", 0.3, [25, 10], 8),
    ("random-3000-40000-3", 0.0, [10, 10], 8),
    ("random-3000-40000-4", 1.0, [10, 10], 8),
    ("random-3000-40000-5", 0.2, [64, 1, 7], 100),
    ("chunglu-10k-d64", 0.3, [5, 5], 4),
    ("chunglu-10k-d64", 0.1, [25, 10, 5], 65536),
]


@pytest.mark.parametrize("i64", [False, True])
@pytest.mark.parametrize("case", BIASED_CASES, ids=lambda c: f"{c[0]}-r{c[1]}-{'_'.join(map(str, c[2]))}-eta{c[3]}")
def test_biased_sample_parity(G, case, i64):
    name, r, fanouts, eta = case
    say("biased sample", case, i64)
    n, u, v = graph_case(name)
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v, offsets_i64=i64)
    c = G.Cache(g, W.features(n, 4, "f32"), "f32", r)
    _, slot, _ = O.rank_cache(csr, r)
    seeds = W.epoch_permutation(n, 7)[: max(1, min(300, n // 3))]
    for async_ in (False, True):
        b = G.Blocks()
        seeds_d = dev(seeds)
        G.sample_biased(g, c, eta, seeds_d, fanouts, 1234, b, async_=async_)
        if async_:
            b.sync()
        ref = O.sample_blocks(csr, seeds, fanouts, 1234, bias_slot_map=slot, eta=eta)
        compare_blocks(G, b, ref)
        b.close()


def test_biased_sample_errors(G):
    n, u, v = graph_case("random-3000-40000-1")
    g = G.Graph(n, u, v)
    c = G.Cache(g, W.features(n, 4, "f32"), "f32", 0.3)
    n2, u2, v2 = graph_case("path")
    c_other = G.Cache(G.Graph(n2, u2, v2), W.features(n2, 4, "f32"), "f32", 0.5)
    b = G.Blocks()
    seeds = dev(np.arange(10, dtype=np.int32))
    for cache, eta, fan in [(c, 0, [5]), (c, 65537, [5]), (c, 4, [65]), (c_other, 4, [5])]:
        with pytest.raises(G.GnnavError) as e:
            G.sample_biased(g, cache, eta, seeds, fan, 1, b)
        assert e.value.status == 1


def test_biased_step_matches_oracle(G):
    """The full forward step with biased sampling (async path)."""
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    feats = wl.features()
    r, eta = 0.3, 8
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], "f32", seed=11 + l) for l in range(wl.L)]
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, feats, "f32", r)
    step = MiniBatchStep(g, c, to_device_weights(ws, "f32"), wl.dims, wl.fanouts, "f32", eta=eta)
    csr = O.build_csr(wl.n, s, d)
    _, slot, _ = O.rank_cache(csr, r)
    for b in range(3):
        seeds = wl.seeds(b)
        step.enqueue(dev(seeds), wl.rng_seed(b))
        step.finish()
        ref_b = O.sample_blocks(csr, seeds, wl.fanouts, wl.rng_seed(b), bias_slot_map=slot, eta=eta)
        compare_blocks(G, step.blocks, ref_b)
        h0, counts = O.gather(feats, slot, ref_b.nodes)
        assert np.array_equal(host(step.counts), counts)
        logits = O.sage_forward(ref_b, h0.astype(np.float64), [w.astype(np.float64) for w in ws])
        assert_rows_close(host(step.logits[:step.sizes[0]]), logits, FP32_TOL, "logits")
        plain = O.sample_blocks(csr, seeds, wl.fanouts, wl.rng_seed(b))
        _, counts_plain = O.gather(feats, slot, plain.nodes)
        say("hit rate biased / uniform", counts[0] / counts[:2].sum(), counts_plain[0] / counts_plain[:2].sum())


@pytest.mark.parametrize("depth", [1, 2])
@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_biased_sampling_with_dynamic_cache(G, policy, depth):
    """Each batch is sampled against the cache as the previous batch left it."""
    from test_gpu_cache_update import POLICY
    from paper_2404_09544_amd.step import Pipeline, to_device_weights
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    feats = wl.features()
    r, eta = 0.2, 16
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], "f32", seed=11 + l) for l in range(wl.L)]
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, feats, "f32", r)
    ring = c.n_cached // 2
    c.set_policy(policy, ring)
    pipe = Pipeline(g, c, to_device_weights(ws, "f32"), wl.dims, wl.fanouts, "f32", depth=depth, eta=eta)
    csr = O.build_csr(wl.n, s, d)
    dyn = POLICY[policy](csr, r, ring)
    want = []
    for b in range(5):
        ref_b = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b), bias_slot_map=dyn.slot_map.copy(),
                                eta=eta)
        _, counts = dyn.gather(feats, ref_b.nodes)
        want.append((ref_b, counts))
    seeds_dev = [dev(wl.seeds(b)) for b in range(5)]
    for b in range(5):
        say("biased", policy, depth, b)
        slot = pipe.enqueue(seeds_dev[b], wl.rng_seed(b))
        if depth == 1 or b % depth == depth - 1 or b == 4:
            pipe.synchronize()
        if depth == 1:
            slot.finish()
            compare_blocks(G, slot.blocks, want[b][0])
            assert np.array_equal(host(slot.counts), want[b][1])
    pipe.synchronize()
    assert np.array_equal(c.slot_map(), dyn.slot_map)


def test_biased_partition_follows_policy_changes(G):
    """Static cache: rows partitioned once by the slot map; a FIFO period
    moves the map, and the partition is rebuilt when static again."""
    import torch
    n, u, v = graph_case("random-3000-40000-2")
    csr = O.build_csr(n, u, v)
    feats = W.features(n, 8, "f32")
    g = G.Graph(n, u, v)
    c = G.Cache(g, feats, "f32", 0.3)
    seeds = W.epoch_permutation(n, 3)[:200]
    seeds_d = dev(seeds)
    b = G.Blocks()
    for phase in ["static", "fifo", "static"]:
        if phase == "fifo":
            c.set_policy("fifo", c.n_cached // 2)
            ids = dev(W.epoch_permutation(n, 9)[:1500])
            out = torch.zeros((1500, c.ld), device="cuda")
            counts = torch.zeros(3, dtype=torch.int64, device="cuda")
            G.gather(c, ids.data_ptr(), 1500, out, counts)   # moves the slot map
            torch.cuda.synchronize()
        else:
            c.set_policy("static")
        slot = c.slot_map()
        say("biased partition", phase)
        G.sample_biased(g, c, 8, seeds_d, [10, 5], 77, b)
        compare_blocks(G, b, O.sample_blocks(csr, seeds, [10, 5], 77, bias_slot_map=slot, eta=8))
    b.close()
