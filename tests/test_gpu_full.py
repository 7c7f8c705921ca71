"""GPU parity at the full workload sizes.

For each workload: the device CSR equals the oracle's; a batch through
MiniBatchStep's synchronous form gives frontiers, blocks, gathered rows and
hit/miss counts identical to the oracle's, and the logits of sampled seed
rows match the oracle's receptive-field forward within tolerance (the
10M-node R-MAT workload at cache fractions 0, 0.25 and 1).  Then the launch
configuration bench.py times: the first three batches through the Pipeline
(asynchronous sampling, gathers ordered on the host link, grids and GEMM
tiles planned from the Eq. 12 bounds) in each stream and compute-unit
setting the bench may pick, each batch checked in full against the oracle
-- every logits row of F_0 where the oracle's forward takes seconds, sampled
rows on the two largest graphs.  With a self-updating cache (FIFO, LRU) on
the 233k workload: counts, rows and the cache's state after four pipelined
batches.
"""
import sys
import time

import numpy as np
import pytest

import oracle as O
import workloads as W
from parity_util import BF16_TOL, FP32_TOL, assert_rows_close

pytestmark = pytest.mark.gpu

FULL = ["chunglu-169k-d128", "chunglu-233k-d602", "chunglu-2450k-d100", "rmat-10m-d128"]
_state = {}


def say(*a):
    print("[full]", *a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available()
    import paper_2404_09544_amd as g
    yield g
    _state.clear()


def load(G, name):
    if name in _state:
        return _state[name]
    _state.clear()
    t = time.perf_counter()
    wl = W.Workload(name)
    src, dst = wl.edges()
    say(name, f"edges {src.size} pairs ({time.perf_counter() - t:.1f}s)")
    csr = O.build_csr(wl.n, src, dst)
    say(name, f"oracle CSR nnz={csr.nnz} ({time.perf_counter() - t:.1f}s)")
    g = G.Graph(wl.n, src, dst, offsets_i64=wl.cfg["offsets_i64"])
    say(name, f"device CSR ({time.perf_counter() - t:.1f}s)")
    _state[name] = (wl, src, dst, csr, g)
    return _state[name]


@pytest.mark.parametrize("name", FULL)
def test_full_csr(G, name):
    wl, _, _, csr, g = load(G, name)
    rp, col = g.csr_host()
    assert g.offsets_i64 == wl.cfg["offsets_i64"]
    assert np.array_equal(rp, csr.row_ptr)
    assert np.array_equal(col, csr.col)


@pytest.mark.parametrize("name", FULL)
def test_full_batch(G, name):
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl, _, _, csr, g = load(G, name)
    feats = wl.features()
    ws = wl.weights()
    wd = [O.to_f64(w, wl.dtype) for w in ws]
    bf16 = wl.dtype == "bf16"
    tol = BF16_TOL if bf16 else FP32_TOL
    sweep = wl.cfg.get("cache_sweep", [wl.cfg["cache"]])
    for r in sweep:
        t = time.perf_counter()
        c = G.Cache(g, feats, wl.dtype, r, store_on_device=wl.cfg["store_on_device"])
        step = MiniBatchStep(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype)
        _, slot, _ = O.rank_cache(csr, r)
        for b in ([7] if wl.n > 1_000_000 else [0, 1, 2, 7]):
            say(name, f"r={r} batch {b}")
            seeds = wl.seeds(b)
            logits = step.run(torch.from_numpy(seeds).cuda(), wl.rng_seed(b))
            got_logits = logits.cpu().numpy()
            nodes, sizes, ip, nb, ix = step.blocks.to_host()
            ref_b = O.sample_blocks(csr, seeds, wl.fanouts, wl.rng_seed(b))
            assert sizes == ref_b.sizes
            assert np.array_equal(nodes, ref_b.nodes)
            for h in range(wl.L):
                assert np.array_equal(ip[h], ref_b.indptr[h]), f"indptr hop {h + 1}"
                assert np.array_equal(nb[h], ref_b.nbrs[h]), f"neighbours hop {h + 1}"
                assert np.array_equal(ix[h], ref_b.indices[h]), f"indices hop {h + 1}"
            h0, counts = O.gather(feats, slot, ref_b.nodes)
            assert np.array_equal(step.counts.cpu().numpy(), counts)
            got_h0 = step.h0_view().cpu().numpy()[:, :wl.d]
            assert np.array_equal(got_h0.view(np.uint8), h0.view(np.uint8))
            rows = np.random.default_rng(b).choice(sizes[0], size=min(96, sizes[0]), replace=False)
            ref = O.sage_forward_rows(ref_b, O.to_f64(h0, wl.dtype), wd, rows, bf16=bf16)
            assert_rows_close(got_logits[rows], ref, tol, f"{name} r={r} logits")
            say(name, f"r={r} batch {b}: sizes {sizes} hits/misses {counts.tolist()} "
                      f"({time.perf_counter() - t:.1f}s)")
        c.close()


@pytest.mark.parametrize("name", ["chunglu-2450k-d100", "rmat-10m-d128"])
def test_full_large_batch(G, name):
    """A batch of 16,384 seeds (consecutive batches of the epoch permutation
    taken together) on the two largest graphs: frontiers of millions of
    nodes, multi-thousand-tile scans and the widest grids, every block,
    count and gathered row bit-exact, sampled logits rows within tolerance."""
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl, _, _, csr, g = load(G, name)
    feats = wl.features()
    ws = wl.weights()
    wd = [O.to_f64(w, wl.dtype) for w in ws]
    bf16 = wl.dtype == "bf16"
    r = wl.cfg["cache"]
    t = time.perf_counter()
    c = G.Cache(g, feats, wl.dtype, r, store_on_device=wl.cfg["store_on_device"])
    step = MiniBatchStep(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype)
    _, slot, _ = O.rank_cache(csr, r)
    seeds = np.concatenate([wl.seeds(b) for b in range(16384 // wl.batch)])
    rng = wl.rng_seed(99)
    logits = step.run(torch.from_numpy(seeds).cuda(), rng).cpu().numpy()
    nodes, sizes, ip, nb, ix = step.blocks.to_host()
    say(name, f"large batch on the GPU: sizes {sizes} ({time.perf_counter() - t:.1f}s)")
    ref_b = O.sample_blocks(csr, seeds, wl.fanouts, rng)
    assert sizes == ref_b.sizes
    assert np.array_equal(nodes, ref_b.nodes)
    for h in range(wl.L):
        assert np.array_equal(ip[h], ref_b.indptr[h]), f"indptr hop {h + 1}"
        assert np.array_equal(nb[h], ref_b.nbrs[h]), f"neighbours hop {h + 1}"
        assert np.array_equal(ix[h], ref_b.indices[h]), f"indices hop {h + 1}"
    h0, counts = O.gather(feats, slot, ref_b.nodes)
    assert np.array_equal(step.counts.cpu().numpy(), counts)
    got_h0 = step.h0_view().cpu().numpy()[:, :wl.d]
    assert np.array_equal(got_h0.view(np.uint8), h0.view(np.uint8))
    rows = np.random.default_rng(5).choice(sizes[0], size=128, replace=False)
    ref = O.sage_forward_rows(ref_b, O.to_f64(h0, wl.dtype), wd, rows, bf16=bf16)
    assert_rows_close(logits[rows], ref, BF16_TOL if bf16 else FP32_TOL, f"{name} large-batch logits")
    say(name, f"large batch checked: hits/misses {counts.tolist()} ({time.perf_counter() - t:.1f}s)")
    c.close()


# logits rows checked per pipelined batch: every row of F_0 (None) where the
# oracle's double-precision forward of the whole batch takes seconds
PIPE_ROWS = {"chunglu-169k-d128": None, "chunglu-233k-d602": None, "chunglu-2450k-d100": 256,
             "rmat-10m-d128": 256}
# (streams, compute units partitioned): every setting bench.py's pipelined
# leg may time (it keeps the fastest of a short trial of each)
PIPE_CFG = [(3, False), (2, True), (3, True)]


@pytest.mark.parametrize("cfg", PIPE_CFG, ids=lambda c: f"{c[0]}streams-{'shares' if c[1] else 'all'}")
@pytest.mark.parametrize("name", FULL)
def test_full_pipeline(G, name, cfg):
    """Batches 0, 1, 2 through Pipeline.enqueue with the bench's streams,
    compute-unit partition and link-workgroup setting (64), as the bench's
    pipelined leg enqueues them (with two streams: batches 0 and 1 in flight
    together, then batch 2); every batch against the oracle."""
    import torch
    from paper_2404_09544_amd.step import Pipeline, to_device_weights
    wl, _, _, csr, g = load(G, name)
    feats = wl.features()
    ws = wl.weights()
    wd = [O.to_f64(w, wl.dtype) for w in ws]
    bf16 = wl.dtype == "bf16"
    tol = BF16_TOL if bf16 else FP32_TOL
    r = wl.cfg["cache"]
    t = time.perf_counter()
    c = G.Cache(g, feats, wl.dtype, r, store_on_device=wl.cfg["store_on_device"])
    _, slot_map, _ = O.rank_cache(csr, r)
    depth, part = cfg
    pipe = Pipeline(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype, depth=depth,
                    link_workgroups=64, cu_partition=part)
    seeds_dev = [torch.from_numpy(wl.seeds(b)).cuda() for b in range(3)]
    for b in range(3):
        if b % depth == 0:
            slots = [pipe.enqueue(seeds_dev[x], wl.rng_seed(x)) for x in range(b, min(b + depth, 3))]
            pipe.synchronize()
            say(name, f"pipeline of batches {b}..{b + len(slots) - 1} done ({time.perf_counter() - t:.1f}s)")
        st = slots[b % depth]
        logits = st.finish().cpu().numpy()
        nodes, sizes, ip, nb, ix = st.blocks.to_host()
        ref_b = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b))
        assert sizes == ref_b.sizes, f"batch {b} sizes"
        assert np.array_equal(nodes, ref_b.nodes)
        for h in range(wl.L):
            assert np.array_equal(ip[h], ref_b.indptr[h]), f"batch {b} indptr hop {h + 1}"
            assert np.array_equal(nb[h], ref_b.nbrs[h]), f"batch {b} neighbours hop {h + 1}"
            assert np.array_equal(ix[h], ref_b.indices[h]), f"batch {b} indices hop {h + 1}"
        h0, counts = O.gather(feats, slot_map, ref_b.nodes)
        assert np.array_equal(st.counts.cpu().numpy(), counts), f"batch {b} counts"
        got_h0 = st.h0_view().cpu().numpy()[:, :wl.d]
        assert np.array_equal(got_h0.view(np.uint8), h0.view(np.uint8)), f"batch {b} gathered rows"
        k = PIPE_ROWS[name]
        if k is None:
            ref = O.sage_forward(ref_b, O.to_f64(h0, wl.dtype), wd, bf16=bf16)
            got = logits
        else:
            rows = np.random.default_rng(100 + b).choice(sizes[0], size=min(k, sizes[0]), replace=False)
            ref = O.sage_forward_rows(ref_b, O.to_f64(h0, wl.dtype), wd, rows, bf16=bf16)
            got = logits[rows]
        assert_rows_close(got, ref, tol, f"{name} pipelined batch {b} logits ({got.shape[0]} rows)")
        say(name, f"pipelined batch {b}: sizes {sizes} ({time.perf_counter() - t:.1f}s)")
    c.close()


TRAIN_FULL = ["chunglu-169k-d128", "chunglu-233k-d602", "chunglu-2450k-d100"]


@pytest.mark.parametrize("name", TRAIN_FULL)
def test_full_train_step(G, name):
    """One training iteration at full size (the bench's train leg, async):
    loss and every layer's weight gradient against the oracle's train step,
    with the absolute-value sums as each gradient row's rounding scale."""
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl, _, _, csr, g = load(G, name)
    feats = wl.features()
    ws = wl.weights()
    labels = wl.labels()
    t = time.perf_counter()
    c = G.Cache(g, feats, wl.dtype, wl.cfg["cache"], store_on_device=wl.cfg["store_on_device"])
    step = MiniBatchStep(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype)
    grads = [torch.zeros((2 * wl.dims[l], wl.dims[l + 1]), device="cuda") for l in range(wl.L)]
    b, lr = 3, 0.05
    seeds = wl.seeds(b)
    step.train(torch.from_numpy(seeds).cuda(), wl.rng_seed(b), torch.from_numpy(labels).cuda(), lr, grads=grads,
               async_mode=True)
    step.finish()
    loss = float(step.loss.cpu().numpy()[0])
    got = [x.cpu().numpy() for x in grads]
    say(name, f"GPU train step done ({time.perf_counter() - t:.1f}s)")
    ref_b = O.sample_blocks(csr, seeds, wl.fanouts, wl.rng_seed(b))
    H0 = feats[ref_b.nodes].astype(np.float64)
    y = labels[ref_b.nodes[:ref_b.sizes[0]]]
    Wd = [O.to_f64(w, wl.dtype) for w in ws]
    logits, trace = O.sage_forward(ref_b, H0, Wd, keep=True)
    rloss, dZ = O.softmax_xent(logits, y)
    rdW = O.sage_backward(ref_b, H0, Wd, trace, dZ)
    floors = O.sage_backward(ref_b, H0, Wd, trace, dZ, abs_scale=True)
    say(name, f"oracle train step done ({time.perf_counter() - t:.1f}s), loss {rloss:.6f} vs {loss:.6f}")
    assert loss == pytest.approx(rloss, rel=FP32_TOL)
    for l in range(wl.L):
        assert_rows_close(got[l], rdW[l], FP32_TOL, f"{name} dW{l + 1}", floor=np.linalg.norm(floors[l], axis=1))
    c.close()


@pytest.mark.parametrize("name", ["chunglu-233k-d602", "chunglu-2450k-d100"])
def test_full_biased_batch(G, name):
    """A batch through the bench's step with locality-biased sampling."""
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl, _, _, csr, g = load(G, name)
    feats = wl.features()
    ws = wl.weights()
    r, eta, b = wl.cfg["cache"], 8, 5
    c = G.Cache(g, feats, wl.dtype, r, store_on_device=wl.cfg["store_on_device"])
    step = MiniBatchStep(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype, eta=eta)
    _, slot, _ = O.rank_cache(csr, r)
    seeds = wl.seeds(b)
    step.enqueue(torch.from_numpy(seeds).cuda(), wl.rng_seed(b))
    logits = step.finish().cpu().numpy()
    nodes, sizes, ip, nb, ix = step.blocks.to_host()
    ref_b = O.sample_blocks(csr, seeds, wl.fanouts, wl.rng_seed(b), bias_slot_map=slot, eta=eta)
    assert sizes == ref_b.sizes
    assert np.array_equal(nodes, ref_b.nodes)
    for h in range(wl.L):
        assert np.array_equal(nb[h], ref_b.nbrs[h]), f"neighbours hop {h + 1}"
        assert np.array_equal(ix[h], ref_b.indices[h]), f"indices hop {h + 1}"
    h0, counts = O.gather(feats, slot, ref_b.nodes)
    assert np.array_equal(step.counts.cpu().numpy(), counts)
    rows = np.random.default_rng(b).choice(sizes[0], size=64, replace=False)
    ref = O.sage_forward_rows(ref_b, O.to_f64(h0, wl.dtype), [O.to_f64(w, wl.dtype) for w in ws], rows)
    assert_rows_close(logits[rows], ref, FP32_TOL, f"{name} biased logits")
    say(name, f"biased eta={eta}: hits/misses {counts.tolist()}")
    c.close()


@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_full_dynamic_cache(G, policy):
    """The 233k workload with a self-updating cache (ring over half the
    cached rows), four batches through two pipelined streams on halves of
    the compute units: each batch's hit/miss counts and gathered rows, then
    the slot map, every slot's vertex and sampled cached rows, against the
    oracle's policy applied batch after batch."""
    import torch
    from paper_2404_09544_amd.step import Pipeline, to_device_weights
    name = "chunglu-233k-d602"
    wl, _, _, csr, g = load(G, name)
    feats = wl.features()
    r = wl.cfg["cache"]
    t = time.perf_counter()
    c = G.Cache(g, feats, wl.dtype, r, store_on_device=wl.cfg["store_on_device"])
    ring = c.n_cached // 2
    c.set_policy(policy, ring)
    ref = {"fifo": O.FifoCache, "lru": O.LruCache}[policy](csr, r, ring)
    pipe = Pipeline(g, c, to_device_weights(wl.weights(), wl.dtype), wl.dims, wl.fanouts, wl.dtype, depth=2,
                    link_workgroups=64, cu_partition=True)
    seeds_dev = [torch.from_numpy(wl.seeds(b)).cuda() for b in range(4)]
    for b0 in (0, 2):
        slots = [pipe.enqueue(seeds_dev[b], wl.rng_seed(b)) for b in (b0, b0 + 1)]
        pipe.synchronize()
        for b, st in zip((b0, b0 + 1), slots):
            st.finish()
            ref_b = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b))
            h0, counts = ref.gather(feats, ref_b.nodes)
            assert np.array_equal(st.counts.cpu().numpy(), counts), f"batch {b} counts"
            got = st.h0_view().cpu().numpy()[:, :wl.d]
            assert np.array_equal(got.view(np.uint8), h0.view(np.uint8)), f"batch {b} gathered rows"
            say(name, policy, f"batch {b}: hits/misses {counts[:2].tolist()} ({time.perf_counter() - t:.1f}s)")
    pipe.synchronize()
    assert np.array_equal(c.slot_map(), ref.slot_map)
    owners, rows = c.contents()
    assert np.array_equal(owners, ref.owner)
    pick = np.random.default_rng(7).choice(c.n_cached, 4096, replace=False)
    pick = np.concatenate([pick, np.arange(c.n_cached - ring, c.n_cached - ring + 512)])
    assert np.array_equal(rows[pick, :wl.d].view(np.uint8), feats[owners[pick]].view(np.uint8))
    c.close()
