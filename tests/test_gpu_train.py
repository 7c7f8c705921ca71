"""GPU parity of the training half of the iteration (loss, backward, SGD).

Each backward kernel is checked alone on oracle inputs, and the whole
train step (forward with kept activations, loss, backward, update) against
the oracle's train_step.  fp32 throughout: per-row relative L2 within 1e-5,
with the absolute-value sums as the floor of each row's scale where a sum
cancels (the classical bound on its rounding error).  Every sum on the GPU
runs in a fixed order, so repeated runs must give identical bits.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W
from parity_util import FP32_TOL, assert_rows_close
from test_gpu_parity import G, dev, graph_case, host, padded, say  # noqa: F401  (G is a fixture)

pytestmark = pytest.mark.gpu


def f32(a):
    return np.asarray(a, dtype=np.float32)


# ------------------------------------------------------------- softmax-CE

@pytest.mark.parametrize("n,C", [(1, 1), (7, 3), (1000, 41), (4096, 64), (333, 100), (0, 5)])
def test_softmax_xent_parity(G, n, C):
    import torch
    say("softmax_xent", n, C)
    rng = np.random.default_rng(n + C)
    Z = f32(rng.normal(size=(n, C)) * 3)
    y = rng.integers(0, C, n).astype(np.int32)
    ld = G.padded_ld(C, "f32")
    Zd = dev(padded(Z, "f32")) if n else torch.zeros((1, ld), device="cuda")
    dz = torch.full((max(n, 1), ld), 7.0, device="cuda")
    loss = torch.zeros(1, device="cuda")
    G.softmax_xent(Zd, n, C, dev(y) if n else dev(np.zeros(1, np.int32)), dz, loss)
    ref_loss, ref_dz = O.softmax_xent(Z.astype(np.float64), y)
    got = float(host(loss)[0])
    assert got == pytest.approx(ref_loss, rel=FP32_TOL, abs=1e-7)
    if n:
        assert_rows_close(host(dz)[:n, :C], ref_dz, FP32_TOL, "dZ")


def test_softmax_xent_bad_label_gives_nan(G):
    import torch
    Z = f32(np.zeros((3, 4)))
    dz = torch.zeros((3, 4), device="cuda")
    loss = torch.zeros(1, device="cuda")
    G.softmax_xent(dev(Z), 3, 4, dev(np.array([0, 4, 1], np.int32)), dz, loss)
    assert np.isnan(host(loss)[0])
    assert not host(dz)[1].any()
    with pytest.raises(G.GnnavError):
        G.softmax_xent(dev(Z), 3, 5, dev(np.zeros(3, np.int32)), dz, loss)   # ld 4 < 5 classes


# ------------------------------------------------- aggregation adjoint

def _block(kind, seed):
    """(indptr, indices, n_dst, n_src) of a sampled block of the given kind."""
    if kind == "star":
        # every destination row points at the same source: one long column
        n_dst = 3000
        indptr = np.arange(n_dst + 1, dtype=np.int32)
        return indptr, np.zeros(n_dst, np.int32), n_dst, n_dst + 5
    if kind == "empty_rows":
        indptr = np.array([0, 0, 2, 2, 5, 5], np.int32)
        return indptr, np.array([5, 1, 0, 6, 6], np.int32), 5, 9
    n, u, v = graph_case(kind)
    csr = O.build_csr(n, u, v)
    seeds = W.epoch_permutation(n, seed)[: max(1, n // 5)]
    blk = O.sample_blocks(csr, seeds, [12], seed)
    return blk.indptr[0], blk.indices[0], blk.sizes[0], blk.sizes[1]


AGGT_CASES = [("random-5000-30000-7", 64), ("random-5000-30000-7", 602), ("random-5000-30000-7", 3),
              ("random-5000-30000-7", 1), ("random-4000-20000-3", 256), ("chunglu-10k-d64", 100),
              ("star", 64), ("empty_rows", 5)]


@pytest.mark.parametrize("self_term,masked", [(False, False), (True, True), (True, False)])
@pytest.mark.parametrize("kind,d", AGGT_CASES)
def test_aggregate_mean_backward_parity(G, kind, d, self_term, masked):
    import torch
    say("aggregate_t", kind, d, self_term, masked)
    ip, ix, n_dst, n_src = _block(kind, 3)
    rng = np.random.default_rng(d)
    dagg = f32(rng.normal(size=(n_dst, d)))
    dself = f32(rng.normal(size=(n_dst, d))) if self_term else None
    mask = f32(rng.normal(size=(n_src, d))) if masked else None
    ld = G.padded_ld(d, "f32")
    out = torch.full((n_src, ld), 3.0, device="cuda")
    ipd, ixd = dev(ip), dev(ix if ix.size else np.zeros(1, np.int32))
    args = dict(dself=dev(padded(dself, "f32")) if self_term else None,
                mask=dev(padded(mask, "f32")) if masked else None)
    dagg_d = dev(padded(dagg, "f32"))
    G.aggregate_mean_backward(ipd.data_ptr(), ixd.data_ptr(), n_dst, n_src, dagg_d, d, out, **args)
    got = host(out).copy()
    ref = O.aggregate_mean_t(ip, ix, n_src, dagg.astype(np.float64))
    floor = O.aggregate_mean_t(ip, ix, n_src, np.abs(dagg.astype(np.float64)))
    if self_term:
        ref[:n_dst] += dself
        floor[:n_dst] += np.abs(dself)
    if masked:
        ref = ref * (mask > 0)
        floor = floor * (mask > 0)
    assert_rows_close(got[:, :d], ref, FP32_TOL, "dX", floor=np.linalg.norm(floor, axis=1))
    assert not got[:, d:].any(), "padding must be zero"
    # same bits on a second run
    G.aggregate_mean_backward(ipd.data_ptr(), ixd.data_ptr(), n_dst, n_src, dagg_d, d, out, **args)
    assert np.array_equal(host(out), got)


def test_aggregate_mean_backward_many_sources(G):
    """A source range past 2^16 makes the radix sort take three passes."""
    import torch
    n_dst, k = 30000, 4
    n_src = 200000
    rng = np.random.default_rng(5)
    ix = rng.integers(0, n_src, n_dst * k).astype(np.int32)
    ip = (np.arange(n_dst + 1) * k).astype(np.int32)
    dagg = f32(rng.normal(size=(n_dst, 16)))
    out = torch.zeros((n_src, 16), device="cuda")
    ipd, ixd, dagg_d = dev(ip), dev(ix), dev(dagg)      # keep the device copies alive
    G.aggregate_mean_backward(ipd.data_ptr(), ixd.data_ptr(), n_dst, n_src, dagg_d, 16, out)
    ref = O.aggregate_mean_t(ip, ix, n_src, dagg.astype(np.float64))
    floor = O.aggregate_mean_t(ip, ix, n_src, np.abs(dagg.astype(np.float64)))
    assert_rows_close(host(out), ref, FP32_TOL, "dX", floor=np.linalg.norm(floor, axis=1))


# ---------------------------------------------------------- weight grad

# 2 * d_in * d_out not a multiple of 4 takes the reduce's one-element lanes:
# (1, 3, 41) with one split, (3000, 3, 41) with 12, (40000, 5, 33) with 64.
WGRAD_CASES = [(0, 8, 16), (1, 3, 41), (100, 100, 47), (5000, 602, 256), (20902, 602, 256), (95651, 100, 256),
               (13042, 256, 256), (1024, 256, 41), (777, 130, 70), (3000, 3, 41), (40000, 5, 33)]


@pytest.mark.parametrize("m,d_in,d_out", WGRAD_CASES)
def test_weight_grad_parity(G, m, d_in, d_out):
    import torch
    say("wgrad", m, d_in, d_out)
    rng = np.random.default_rng(m + d_in)
    X = f32(rng.normal(size=(m, d_in)))
    A = f32(rng.normal(size=(m, d_in)))
    Gz = f32(rng.normal(size=(m, d_out)) / max(m, 1))
    dw = torch.full((2 * d_in, d_out), 5.0, device="cuda")
    if m:
        Xd, Ad, Gd = dev(padded(X, "f32")), dev(padded(A, "f32")), dev(padded(Gz, "f32"))
    else:
        Xd = Ad = Gd = torch.zeros((1, 16), device="cuda")
    G.weight_grad(Xd, Ad, m, d_in, Gd, d_out, dw)
    got = host(dw).copy()
    cat = np.concatenate([X, A], axis=1).astype(np.float64)
    ref = cat.T @ Gz.astype(np.float64)
    floor = np.linalg.norm(np.abs(cat).T @ np.abs(Gz.astype(np.float64)), axis=1)
    if m == 0:
        assert not got.any()
        return
    assert_rows_close(got, ref, FP32_TOL, "dW", floor=floor)
    G.weight_grad(Xd, Ad, m, d_in, Gd, d_out, dw)
    assert np.array_equal(host(dw), got), "weight gradient must be bitwise reproducible"


# ------------------------------------------------------------- train step

def _train_case(n, u, v, feats, dims, fanouts, seeds, rng_seed, r=0.3):
    ws = [W.glorot(dims[l], dims[l + 1], "f32", seed=21 + l) for l in range(len(fanouts))]
    labels = W.labels(n, dims[-1], seed=8)
    return ws, labels


def _oracle_train(n, u, v, feats, dims, fanouts, seeds, rng_seed, ws, labels, lr):
    csr = O.build_csr(n, u, v)
    blk = O.sample_blocks(csr, seeds, fanouts, rng_seed)
    H0 = feats[blk.nodes].astype(np.float64)
    y = labels[blk.nodes[:blk.sizes[0]]]
    loss, logits, dWs, _ = O.train_step(blk, H0, ws, y, lr)
    # rounding scale of each weight-gradient row: the same sum over absolute
    # values, |[X | agg]|^T |dZ_l|, from the oracle's activations and dZ_l
    Wd = [np.asarray(w, np.float64) for w in ws]
    _, trace = O.sage_forward(blk, H0, Wd, keep=True)
    _, dZ = O.softmax_xent(logits, y)
    floors = [np.linalg.norm(f, axis=1) for f in O.sage_backward(blk, H0, Wd, trace, dZ, abs_scale=True)]
    return loss, logits, dWs, floors


def _check_train(G, step_out, ref, ws0, lr, dims):
    loss, logits, grads, weights = step_out
    rloss, rlogits, rdW, floors = ref
    assert loss == pytest.approx(rloss, rel=FP32_TOL)
    assert_rows_close(logits, rlogits, FP32_TOL, "logits")
    for l, (g, rg) in enumerate(zip(grads, rdW)):
        assert_rows_close(g, rg, FP32_TOL, f"dW{l + 1}", floor=floors[l])
        # the update is W - lr * dW applied to the GPU's own dW, within one
        # float32 rounding of the result
        want = ws0[l].astype(np.float64) - np.float64(np.float32(lr)) * g.astype(np.float64)
        np.testing.assert_allclose(weights[l], want, rtol=2.0 ** -22, atol=1e-30)


def _run_gpu_train(G, g, c, ws, dims, fanouts, seeds, rng_seed, labels, lr, async_mode):
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wdev = to_device_weights(ws, "f32")
    step = MiniBatchStep(g, c, wdev, dims, fanouts, "f32")
    lab = dev(labels)
    grads = [torch.zeros((2 * dims[l], dims[l + 1]), device="cuda") for l in range(len(fanouts))]
    out = step.train(dev(seeds), rng_seed, lab, lr, grads=grads, async_mode=async_mode)
    if async_mode:
        out = step.finish()
    torch.cuda.synchronize()
    return step, (float(host(step.loss)[0]), host(out).copy(), [host(x).copy() for x in grads],
                  [host(w).copy() for w in wdev])


@pytest.mark.parametrize("async_mode", [False, True])
@pytest.mark.parametrize("case", ["tiny2", "tiny3", "chunglu-10k"])
def test_train_step_matches_oracle(G, case, async_mode):
    say("train step", case, async_mode)
    if case == "chunglu-10k":
        wl = W.Workload("chunglu-10k-d64")
        n, (u, v) = wl.n, wl.edges()
        feats, dims, fanouts, seeds, rs = wl.features(), wl.dims, wl.fanouts, wl.seeds(1), wl.rng_seed(1)
    else:
        n, u, v = W.random_graph(3000, 20000, 4)
        feats = W.features(n, 37, "f32", seed=2)
        dims, fanouts = ([37, 48, 11], [6, 4]) if case == "tiny2" else ([37, 24, 20, 9], [5, 3, 4])
        seeds, rs = W.epoch_permutation(n)[:200], 17
    ws, labels = _train_case(n, u, v, feats, dims, fanouts, seeds, rs)
    lr = 0.1
    g = G.Graph(n, u, v)
    c = G.Cache(g, feats, "f32", 0.3)
    _, got = _run_gpu_train(G, g, c, ws, dims, fanouts, seeds, rs, labels, lr, async_mode)
    ref = _oracle_train(n, u, v, feats, dims, fanouts, seeds, rs, ws, labels, lr)
    _check_train(G, got, ref, ws, lr, dims)
    # identical bits on a repeat from the same starting weights
    _, again = _run_gpu_train(G, g, c, ws, dims, fanouts, seeds, rs, labels, lr, async_mode)
    assert again[0] == got[0]
    for a, b in zip(again[2], got[2]):
        assert np.array_equal(a, b)


def test_train_steps_lower_the_loss(G):
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, wl.features(), "f32", 0.3)
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], "f32", seed=3 + l) for l in range(wl.L)]
    step = MiniBatchStep(g, c, to_device_weights(ws, "f32"), wl.dims, wl.fanouts, "f32")
    lab = dev(W.labels(wl.n, wl.dims[-1]))
    seeds = dev(wl.seeds(0))
    losses = []
    for it in range(8):
        step.train(seeds, wl.rng_seed(0), lab, 0.5)
        torch.cuda.synchronize()
        losses.append(float(host(step.loss)[0]))
    say("losses", losses)
    assert losses[-1] < losses[0]


@pytest.mark.parametrize("policy", ["fifo", "lru"])
def test_train_with_dynamic_cache(G, policy):
    """Training batches through a self-updating cache (ring over half the
    cached rows), on one stream and on two streams over halves of the
    compute units: bit-identical weights and losses, and both caches end as
    the oracle's policy leaves them after gathering the same frontiers."""
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, Pipeline, to_device_weights
    from test_gpu_cache_update import POLICY, check_cache
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    csr = O.build_csr(wl.n, s, d)
    g = G.Graph(wl.n, s, d)
    feats = wl.features()
    r = 0.3
    caches = [G.Cache(g, feats, "f32", r) for _ in range(2)]
    ring = caches[0].n_cached // 2
    for c in caches:
        c.set_policy(policy, ring)
    ref = POLICY[policy](csr, r, ring)
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], "f32", seed=3 + l) for l in range(wl.L)]
    lab = dev(W.labels(wl.n, wl.dims[-1]))
    seeds = [dev(wl.seeds(b)) for b in range(6)]
    w_seq = to_device_weights(ws, "f32")
    step = MiniBatchStep(g, caches[0], w_seq, wl.dims, wl.fanouts, "f32")
    for b in range(6):
        say("train", policy, "sequential", b)
        step.train(seeds[b], wl.rng_seed(b), lab, 0.3, async_mode=True)
        torch.cuda.synchronize()
        ref.gather(feats, O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b)).nodes)
    loss_seq = float(host(step.loss)[0])
    w_pipe = to_device_weights(ws, "f32")
    pipe = Pipeline(g, caches[1], w_pipe, wl.dims, wl.fanouts, "f32", depth=2, cu_partition=True)
    say("train", policy, "pipeline")
    slots = [pipe.enqueue_train(seeds[b], wl.rng_seed(b), lab, 0.3) for b in range(6)]
    pipe.synchronize()
    for a, b in zip(w_seq, w_pipe):
        assert np.array_equal(host(a), host(b))
    assert float(host(slots[-1].loss)[0]) == loss_seq
    for c in caches:
        check_cache(c, ref, feats)


def test_train_pipeline_matches_sequential(G):
    """Training batches on two streams (each batch's forward waits for the
    previous update), also on two shares of the compute units, end with the
    same weights as one stream."""
    import torch
    from paper_2404_09544_amd.step import MiniBatchStep, Pipeline, to_device_weights
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, wl.features(), "f32", 0.3)
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], "f32", seed=3 + l) for l in range(wl.L)]
    lab = dev(W.labels(wl.n, wl.dims[-1]))
    seeds = [dev(wl.seeds(b)) for b in range(6)]
    w_seq = to_device_weights(ws, "f32")
    step = MiniBatchStep(g, c, w_seq, wl.dims, wl.fanouts, "f32")
    seq_losses = []
    for b in range(6):
        step.train(seeds[b], wl.rng_seed(b), lab, 0.3, async_mode=True)
        torch.cuda.synchronize()
        seq_losses.append(float(host(step.loss)[0]))
    for link, part in ((None, False), (32, False), (1, False), (64, True)):
        say("train pipeline", link, part)
        w_pipe = to_device_weights(ws, "f32")
        pipe = Pipeline(g, c, w_pipe, wl.dims, wl.fanouts, "f32", depth=2, link_workgroups=link,
                        cu_partition=part)
        slots = [pipe.enqueue_train(seeds[b], wl.rng_seed(b), lab, 0.3) for b in range(6)]
        pipe.synchronize()
        for a, b in zip(w_seq, w_pipe):
            assert np.array_equal(host(a), host(b))
        assert float(host(slots[-1].loss)[0]) == seq_losses[-1]
    c.set_link_workgroups(64)
