"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bit-exact for integer work (CSR, slot map, sampled neighbours, frontiers,
local ids, gathered rows, hit/miss counts); per-row relative L2 error
within 1e-5 (fp32) or 2e-2 (bf16) for aggregation, combine and the full
forward.  Every oracle input is generated here or by the workload
generators; nothing the GPU computes is fed to the oracle.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W
from parity_util import BF16_TOL, FP32_TOL, assert_rows_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    import paper_2404_09544_amd as g
    return g


def say(*a):
    print("[case]", *a, flush=True)


def dev(a, dtype=None):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to("cuda")


def host(t, dtype="f32"):
    a = t.detach().cpu().numpy()
    return a.view(np.uint16) if dtype == "bf16" else a


def padded(x: np.ndarray, dtype: str) -> np.ndarray:
    """Copy rows into a zero-padded 16-byte stride."""
    import paper_2404_09544_amd as g
    ld = g.padded_ld(x.shape[1], dtype)
    out = np.zeros((x.shape[0], ld), x.dtype)
    out[:, :x.shape[1]] = x
    return out


GRAPHS = ["empty", "one_edge", "path", "star", "clique", "isolated", "deg_k"]


def graph_case(name):
    if name in GRAPHS:
        return W.tiny_graph(name)
    if name.startswith("random"):
        _, n, m, s = name.split("-")
        return W.random_graph(int(n), int(m), int(s))
    wl = W.Workload(name)
    s, d = wl.edges()
    return wl.n, s, d


# ------------------------------------------------------------ CSR, cache

@pytest.mark.parametrize("name", GRAPHS + ["random-3000-40000-1", "chunglu-10k-d64"])
@pytest.mark.parametrize("i64", [False, True])
def test_csr_and_slot_map(G, name, i64):
    say("csr", name, i64)
    n, u, v = graph_case(name)
    ref = O.build_csr(n, u, v)
    g = G.Graph(n, u, v, offsets_i64=i64)
    rp, col = g.csr_host()
    assert g.nnz == ref.nnz and g.offsets_i64 == i64
    assert np.array_equal(rp, ref.row_ptr) and np.array_equal(col, ref.col)
    assert g.max_degree == (int(ref.degrees().max()) if n else 0)
    feats = W.features(n, 3, "f32", seed=7)
    for r in [0.0, 1.0 / max(n, 1), 0.5, 1.0]:
        c = G.Cache(g, feats, "f32", r)
        _, slot, cnum = O.rank_cache(ref, r)
        assert c.n_cached == cnum
        assert np.array_equal(c.slot_map(), slot)


def test_build_errors(G):
    with pytest.raises(G.GnnavError) as e:
        G.Graph(3, [0, 1], [1, 3])
    assert e.value.status == 2
    g = G.Graph(3, [0, 1], [1, 2])
    with pytest.raises(G.GnnavError) as e:
        G.Cache(g, np.zeros((3, 4), np.float32), "f32", 1.5)
    assert e.value.status == 1
    with pytest.raises(G.GnnavError):
        G.Cache(g, np.zeros((3, 4), np.float32), "f32", float("nan"))


# ---------------------------------------------------------------- sample

def compare_blocks(G, g_blocks, ref: "O.Blocks"):
    nodes, sizes, ip, nb, ix = g_blocks.to_host()
    assert sizes == ref.sizes
    assert np.array_equal(nodes, ref.nodes)
    for h in range(len(ip)):
        assert np.array_equal(ip[h], ref.indptr[h]), f"indptr hop {h + 1}"
        assert np.array_equal(nb[h], ref.nbrs[h]), f"neighbours hop {h + 1}"
        assert np.array_equal(ix[h], ref.indices[h]), f"indices hop {h + 1}"


SAMPLE_CASES = [
    *[(k, "all", [5, 5]) for k in GRAPHS],
    *[(k, "one", [1, 0, 2]) for k in GRAPHS],
    ("star", "all", [150, 3]),            # k > 64: LDS selection path, many collisions
    ("star", "one", [64, 65]),
    ("random-3000-40000-1", "rand", [25, 10]),
    ("random-3000-40000-2", "rand", [100, 3]),
    ("random-3000-40000-3", "rand", [-1, 2]),
    ("random-3000-40000-4", "rand", [64, 65, 1]),
    ("random-3000-40000-5", "none", [5, 5]),
    ("chunglu-10k-d64", "batch", [5, 5]),
    ("chunglu-10k-d64", "batch", [25, 10, 5]),
    # edges of the rows-per-wavefront selection (8, 16 and 32 lanes per row)
    ("random-3000-40000-6", "rand", [8, 9]),
    ("random-3000-40000-7", "rand", [16, 17, 2]),
    ("random-3000-40000-8", "rand", [32, 33]),
    ("star", "all", [8, 16]),
    # one hop (its relabel is the only one) and four hops (each relabel rides
    # with the next hop's first scan)
    ("random-3000-40000-9", "rand", [7]),
    ("chunglu-10k-d64", "batch", [3, 4, 3, 2]),
]


@pytest.mark.parametrize("i64", [False, True])
@pytest.mark.parametrize("case", SAMPLE_CASES, ids=lambda c: f"{c[0]}-{c[1]}-{'_'.join(map(str, c[2]))}")
def test_sample_parity(G, case, i64):
    name, seeds_kind, fanouts = case
    say("sample", name, seeds_kind, fanouts, i64)
    n, u, v = graph_case(name)
    ref_csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v, offsets_i64=i64)
    rng = np.random.default_rng(len(name) + len(fanouts))
    if seeds_kind == "all":
        seeds = np.arange(n, dtype=np.int32)[::-1].copy()
    elif seeds_kind == "one":
        seeds = np.array([0], np.int32)[:min(1, n)]
    elif seeds_kind == "rand":
        seeds = rng.integers(0, n, 700).astype(np.int32)       # with repeats
    elif seeds_kind == "none":
        seeds = np.zeros(0, np.int32)
    else:
        seeds = W.Workload(name).seeds(1)
    blocks = G.Blocks()
    for b in range(2):
        rs = W.rng_seed_for_batch(b)
        ref = O.sample_blocks(ref_csr, seeds, fanouts, rs)
        G.sample(g, dev(seeds), fanouts, rs, blocks)
        compare_blocks(G, blocks, ref)


def test_sample_bad_seed_then_reuse(G):
    n, u, v = graph_case("random-3000-40000-1")
    g = G.Graph(n, u, v)
    blocks = G.Blocks()
    say("sample bad seed")
    with pytest.raises(G.GnnavError) as e:
        G.sample(g, dev(np.array([5, n, 7, -1], np.int32)), [3, 2], 9, blocks)
    assert e.value.status == 2
    seeds = np.array([5, 7, 11, 5], np.int32)
    G.sample(g, dev(seeds), [3, 2], 9, blocks)
    compare_blocks(G, blocks, O.sample_blocks(O.build_csr(n, u, v), seeds, [3, 2], 9))
    with pytest.raises(G.GnnavError) as e:
        G.sample(g, dev(seeds), [2000], 9, blocks)
    assert e.value.status == 1


def test_sample_blocks_reused_across_graphs(G):
    """One Blocks object (one node table, never cleared between calls) sampling
    a larger graph, a smaller one, and the larger one again: entries left by
    earlier calls must count as unseen."""
    big = graph_case("random-3000-40000-1")
    n2, u2, v2 = graph_case("random-3000-40000-2")
    keep = (u2 < 2000) & (v2 < 2000)
    small = (2000, u2[keep], v2[keep])
    blocks = G.Blocks()
    for i, (n, u, v) in enumerate([big, small, big, small]):
        say("blocks reuse", i, n)
        g = G.Graph(n, u, v)
        seeds = np.random.default_rng(i).integers(0, n, 500).astype(np.int32)
        G.sample(g, dev(seeds), [10, 5], 40 + i, blocks)
        compare_blocks(G, blocks, O.sample_blocks(O.build_csr(n, u, v), seeds, [10, 5], 40 + i))


# ---------------------------------------------------------------- gather

GATHER_CASES = [(1, "f32"), (3, "f32"), (64, "f32"), (100, "f32"), (602, "f32"),
                (3, "bf16"), (128, "bf16"), (200, "bf16")]


@pytest.mark.parametrize("store_on_device", [False, True])
@pytest.mark.parametrize("d,dtype", GATHER_CASES)
def test_gather_parity(G, d, dtype, store_on_device):
    import torch
    n, u, v = graph_case("random-5000-30000-7")
    ref_csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, d, dtype, seed=d)
    rng = np.random.default_rng(d)
    ids = rng.integers(0, n, 3001).astype(np.int32)
    ids[[5, 77, 3000]] = [-1, n, n + 5]
    for r in [0.0, 1.0 / n, 0.5, 1.0]:
        say("gather", d, dtype, store_on_device, r)
        c = G.Cache(g, feats, dtype, r, store_on_device=store_on_device)
        _, slot, _ = O.rank_cache(ref_csr, r)
        ref_rows, ref_counts = O.gather(feats, slot, ids)
        out = torch.full((ids.size, c.ld), -7, dtype=torch.int16 if dtype == "bf16" else torch.float32,
                         device="cuda")
        counts = torch.zeros(3, dtype=torch.int64, device="cuda")
        ids_d = dev(ids)
        G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
        got = host(out, dtype)
        assert np.array_equal(host(counts), ref_counts)
        assert np.array_equal(got[:, :d].view(np.uint8), ref_rows.view(np.uint8))
        elt = 2 if dtype == "bf16" else 4
        tail = (-(d * elt)) % 16 // elt
        if tail:
            assert not got[:, d:d + tail].any(), "padding up to the 16-byte boundary must be zero"


@pytest.mark.parametrize("wait", [False, True])
def test_gather_device_count(G, wait):
    """gather_n reads the request count from device memory; with copy_after
    the row copies wait for an event recorded on another stream."""
    import torch
    n, u, v = graph_case("random-5000-30000-7")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, 100, "f32", seed=4)
    c = G.Cache(g, feats, "f32", 0.3)
    _, slot, _ = O.rank_cache(csr, 0.3)
    ids = np.random.default_rng(9).integers(0, n, 3001).astype(np.int32)
    ids_d = dev(ids)
    other = torch.cuda.Stream()
    for m in [3001, 1777, 0, 1]:
        say("gather_n", wait, m)
        n_d = dev(np.array([m], np.int32))
        out = torch.full((ids.size, c.ld), -7.0, device="cuda")
        counts = torch.full((3,), 9, dtype=torch.int64, device="cuda")
        ev = None
        if wait:
            # work on another stream whose end the copies must see: it fills
            # the output, and the gather then overwrites the requested rows
            ev = torch.cuda.Event()
            other.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(other):
                torch.cuda._sleep(2000000)
                out.fill_(-5.0)
                ev.record(other)
        G.gather_n(c, ids_d.data_ptr(), n_d.data_ptr(), ids.size, out, counts, copy_after=ev)
        torch.cuda.synchronize()
        ref_rows, ref_counts = O.gather(feats, slot, ids[:m])
        got = host(out)
        assert np.array_equal(host(counts), ref_counts)
        assert np.array_equal(got[:m, :100].view(np.uint8), ref_rows.view(np.uint8))
        if wait:
            assert (got[m:] == -5.0).all()


def test_gather_link_workgroups(G):
    """The number of host-link workgroups changes nothing in the result."""
    import torch
    n, u, v = graph_case("random-5000-30000-7")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    feats = W.features(n, 602, "f32", seed=5)
    c = G.Cache(g, feats, "f32", 0.2)
    _, slot, _ = O.rank_cache(csr, 0.2)
    ids = np.random.default_rng(3).integers(0, n, 4000).astype(np.int32)
    ids_d = dev(ids)
    ref_rows, ref_counts = O.gather(feats, slot, ids)
    for wgs in (1, 3, 32, 64, 4096):
        say("gather link workgroups", wgs)
        c.set_link_workgroups(wgs)
        out = torch.full((ids.size, c.ld), -7.0, device="cuda")
        counts = torch.zeros(3, dtype=torch.int64, device="cuda")
        G.gather(c, ids_d.data_ptr(), ids.size, out, counts)
        assert np.array_equal(host(counts), ref_counts)
        assert np.array_equal(host(out)[:, :602].view(np.uint8), ref_rows.view(np.uint8))
    for bad in (0, 4097, -1):
        with pytest.raises(G.GnnavError) as e:
            c.set_link_workgroups(bad)
        assert e.value.status == 1
    c.set_link_workgroups(64)


def test_profile_records_every_launch(G):
    """Recording counts each timed launch once; per-launch durations add up
    to the total and the CSR row pointers come back without the columns."""
    import torch
    n, u, v = graph_case("random-3000-40000-1")
    csr = O.build_csr(n, u, v)
    g = G.Graph(n, u, v)
    rp, col = g.csr_host(with_col=False)
    assert col is None and np.array_equal(rp, csr.row_ptr)
    c = G.Cache(g, W.features(n, 16, "f32"), "f32", 0.5)
    ids = dev(np.arange(0, n, 2, dtype=np.int32))
    out = torch.zeros((ids.numel(), c.ld), device="cuda")
    counts = torch.zeros(3, dtype=torch.int64, device="cuda")
    G.profile_start()
    for _ in range(5):
        G.gather(c, ids.data_ptr(), ids.numel(), out, counts)
    prof = G.profile_stop()
    smp = G.profile_samples()
    assert prof["gather_rows"][0] == 5 and prof["classify"][0] == 5
    for name, (launches, ms) in prof.items():
        assert smp[name].size == launches
        assert abs(float(smp[name].astype(np.float64).sum()) - ms) <= 1e-3 * max(ms, 1e-3)
        assert (smp[name] >= 0).all()


def test_gather_empty_and_errors(G):
    import torch
    n, u, v = graph_case("path")
    g = G.Graph(n, u, v)
    c = G.Cache(g, W.features(n, 4, "f32"), "f32", 0.5)
    counts = torch.full((3,), 9, dtype=torch.int64, device="cuda")
    out = torch.zeros((1, c.ld), device="cuda")
    G.gather(c, 0, 0, out, counts)
    assert host(counts).tolist() == [0, 0, 0]
    bad = torch.zeros((4, 5), device="cuda")       # 20-byte rows: not 16-byte aligned
    ids0 = dev(np.zeros(4, np.int32))
    with pytest.raises(G.GnnavError):
        G.gather(c, ids0.data_ptr(), 4, bad, counts)


# ----------------------------------------------------- aggregate, combine

AGG_CASES = [(1, "f32"), (3, "f32"), (64, "f32"), (100, "f32"), (256, "f32"), (602, "f32"),
             (1100, "f32"), (3, "bf16"), (128, "bf16"), (256, "bf16")]


@pytest.mark.parametrize("d,dtype", AGG_CASES)
def test_aggregate_mean_parity(G, d, dtype):
    import torch
    say("aggregate", d, dtype)
    n, u, v = graph_case("isolated" if d == 3 else "random-4000-20000-3")
    csr = O.build_csr(n, u, v)
    seeds = np.arange(0, n, 2, dtype=np.int32)
    ref_b = O.sample_blocks(csr, seeds, [7], 5)
    ip, ix = ref_b.indptr[0], ref_b.indices[0]
    X = W.features(ref_b.sizes[1], d, dtype, seed=d + 1)
    Xd = dev(padded(X, dtype))
    ld = G.padded_ld(d, dtype)
    out = torch.full((ip.size - 1, ld), 3, dtype=Xd.dtype, device="cuda")
    ip_d, ix_d = dev(ip), dev(ix)          # keep the device copies alive until the kernel ran
    G.aggregate_mean(ip_d.data_ptr(), ix_d.data_ptr(), ip.size - 1, Xd, d, dtype, out)
    torch.cuda.synchronize()
    got = O.to_f64(host(out, dtype)[:, :d], dtype)
    Wt = np.concatenate([np.zeros((d, 1)), np.zeros((d, 1))])
    _, agg = O.sage_layer(ip, ix, O.to_f64(X, dtype), Wt, relu=False, bf16=dtype == "bf16",
                          round_out=False, want_agg=True)
    _, agg_abs = O.sage_layer(ip, ix, np.abs(O.to_f64(X, dtype)), Wt, relu=False, bf16=False,
                              round_out=False, want_agg=True)
    empty = np.diff(ip) == 0
    assert not got[empty].any()
    assert_rows_close(got[~empty], agg[~empty], BF16_TOL if dtype == "bf16" else FP32_TOL, "aggregate",
                      floor=np.linalg.norm(agg_abs[~empty], axis=1))
    if ld > d:
        elt = 2 if dtype == "bf16" else 4
        tail = (-(d * elt)) % 16 // elt
        assert not host(out, dtype)[:, d:d + tail].any()


# Small M runs the skinny kernel (fewer than 160 64x64 tiles; 16 wavefronts
# per 16x16 output while there are at most 512 of those, else 8: 8000 and
# 2100 rows here).  Larger M: fp32 runs the split-bf16 kernel on 128x128 or
# 64x64 tiles (both taken here, e.g. 20000 x 602 x 256 and 40000 x 37 x
# 130), bf16 the ring kernel on 128x64 / 64x64 / 128x128 tiles.  K tails:
# d_in not a multiple of the 32 (fp32) or 64 (bf16) k step; ragged M and N.
# fp32 tail split (d_in >= 128, 256 < 128x128 tiles <= 640), three k-pieces
# per tail tile: 20000 x 602 x 256, 24001 x 300 x 250, 40000 x 128 x 100 (one
# tile column); two: 33000 x 300 x 256, 20000 x 160 x 300 (three columns).
COMBINE_CASES = [(1, 3, 16), (63, 64, 41), (64, 100, 47), (65, 602, 256), (1000, 128, 64),
                 (777, 256, 256), (130, 5, 300), (20000, 602, 256), (12000, 64, 41),
                 (12001, 100, 100), (9000, 256, 256), (10240, 3, 47), (6000, 128, 260),
                 (66000, 100, 256), (40000, 37, 130), (33000, 300, 256), (24001, 300, 250),
                 (8000, 256, 64), (2100, 128, 100), (40000, 128, 100), (20000, 160, 300)]


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("m,d_in,d_out", COMBINE_CASES)
@pytest.mark.parametrize("mode", ["f32", "bf16", "bf16_f32out"])
def test_combine_parity(G, m, d_in, d_out, relu, mode):
    import torch
    say("combine", m, d_in, d_out, relu, mode)
    dtype = "f32" if mode == "f32" else "bf16"
    out_bf16 = mode == "bf16"
    S = W.features(m, d_in, dtype, seed=m + d_in)
    A = W.features(m, d_in, dtype, seed=m + d_in + 1)
    Wt = W.glorot(d_in, d_out, dtype, seed=d_out)
    Sd, Ad, Wd = dev(padded(S, dtype)), dev(padded(A, dtype)), dev(Wt)
    ld_o = G.padded_ld(d_out, "bf16" if out_bf16 else "f32")
    out = torch.zeros((m, ld_o), dtype=torch.int16 if out_bf16 else torch.float32, device="cuda")
    G.combine(Sd, Ad, m, d_in, Wd, d_out, dtype, relu, out_bf16, out)
    got = O.to_f64(host(out, "bf16" if out_bf16 else "f32")[:, :d_out], "bf16" if out_bf16 else "f32")
    z = np.concatenate([O.to_f64(S, dtype), O.to_f64(A, dtype)], axis=1) @ O.to_f64(Wt, dtype)
    if relu:
        z = np.maximum(z, 0)
    if out_bf16:
        z = O.round_bf16_array(z)
    assert_rows_close(got, z, BF16_TOL if dtype == "bf16" else FP32_TOL, "combine")


# bf16 output rows that are not 16-byte aligned (odd stride, base one element
# in): the kernels fall back from 16-byte row stores to element stores.  The
# words around each row must keep their sentinel.
@pytest.mark.parametrize("m,d_in,d_out", [(20000, 128, 256), (12001, 100, 47), (40000, 37, 130), (500, 64, 33)])
def test_combine_bf16_unaligned_out(G, m, d_in, d_out):
    import torch
    say("combine unaligned out", m, d_in, d_out)
    S = W.features(m, d_in, "bf16", seed=m + 5)
    A = W.features(m, d_in, "bf16", seed=m + 6)
    Wt = W.glorot(d_in, d_out, "bf16", seed=d_out + 1)
    Sd, Ad, Wd = dev(padded(S, "bf16")), dev(padded(A, "bf16")), dev(Wt)
    ld_o = d_out + 1 if d_out % 2 == 0 else d_out + 2
    buf = torch.full((m * ld_o + 2,), -7, dtype=torch.int16, device="cuda")
    out = buf[1:1 + m * ld_o].view(m, ld_o)
    G.combine(Sd, Ad, m, d_in, Wd, d_out, "bf16", True, True, out)
    got_all = buf.cpu().numpy()
    rows = got_all[1:1 + m * ld_o].reshape(m, ld_o)
    assert got_all[0] == -7 and got_all[-1] == -7 and (rows[:, d_out:] == -7).all()
    got = O.to_f64(rows[:, :d_out].view(np.uint16), "bf16")
    z = np.concatenate([O.to_f64(S, "bf16"), O.to_f64(A, "bf16")], axis=1) @ O.to_f64(Wt, "bf16")
    z = O.round_bf16_array(np.maximum(z, 0))
    assert_rows_close(got, z, BF16_TOL, "combine")


# -------------------------------------------------------------- end to end

def run_pipeline_case(G, n, u, v, feats, dtype, dims, fanouts, r, seeds, rng_seed,
                      store_on_device=False, i64=False):
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    ws = [W.glorot(dims[l], dims[l + 1], dtype, seed=11 + l) for l in range(len(fanouts))]
    g = G.Graph(n, u, v, offsets_i64=i64)
    c = G.Cache(g, feats, dtype, r, store_on_device=store_on_device)
    step = MiniBatchStep(g, c, to_device_weights(ws, dtype), dims, fanouts, dtype)
    logits = step.run(dev(seeds), rng_seed)
    got_logits = host(logits).copy()
    got_h0 = host(step.h0_view(), dtype)[:, :feats.shape[1]].copy()
    got_counts = host(step.counts).copy()
    # oracle
    csr = O.build_csr(n, u, v)
    ref_b = O.sample_blocks(csr, seeds, fanouts, rng_seed)
    compare_blocks(G, step.blocks, ref_b)
    _, slot, _ = O.rank_cache(csr, r)
    h0, counts = O.gather(feats, slot, ref_b.nodes)
    assert np.array_equal(got_counts, counts)
    assert np.array_equal(got_h0.view(np.uint8), h0.view(np.uint8))
    ref = O.sage_forward(ref_b, O.to_f64(h0, dtype), [O.to_f64(w, dtype) for w in ws],
                         bf16=dtype == "bf16")
    assert_rows_close(got_logits, ref, BF16_TOL if dtype == "bf16" else FP32_TOL, "logits")
    return step


@pytest.mark.parametrize("batch", [0, 1, 2])
def test_forward_tiny_workload(G, batch):
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    say("forward", wl.name, batch)
    run_pipeline_case(G, wl.n, s, d, wl.features(), wl.dtype, wl.dims, wl.fanouts, wl.cfg["cache"],
                      wl.seeds(batch), wl.rng_seed(batch), store_on_device=True)


@pytest.mark.parametrize("r", [0.0, 0.3, 1.0])
def test_forward_tiny_workload_host_store(G, r):
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    say("forward host store", r)
    run_pipeline_case(G, wl.n, s, d, wl.features(), wl.dtype, wl.dims, wl.fanouts, r,
                      wl.seeds(3), wl.rng_seed(3))


@pytest.mark.parametrize("i64", [False, True])
def test_forward_bf16_three_hops(G, i64):
    n, u, v = W.random_graph(6000, 50000, 21)
    say("forward bf16", i64)
    feats = W.features(n, 128, "bf16", seed=3)
    seeds = W.epoch_permutation(n)[:300]
    run_pipeline_case(G, n, u, v, feats, "bf16", [128, 64, 48, 10], [6, 4, 3], 0.25, seeds, 77,
                      i64=i64)


def test_forward_f32_wide_rows(G):
    n, u, v = W.random_graph(3000, 60000, 5)
    say("forward f32 d=602")
    feats = W.features(n, 602, "f32", seed=4)
    seeds = W.epoch_permutation(n)[:128]
    run_pipeline_case(G, n, u, v, feats, "f32", [602, 256, 41], [25, 10], 0.5, seeds, 1234)


def test_determinism(G):
    """Same inputs, fresh handles: bit-identical frontiers, rows and logits."""
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    say("determinism")
    outs = []
    for _ in range(2):
        step = run_pipeline_case(G, wl.n, s, d, wl.features(), wl.dtype, wl.dims, wl.fanouts, 0.4,
                                 wl.seeds(5), wl.rng_seed(5))
        outs.append((host(step.logits[:step.sizes[0]]).copy(), step.blocks.to_host()))
    assert np.array_equal(outs[0][0].view(np.uint32), outs[1][0].view(np.uint32))
    for a, b in zip(outs[0][1][2:], outs[1][1][2:]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


# ------------------------------------------------ async step, two streams

def oracle_batch(n, u, v, feats, dtype, dims, fanouts, r, seeds, rng_seed, ws):
    csr = O.build_csr(n, u, v)
    ref_b = O.sample_blocks(csr, seeds, fanouts, rng_seed)
    _, slot, _ = O.rank_cache(csr, r)
    h0, counts = O.gather(feats, slot, ref_b.nodes)
    logits = O.sage_forward(ref_b, O.to_f64(h0, dtype), [O.to_f64(w, dtype) for w in ws],
                            bf16=dtype == "bf16")
    return ref_b, h0, counts, logits


def check_step(G, step, ref, dtype, d):
    ref_b, h0, counts, logits = ref
    compare_blocks(G, step.blocks, ref_b)
    assert np.array_equal(host(step.counts), counts)
    got_h0 = host(step.h0_view(), dtype)[:, :d]
    assert np.array_equal(got_h0.view(np.uint8), h0.view(np.uint8))
    got = host(step.logits[:step.sizes[0]])
    assert_rows_close(got, logits, BF16_TOL if dtype == "bf16" else FP32_TOL, "logits")


@pytest.mark.parametrize("r,on_device", [(0.0, True), (0.3, False)])
def test_async_step_matches_oracle(G, r, on_device):
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    feats = wl.features()
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], wl.dtype, seed=11 + l) for l in range(wl.L)]
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, feats, wl.dtype, r, store_on_device=on_device)
    step = MiniBatchStep(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype)
    for b in range(3):
        say("async step", r, on_device, b)
        seeds = wl.seeds(b)
        step.enqueue(dev(seeds), wl.rng_seed(b))
        step.finish()
        check_step(G, step, oracle_batch(wl.n, s, d, feats, wl.dtype, wl.dims, wl.fanouts, r, seeds,
                                         wl.rng_seed(b), ws), wl.dtype, wl.d)


def test_async_step_bf16_three_hops(G):
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    n, u, v = W.random_graph(6000, 50000, 21)
    feats = W.features(n, 128, "bf16", seed=3)
    dims, fanouts = [128, 64, 48, 10], [6, 4, 3]
    ws = [W.glorot(dims[l], dims[l + 1], "bf16", seed=11 + l) for l in range(3)]
    g = G.Graph(n, u, v, offsets_i64=True)
    c = G.Cache(g, feats, "bf16", 0.25)
    step = MiniBatchStep(g, c, to_device_weights(ws, "bf16"), dims, fanouts, "bf16")
    seeds = W.epoch_permutation(n)[:300]
    say("async bf16")
    step.enqueue(dev(seeds), 77)
    step.finish()
    check_step(G, step, oracle_batch(n, u, v, feats, "bf16", dims, fanouts, 0.25, seeds, 77, ws), "bf16", 128)


def test_async_bad_seed_reported_at_sync(G):
    from paper_2404_09544_amd.step import MiniBatchStep, to_device_weights
    n, u, v = W.random_graph(500, 4000, 2)
    g = G.Graph(n, u, v)
    c = G.Cache(g, W.features(n, 8, "f32"), "f32", 0.5)
    ws = [W.glorot(8, 4, "f32", seed=1)]
    step = MiniBatchStep(g, c, to_device_weights(ws, "f32"), [8, 4], [3], "f32")
    say("async bad seed")
    step.enqueue(dev(np.array([1, n + 3, 2], np.int32)), 5)
    with pytest.raises(G.GnnavError) as e:
        step.finish()
    assert e.value.status == 2


@pytest.mark.parametrize("on_device", [False, True])
@pytest.mark.parametrize("cu_partition", [False, True])
@pytest.mark.parametrize("depth", [2, 3])
def test_pipeline_matches_oracle(G, depth, cu_partition, on_device):
    """Batches on alternating streams give each batch's oracle result, also
    with each stream on its own share of the compute units, and with the
    whole store in HBM (then the gathers are not ordered on the link)."""
    from paper_2404_09544_amd.step import Pipeline, to_device_weights
    wl = W.Workload("chunglu-10k-d64")
    s, d = wl.edges()
    feats = wl.features()
    r = 0.3
    ws = [W.glorot(wl.dims[l], wl.dims[l + 1], wl.dtype, seed=11 + l) for l in range(wl.L)]
    g = G.Graph(wl.n, s, d)
    c = G.Cache(g, feats, wl.dtype, r, store_on_device=on_device)
    pipe = Pipeline(g, c, to_device_weights(ws, wl.dtype), wl.dims, wl.fanouts, wl.dtype, depth=depth,
                    cu_partition=cu_partition)
    seeds_dev = [dev(wl.seeds(b)) for b in range(2 * depth)]
    for rnd in range(2):
        slots = []
        for k in range(depth):
            b = rnd * depth + k
            say("pipeline", depth, cu_partition, on_device, b)
            slots.append((b, pipe.enqueue(seeds_dev[b], wl.rng_seed(b))))
        for b, slot in slots:
            slot.finish()
            check_step(G, slot, oracle_batch(wl.n, s, d, feats, wl.dtype, wl.dims, wl.fanouts, r,
                                             wl.seeds(b), wl.rng_seed(b), ws), wl.dtype, wl.d)
