"""Pins of the CPU oracle against facts it does not compute itself.

Each test fixes a part of the oracle with something outside it: published
known-answer vectors, brute force on tiny inputs, closed forms, invariants
the paper states, special cases that reduce to a library routine, or the
distribution the paper's Eq. 2 demands.  No GPU is involved.
"""
import itertools
import math
import os

import numpy as np
import pytest

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _built():
    O.build(force=False)


# ------------------------------------------------------------- Philox ---

def test_philox_known_answers():
    """Philox4x32-10 against the published known-answer vectors."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        got = O.philox4x32_10(v[0:4], v[4:6])
        assert [int(x) for x in got] == v[6:10]


def test_draw_uses_counter_and_key_layout():
    """draw(seed, hop, v, j) is word 0 of Philox(ctr=(j, lo v, hi v, hop), key=(lo, hi seed))."""
    seed = (0x12345678 << 32) | 0x9abcdef0
    v = (7 << 32) | 3
    got = O.draw(seed, 5, v, 11)
    ref = O.philox4x32_10([11, 3, 7, 5], [0x9abcdef0, 0x12345678])[0]
    assert got == int(ref)
    # each component of the key changes the draw
    assert O.draw(seed, 6, v, 11) != got
    assert O.draw(seed, 5, v + 1, 11) != got
    assert O.draw(seed, 5, v, 12) != got
    assert O.draw(seed ^ 1, 5, v, 11) != got


# -------------------------------------------------------- range map O4 ---

@pytest.mark.parametrize("b", [1, 2, 3, 7, 10, 1000, 99991, 2**31 - 1, 2**32 - 1])
def test_below_inverse_boundaries(b):
    """floor(x*b/2^32): the first x mapping to t is ceil(t*2^32/b)."""
    rng = np.random.default_rng(b)
    ts = {0, b - 1} | set(int(t) for t in rng.integers(0, b, 50))
    for t in ts:
        x0 = -(-(t << 32) // b)          # ceil(t * 2^32 / b)
        assert O.below(x0, b) == t
        if x0 > 0:
            assert O.below(x0 - 1, b) == t - 1
    assert O.below(0xFFFFFFFF, b) == b - 1
    assert O.below(0, b) == 0


# ---------------------------------------------------------- CSR, O1 -------

@pytest.mark.parametrize("seed", range(6))
def test_csr_brute_force(seed):
    n, u, v = W.random_graph(n=40, m=200, seed=seed)
    csr = O.build_csr(n, u, v, symmetrize=True)
    adj = [set() for _ in range(n)]
    for a, b in zip(u.tolist(), v.tolist()):
        if a != b:
            adj[a].add(b)
            adj[b].add(a)
    assert csr.row_ptr[0] == 0
    for x in range(n):
        row = csr.col[csr.row_ptr[x]:csr.row_ptr[x + 1]].tolist()
        assert row == sorted(adj[x])
    assert csr.nnz % 2 == 0


def test_csr_directed_and_edge_cases():
    n, u, v = W.tiny_graph("isolated")
    csr = O.build_csr(n, u, v, symmetrize=False)
    expect = [set() for _ in range(n)]
    for a, b in zip(u.tolist(), v.tolist()):
        if a != b:
            expect[a].add(b)
    for x in range(n):
        assert csr.col[csr.row_ptr[x]:csr.row_ptr[x + 1]].tolist() == sorted(expect[x])
    e = O.build_csr(5, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert e.nnz == 0 and e.row_ptr.tolist() == [0] * 6
    with pytest.raises(ValueError):
        O.build_csr(3, [0], [3])


# -------------------------------------------------- degree ranking, O2 ---

@pytest.mark.parametrize("r", [0.0, 0.05, 0.2, 0.5, 1.0, 1e-9, 0.999999])
def test_rank_cache_brute_force(r):
    n, u, v = W.random_graph(n=300, m=900, seed=3)
    csr = O.build_csr(n, u, v)
    deg = csr.degrees()
    rank, slot, c = O.rank_cache(csr, r)
    assert rank.tolist() == sorted(range(n), key=lambda x: (-int(deg[x]), x))
    assert c == math.floor(r * n)
    cached = [x for x in range(n) if slot[x] >= 0]
    assert sorted(slot[cached].tolist()) == list(range(c))     # bijection onto [0, C)
    for s in range(c):
        assert slot[rank[s]] == s


# ------------------------------------------------- Floyd sampler, O5 ------

def _star(n):
    _, u, v = W.tiny_graph("star") if n == 200 else (None, np.zeros(n - 1, np.int32),
                                                       np.arange(1, n, dtype=np.int32))
    return O.build_csr(n, u, v)


def test_sample_node_properties():
    n, u, v = W.random_graph(n=60, m=700, seed=9)
    csr = O.build_csr(n, u, v)
    for node in range(n):
        row = csr.col[csr.row_ptr[node]:csr.row_ptr[node + 1]]
        for k in [0, 1, 3, 5, 10, 100, -1]:
            s = O.sample_node(csr, node, k, rng_seed=77, hop=1)
            want = len(row) if k < 0 else min(len(row), k)
            assert s.size == want
            assert len(set(s.tolist())) == s.size            # distinct
            assert set(s.tolist()) <= set(row.tolist())        # subset of the row
            if k < 0 or len(row) <= k:
                assert s.tolist() == row.tolist()              # whole row, CSR order


def test_sample_subsets_uniform():
    """Eq. 2 with fixed size: every k-subset of a deg-6 row equally likely."""
    csr = _star(7)                     # hub 0 has neighbours 1..6
    d, k, trials = 6, 3, 40000
    subsets = {frozenset(c): 0 for c in itertools.combinations(range(1, d + 1), k)}
    for t in range(trials):
        s = O.sample_node(csr, 0, k, rng_seed=(123 << 32) | t, hop=0)
        subsets[frozenset(s.tolist())] += 1
    exp = trials / len(subsets)
    chi2 = sum((c - exp) ** 2 / exp for c in subsets.values())
    # 19 degrees of freedom: P(chi2 > 50) < 1e-4
    assert chi2 < 50, chi2


def test_sample_marginal_inclusion():
    """Each neighbour of v is kept with probability k/deg (Eq. 2's indicator)."""
    csr = _star(200)                   # hub degree 199
    k, trials = 10, 6000
    hits = np.zeros(200, np.int64)
    for t in range(trials):
        s = O.sample_node(csr, 0, k, rng_seed=t, hop=1)
        hits[s] += 1
    p = k / 199
    frac = hits[1:] / trials
    sd = math.sqrt(p * (1 - p) / trials)
    assert np.all(np.abs(frac - p) < 5 * sd)
    assert abs(frac.mean() - p) < 1e-12 + 5 * sd / math.sqrt(199)


def test_sample_k1_uniform_single_draw():
    csr = _star(9)                     # hub degree 8
    counts = np.zeros(9, np.int64)
    trials = 16000
    for t in range(trials):
        s = O.sample_node(csr, 0, 1, rng_seed=99, hop=t)
        counts[s[0]] += 1
    exp = trials / 8
    chi2 = ((counts[1:] - exp) ** 2 / exp).sum()
    assert chi2 < 30                   # 7 dof


def test_sample_reproducible_per_node():
    """S_h(v) depends only on (rng_seed, hop, v): same in any batch."""
    n, u, v = W.random_graph(n=500, m=6000, seed=4)
    csr = O.build_csr(n, u, v)
    seed = W.rng_seed_for_batch(3)
    b1 = O.sample_blocks(csr, [5, 17, 42], [4, 3], seed)
    b2 = O.sample_blocks(csr, [42, 99, 5], [4, 3], seed)

    def rows(b):
        out = {}
        for i in range(b.sizes[0]):
            node = int(b.nodes[i])
            out[node] = b.nbrs[0][b.indptr[0][i]:b.indptr[0][i + 1]].tolist()
        return out
    r1, r2 = rows(b1), rows(b2)
    for node in (5, 42):
        assert r1[node] == r2[node]
        assert r1[node] == O.sample_node(csr, node, 4, seed, 0).tolist()


# --------------------------------------------------- hop expansion, O6 ----

def _check_blocks(csr, seeds, fanouts, rng_seed):
    b = O.sample_blocks(csr, seeds, fanouts, rng_seed)
    L = len(fanouts)
    # F_0: seeds, first occurrences, independent dict-based build
    f0 = list(dict.fromkeys(int(s) for s in seeds))
    assert b.nodes[:b.sizes[0]].tolist() == f0
    for h in range(1, L + 1):
        n_prev, n_h = b.sizes[h - 1], b.sizes[h]
        ip, nb, ix = b.indptr[h - 1], b.nbrs[h - 1], b.indices[h - 1]
        assert ip.size == n_prev + 1 and ip[0] == 0
        for i in range(n_prev):
            node = int(b.nodes[i])
            got = nb[ip[i]:ip[i + 1]].tolist()
            assert got == O.sample_node(csr, node, fanouts[h - 1], rng_seed, h - 1).tolist()
        # F_h = F_(h-1) + new ids in first-occurrence order
        seen = dict.fromkeys(b.nodes[:n_prev].tolist())
        for x in nb.tolist():
            seen.setdefault(x, None)
        assert b.nodes[:n_h].tolist() == list(seen)
        # indices map N_h into F_h; bijection and prefix property
        assert np.array_equal(b.nodes[ix], nb)
        assert ix.size == 0 or (ix.min() >= 0 and ix.max() < n_h)
        assert len(set(b.nodes[:n_h].tolist())) == n_h
        # Eq. 12 bound (tau = 1, no overlap)
        assert n_h <= n_prev * (1 + max(fanouts[h - 1], 0)) or fanouts[h - 1] < 0
        assert ip[-1] <= n_prev * max(fanouts[h - 1], 0) or fanouts[h - 1] < 0
    return b


@pytest.mark.parametrize("seed", range(4))
def test_blocks_random(seed):
    n, u, v = W.random_graph(n=400, m=3000, seed=seed)
    csr = O.build_csr(n, u, v)
    rng = np.random.default_rng(seed)
    seeds = rng.integers(0, n, 40).astype(np.int32)      # repeats allowed
    _check_blocks(csr, seeds, [5, 3, 2], W.rng_seed_for_batch(seed))


@pytest.mark.parametrize("kind", ["empty", "one_edge", "path", "star", "clique", "isolated", "deg_k"])
def test_blocks_tiny_graphs(kind):
    n, u, v = W.tiny_graph(kind)
    csr = O.build_csr(n, u, v)
    seeds = np.arange(n, dtype=np.int32)[::-1].copy()
    _check_blocks(csr, seeds, [5, 5], 7)
    _check_blocks(csr, seeds[:1], [1, 0, 2], 8)


def test_blocks_full_neighbourhood_is_whole_csr():
    """seeds = V in id order, k >= max degree: block 1 is the CSR itself."""
    n, u, v = W.random_graph(n=150, m=700, seed=11)
    csr = O.build_csr(n, u, v)
    maxdeg = int(csr.degrees().max())
    b = O.sample_blocks(csr, np.arange(n, dtype=np.int32), [maxdeg, maxdeg + 3], 1)
    assert b.sizes == [n, n, n]
    for h in range(2):
        assert np.array_equal(b.indptr[h], csr.row_ptr.astype(np.int32))
        assert np.array_equal(b.indices[h], csr.col)
        assert np.array_equal(b.nbrs[h], csr.col)


def test_blocks_bad_seed():
    csr = O.build_csr(4, [0, 1], [1, 2])
    with pytest.raises(ValueError):
        O.sample_blocks(csr, [0, 4], [2], 1)


# --------------------------------------------------------- gather, O7 -----

def test_gather_rows_and_counts():
    n, u, v = W.random_graph(n=200, m=1500, seed=2)
    csr = O.build_csr(n, u, v)
    feats = W.features(n, 7, "f32", seed=5)
    _, slot, c = O.rank_cache(csr, 0.3)
    ids = np.array([3, 3, 199, 0, 250, -1, 17], np.int32)
    rows, counts = O.gather(feats, slot, ids)
    for i, x in enumerate(ids.tolist()):
        if 0 <= x < n:
            assert rows[i].tobytes() == feats[x].tobytes()
        else:
            assert not rows[i].any()
    valid = [x for x in ids.tolist() if 0 <= x < n]
    assert counts.tolist() == [sum(slot[x] >= 0 for x in valid),
                               sum(slot[x] < 0 for x in valid), 2]


def test_gather_closed_form_hits():
    """Seeds = V, k >= max degree: gathering N_1 hits sum of degrees of the top C."""
    n, u, v = W.random_graph(n=300, m=2500, seed=6)
    csr = O.build_csr(n, u, v)
    deg = csr.degrees()
    maxdeg = int(deg.max())
    b = O.sample_blocks(csr, np.arange(n, dtype=np.int32), [maxdeg], 3)
    feats = W.features(n, 4, "bf16", seed=1)
    prev = -1
    for r in [0.0, 0.1, 0.25, 0.5, 1.0]:
        rank, slot, c = O.rank_cache(csr, r)
        _, counts = O.gather(feats, slot, b.nbrs[0])
        assert counts[0] == int(deg[rank[:c]].sum())
        assert counts[0] + counts[1] == csr.nnz
        assert counts[0] >= prev
        prev = counts[0]
    assert prev == csr.nnz


# ------------------------------------------------------------ bf16 RNE ----

def test_round_bf16_special_cases():
    r = O.round_bf16
    assert r(1.0) == 1.0
    assert r(1.0 + 2**-8) == 1.0                       # tie, even below
    assert r(1.0 + 3 * 2**-8) == 1.0 + 2**-6           # tie, even above
    assert r(1.0 + 2**-8 + 2**-40) == 1.0 + 2**-7      # not a tie in double
    assert r(-(1.0 + 3 * 2**-8)) == -(1.0 + 2**-6)
    mx = (2 - 2**-7) * 2.0**127
    assert r(mx) == mx
    assert r(mx * (1 + 2**-9)) == mx
    assert math.isinf(r((2 - 2**-8) * 2.0**127))       # overflow threshold
    assert math.isinf(r(1e300)) and r(-1e300) < 0
    assert r(2.0**-133) == 2.0**-133                   # smallest subnormal
    assert r(2.0**-134) == 0.0                         # tie to even (zero)
    assert r(3 * 2.0**-134) == 2.0**-132               # tie to even (2 ulps)
    assert math.isnan(r(float("nan")))
    assert r(0.0) == 0.0 and math.copysign(1, r(-0.0)) < 0


def test_round_bf16_matches_library_cast():
    """For every float32 exponent/mantissa-high pattern and every rounding
    class of the low half, the oracle equals torch's float32 -> bfloat16."""
    torch = pytest.importorskip("torch")
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xC000, 0xFFFF], np.uint32)
    bits = (hi[:, None] | lows[None, :]).ravel()
    rng = np.random.default_rng(0)
    bits = np.concatenate([bits, rng.integers(0, 1 << 32, 2_000_000, dtype=np.uint64).astype(np.uint32)])
    f = bits.view(np.float32)
    ours = O.round_bf16_array(f.astype(np.float64))
    lib = torch.from_numpy(f.copy()).to(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(f)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], lib[~nan])


# --------------------------------------------------- SAGE forward, O8 -----

def _dense_layer(indptr, indices, X, Wt, relu):
    """Dense brute force: A_mean (n_dst x n_src) @ X, then [X_dst | agg] @ W."""
    n_dst = indptr.size - 1
    A = np.zeros((n_dst, X.shape[0]))
    for i in range(n_dst):
        cnt = indptr[i + 1] - indptr[i]
        for p in range(indptr[i], indptr[i + 1]):
            A[i, indices[p]] += 1.0 / cnt
    agg = A @ X
    z = np.concatenate([X[:n_dst], agg], axis=1) @ Wt
    return (np.maximum(z, 0) if relu else z), agg


@pytest.mark.parametrize("seed", range(3))
def test_sage_forward_dense_brute_force(seed):
    n, u, v = W.random_graph(n=120, m=500, seed=seed)
    csr = O.build_csr(n, u, v)
    b = O.sample_blocks(csr, np.arange(0, n, 9, dtype=np.int32), [4, 3], 55 + seed)
    dims = [5, 6, 3]
    feats = W.features(n, dims[0], "f32", seed=seed)
    H0 = O.to_f64(feats[b.nodes], "f32")
    Ws = [O.to_f64(W.glorot(dims[l], dims[l + 1], "f32", seed + l), "f32") for l in range(2)]
    got, trace = O.sage_forward(b, H0, Ws, keep=True)
    X = H0
    for l in range(1, 3):
        hb = 2 - l + 1
        X, agg = _dense_layer(b.indptr[hb - 1], b.indices[hb - 1], X, Ws[l - 1], relu=l < 2)
        np.testing.assert_allclose(trace[l - 1][0], agg, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(got, X, rtol=1e-12, atol=1e-12)


def test_sage_full_neighbourhood_is_DinvAX():
    """Seeds = V and k >= max degree: aggregation is D^-1 A X (zero rows for isolated)."""
    n, u, v = W.tiny_graph("isolated")
    csr = O.build_csr(n, u, v)
    b = O.sample_blocks(csr, np.arange(n, dtype=np.int32), [50], 1)
    X = np.random.default_rng(1).standard_normal((n, 4))
    Wt = np.concatenate([np.zeros((4, 4)), np.eye(4)])   # passes the aggregate
    out = O.sage_layer(b.indptr[0], b.indices[0], X, Wt, relu=False, bf16=False, round_out=False)
    A = np.zeros((n, n))
    for x in range(n):
        for y in csr.col[csr.row_ptr[x]:csr.row_ptr[x + 1]]:
            A[x, y] = 1
    deg = A.sum(1)
    expect = np.divide(A @ X, deg[:, None], out=np.zeros_like(X), where=deg[:, None] > 0)
    np.testing.assert_allclose(out, expect, rtol=1e-13, atol=0)
    assert not out[10:].any()                          # isolated nodes -> zero rows


def test_sage_combine_identities_and_linearity():
    n, u, v = W.random_graph(n=50, m=300, seed=8)
    csr = O.build_csr(n, u, v)
    b = O.sample_blocks(csr, np.arange(0, n, 3, dtype=np.int32), [1], 9)
    X = np.random.default_rng(2).standard_normal((b.sizes[1], 6))
    ip, ix = b.indptr[0], b.indices[0]
    I, Z = np.eye(6), np.zeros((6, 6))
    self_pass = O.sage_layer(ip, ix, X, np.concatenate([I, Z]), False, False, False)
    np.testing.assert_array_equal(self_pass, X[:ip.size - 1])
    agg_pass = O.sage_layer(ip, ix, X, np.concatenate([Z, I]), False, False, False)
    for i in range(ip.size - 1):                        # k = 1 copies one row exactly
        if ip[i + 1] > ip[i]:
            np.testing.assert_array_equal(agg_pass[i], X[ix[ip[i]]])
        else:
            assert not agg_pass[i].any()
    W1 = np.random.default_rng(3).standard_normal((12, 4))
    W2 = np.random.default_rng(4).standard_normal((12, 4))
    a = O.sage_layer(ip, ix, X, W1, False, False, False)
    c = O.sage_layer(ip, ix, X, W2, False, False, False)
    s = O.sage_layer(ip, ix, X, 2 * W1 - W2, False, False, False)
    np.testing.assert_allclose(s, 2 * a - c, rtol=1e-12, atol=1e-12)
    r = O.sage_layer(ip, ix, X, W1, True, False, False)
    np.testing.assert_array_equal(r, np.maximum(a, 0))


def test_sage_bf16_rounding_points():
    """bf16 mode rounds the aggregate and the hidden output, not the logits."""
    n, u, v = W.random_graph(n=80, m=400, seed=12)
    csr = O.build_csr(n, u, v)
    b = O.sample_blocks(csr, np.arange(0, n, 4, dtype=np.int32), [3], 2)
    X = O.to_f64(W.features(b.sizes[1], 8, "bf16", seed=3), "bf16")
    Wt = O.to_f64(W.glorot(8, 5, "bf16", 1), "bf16")
    ip, ix = b.indptr[0], b.indices[0]
    z, agg = O.sage_layer(ip, ix, X, Wt, relu=True, bf16=True, round_out=True, want_agg=True)
    np.testing.assert_array_equal(agg, O.round_bf16_array(agg))
    np.testing.assert_array_equal(z, O.round_bf16_array(z))
    z64, agg64 = O.sage_layer(ip, ix, X, Wt, relu=True, bf16=False, round_out=False, want_agg=True)
    np.testing.assert_array_equal(agg, O.round_bf16_array(agg64))
    logits = O.sage_layer(ip, ix, X, Wt, relu=False, bf16=True, round_out=False)
    expect = np.concatenate([X[:ip.size - 1], agg], axis=1) @ Wt
    np.testing.assert_allclose(logits, expect, rtol=1e-12, atol=1e-12)


def test_sage_rows_subset_matches_full():
    n, u, v = W.random_graph(n=100, m=600, seed=13)
    csr = O.build_csr(n, u, v)
    b = O.sample_blocks(csr, np.arange(0, n, 2, dtype=np.int32), [5], 4)
    X = np.random.default_rng(5).standard_normal((b.sizes[1], 7))
    Wt = np.random.default_rng(6).standard_normal((14, 3))
    full = O.sage_layer(b.indptr[0], b.indices[0], X, Wt, True, False, False)
    rows = np.array([0, 7, 3, 49], np.int64)
    part = O.sage_layer(b.indptr[0], b.indices[0], X, Wt, True, False, False, rows=rows)
    np.testing.assert_array_equal(part, full[rows])


@pytest.mark.parametrize("bf16", [False, True])
def test_forward_rows_matches_full_forward(bf16):
    """The receptive-field forward equals the full forward on the rows asked for."""
    n, u, v = W.random_graph(n=400, m=3000, seed=17)
    csr = O.build_csr(n, u, v)
    b = O.sample_blocks(csr, np.arange(0, n, 5, dtype=np.int32), [4, 3, 2], 21)
    dt = "bf16" if bf16 else "f32"
    dims = [6, 5, 4, 3]
    H0 = O.to_f64(W.features(b.sizes[3], dims[0], dt, seed=2), dt)
    Ws = [O.to_f64(W.glorot(dims[l], dims[l + 1], dt, seed=l), dt) for l in range(3)]
    full = O.sage_forward(b, H0, Ws, bf16=bf16)
    rows = np.array([7, 0, 79, 33, 7], np.int64)
    part = O.sage_forward_rows(b, H0, Ws, rows, bf16=bf16)
    np.testing.assert_array_equal(part, full[rows])


# ------------------------------------------------- FIFO cache update, O7 --

def _deque_fifo(rank, c, ring_n, batches, n):
    """Independent FIFO model: a deque of (slot, vertex) plus a set lookup."""
    from collections import deque
    static = set(int(x) for x in rank[:c - ring_n])
    ring = deque(int(x) for x in rank[c - ring_n:c])     # oldest first
    hist = []
    for ids in batches:
        cached = static | set(ring)
        misses = [int(v) for v in ids if 0 <= v < n and int(v) not in cached]
        hits = sum(1 for v in ids if 0 <= v < n and int(v) in cached)
        hist.append((hits, len(misses)))
        for v in misses:
            if ring_n:
                ring.popleft()
                ring.append(v)
    return hist, static | set(ring)


@pytest.mark.parametrize("r,frac", [(0.1, 1.0), (0.2, 0.5), (0.05, 0.25), (0.3, 0.0)])
def test_fifo_cache_matches_deque_model(r, frac):
    n, u, v = W.random_graph(n=600, m=5000, seed=31)
    csr = O.build_csr(n, u, v)
    rank, _, c = O.rank_cache(csr, r)
    ring_n = int(c * frac)
    rng = np.random.default_rng(7)
    batches = [np.unique(rng.integers(0, n, 120)).astype(np.int32)[rng.permutation(0)] if False else
               rng.permutation(np.unique(rng.integers(0, n, 120))).astype(np.int32) for _ in range(8)]
    feats = W.features(n, 3, "f32", seed=1)
    cache = O.FifoCache(csr, r, ring_n)
    got = []
    for ids in batches:
        rows, counts = cache.gather(feats, ids)
        got.append((int(counts[0]), int(counts[1])))
        assert rows.tobytes() == feats[ids].tobytes()
    hist, final = _deque_fifo(rank, c, ring_n, batches, n)
    assert got == hist
    cached = {int(x) for x in np.nonzero(cache.slot_map >= 0)[0]}
    assert cached == final
    # owner <-> slot_map bijection
    for s, x in enumerate(cache.owner):
        assert x >= 0 and cache.slot_map[x] == s
    assert (cache.slot_map >= 0).sum() == c


@pytest.mark.parametrize("r,frac", [(0.1, 1.0), (0.2, 0.5), (0.05, 0.1)])
def test_fifo_cache_repeated_ids_match_deque_model(r, frac):
    """Batches that request some vertices several times: each request that
    misses is admitted, so a repeated vertex takes two ring slots; the vertex
    stays cached while any of its copies is in the ring (the deque model's
    set semantics), and every mapped vertex's slot holds that vertex."""
    n, u, v = W.random_graph(n=500, m=4000, seed=33)
    csr = O.build_csr(n, u, v)
    rank, _, c = O.rank_cache(csr, r)
    ring_n = max(1, int(c * frac))
    rng = np.random.default_rng(8)
    batches = []
    for _ in range(10):
        ids = rng.integers(0, n, 90).astype(np.int32)
        ids[rng.integers(0, 90, 20)] = ids[rng.integers(0, 90, 20)]   # plant repeats
        batches.append(ids)
    assert any(np.unique(b).size < b.size for b in batches)
    feats = W.features(n, 3, "f32", seed=4)
    cache = O.FifoCache(csr, r, ring_n)
    got = []
    for ids in batches:
        rows, counts = cache.gather(feats, ids)
        got.append((int(counts[0]), int(counts[1])))
        assert rows.tobytes() == feats[ids].tobytes()
    hist, final = _deque_fifo(rank, c, ring_n, batches, n)
    assert got == hist
    assert {int(x) for x in np.nonzero(cache.slot_map >= 0)[0]} == final
    for x in np.nonzero(cache.slot_map >= 0)[0]:
        assert cache.owner[cache.slot_map[x]] == x


def test_fifo_cache_repeat_batch_hits():
    """A batch of m <= ring uncached vertices is fully cached after one pass:
    repeating it right away hits every request."""
    n, u, v = W.random_graph(n=400, m=3000, seed=32)
    csr = O.build_csr(n, u, v)
    feats = W.features(n, 2, "f32", seed=2)
    cache = O.FifoCache(csr, 0.5, ring_n=120)
    cold = np.nonzero(cache.slot_map < 0)[0]
    ids = np.random.default_rng(3).permutation(cold)[:100].astype(np.int32)
    _, c1 = cache.gather(feats, ids)
    _, c2 = cache.gather(feats, ids)
    assert c1.tolist() == [0, 100, 0]
    assert c2.tolist() == [100, 0, 0]
    # the 20 oldest ring entries survived; the first 100 were replaced in order
    ring = cache.owner[cache.c - 120:]
    assert ring[:100].tolist() == ids.tolist()


# -------------------------------------------------- LRU cache update, O7 --

def _hub_graph(n, hubs):
    """Vertices `hubs` joined to every other vertex, nothing else: the hubs
    rank first (ties by id), so they are the cache's initial contents."""
    u = [h for h in hubs for x in range(n) if x not in hubs]
    v = [x for h in hubs for x in range(n) if x not in hubs]
    return O.build_csr(n, u, v)


def _faults(cache, refs, n):
    feats = W.features(n, 2, "f32", seed=0)
    misses = 0
    for x in refs:
        _, counts = cache.gather(feats, np.array([x], np.int32))
        misses += int(counts[1])
    return misses


# Page-replacement textbook values (one request per batch, frames = ring
# slots, the ring's initial vertices never requested, so it starts "empty"):
#   Silberschatz, Galvin, Gagne, Operating System Concepts, ch. "Virtual
#   Memory": reference string 7 0 1 2 0 3 0 4 2 3 0 3 2 1 2 0 1 7 0 1 with 3
#   frames gives 15 faults under FIFO and 12 under LRU;
#   Belady, Nelson, Shedler, CACM 12(6) 1969: 1 2 3 4 1 2 5 1 2 3 4 5 gives 9
#   FIFO faults with 3 frames and 10 with 4 (Belady's anomaly); LRU, a stack
#   algorithm (Mattson et al., IBM Syst. J. 9(2) 1970), gives 10 and 8.
_SILBERSCHATZ = [7, 0, 1, 2, 0, 3, 0, 4, 2, 3, 0, 3, 2, 1, 2, 0, 1, 7, 0, 1]
_BELADY = [1, 2, 3, 4, 1, 2, 5, 1, 2, 3, 4, 5]


@pytest.mark.parametrize("refs,frames,fifo,lru", [(_SILBERSCHATZ, 3, 15, 12), (_BELADY, 3, 9, 10),
                                                  (_BELADY, 4, 10, 8)])
def test_cache_policies_textbook_fault_counts(refs, frames, fifo, lru):
    n = 20
    csr = _hub_graph(n, list(range(n - frames, n)))
    r = (frames + 0.5) / n
    f, l = O.FifoCache(csr, r, frames), O.LruCache(csr, r, frames)
    assert f.c == frames and sorted(f.owner.tolist()) == list(range(n - frames, n))
    assert _faults(f, refs, n) == fifo
    assert _faults(l, refs, n) == lru


def test_lru_cache_worked_batches():
    """Three multi-request batches on a ring of 4 slots, worked by hand.
    Slots 0..3 start with A..D = vertices 16..19, least recent first.
      batch [C, X, A, Y]: C, A hit; recency 1 3 0 2 (untouched B, D first,
        then the hit slots in their earlier order); X takes slot 1 (B out),
        Y slot 3 (D out); recency 0 2 1 3.
      batch [Z, D, B, W, V]: five misses for four slots: Z -> 0 (A out),
        D -> 2 (C out), B -> 1 (X out), W -> 3 (Y out), V -> 0 (Z out);
        recency 2 1 3 0.
      batch [W, Q, B]: W, B hit; recency 2 0 1 3; Q takes slot 2 (D out);
        recency 0 1 3 2."""
    n = 20
    csr = _hub_graph(n, [16, 17, 18, 19])
    A, B, C, D = 16, 17, 18, 19
    X, Y, Z, Wv, V, Q = 1, 2, 3, 4, 5, 6
    cache = O.LruCache(csr, 0.2, 4)
    feats = W.features(n, 3, "f32", seed=5)
    steps = [([C, X, A, Y], [2, 2, 0], [A, X, C, Y], [0, 2, 1, 3]),
             ([Z, D, B, Wv, V], [0, 5, 0], [V, B, D, Wv], [2, 1, 3, 0]),
             ([Wv, Q, B], [2, 1, 0], [V, B, Q, Wv], [0, 1, 3, 2])]
    for ids, counts, owners, recency in steps:
        rows, got = cache.gather(feats, np.array(ids, np.int32))
        assert rows.tobytes() == feats[ids].tobytes()
        assert got.tolist() == counts
        assert cache.owner.tolist() == owners
        assert cache.recency().tolist() == recency
        for s, x in enumerate(owners):
            assert cache.slot_map[x] == s
        assert (cache.slot_map >= 0).sum() == 4
    assert cache.slot_map[[A, C, X, Y, Z, D]].tolist() == [-1] * 6


def test_lru_cache_repeated_miss_keeps_later_copy():
    """A vertex missed twice in one batch takes two slots and stays mapped to
    the later one; evicting the earlier (stale) copy must not unmap it.
    Ring of 3 slots holding hubs 17, 18, 19 (least recent first):
      [X, X]: X -> slot 0, X -> slot 1 (mapped); recency 2 0 1.
      [Y]: Y -> slot 2 (19 out); recency 0 1 2.
      [Z]: Z -> slot 0, whose stale X copy goes; X stays mapped to slot 1;
        recency 1 2 0.
      [X]: a hit on slot 1; recency 2 0 1."""
    n = 20
    csr = _hub_graph(n, [17, 18, 19])
    X, Y, Z = 3, 4, 5
    cache = O.LruCache(csr, 3.5 / n, 3)
    feats = W.features(n, 2, "f32", seed=7)
    steps = [([X, X], [0, 2, 0], [X, X, 19], 1), ([Y], [0, 1, 0], [X, X, Y], 1), ([Z], [0, 1, 0], [Z, X, Y], 1),
             ([X], [1, 0, 0], [Z, X, Y], 1)]
    for ids, counts, owners, x_slot in steps:
        _, got = cache.gather(feats, np.array(ids, np.int32))
        assert got.tolist() == counts
        assert cache.owner.tolist() == owners
        assert cache.slot_map[X] == x_slot
    assert cache.recency().tolist() == [2, 0, 1]


def _list_lru(rank, c, ring_n, batches, n):
    """Independent LRU model: a Python list of [slot, vertex] pairs, least
    recent first, and a dict of the mapped ring vertices."""
    lo = c - ring_n
    static = set(int(x) for x in rank[:lo])
    ring = [[lo + j, int(rank[lo + j])] for j in range(ring_n)]
    mapped = {v: s for s, v in ring}
    hist, ring_hits = [], 0
    for ids in batches:
        cached = static | set(mapped)
        req = [int(v) for v in ids if 0 <= v < n]
        hits = [v for v in req if v in cached]
        misses = [v for v in req if v not in cached]
        hist.append((len(hits), len(misses)))
        touched = {mapped[v] for v in hits if v in mapped}
        ring_hits += len(touched)
        ring = [e for e in ring if e[0] not in touched] + [e for e in ring if e[0] in touched]
        for v in misses:
            if not ring:
                break
            s, old = ring.pop(0)
            if mapped.get(old) == s:
                del mapped[old]
            mapped[v] = s
            ring.append([s, v])
    return hist, static | set(mapped), [s for s, _ in ring], ring_hits


@pytest.mark.parametrize("r,frac,repeats", [(0.1, 1.0, False), (0.2, 0.5, False), (0.05, 0.25, True),
                                            (0.3, 0.0, False), (0.1, 0.1, True), (0.3, 1.0, True)])
def test_lru_cache_matches_list_model(r, frac, repeats):
    """Batches drawn with a hot set (so ring slots are hit again), some with
    repeated vertices and with out-of-range ids."""
    n, u, v = W.random_graph(n=600, m=5000, seed=35)
    csr = O.build_csr(n, u, v)
    rank, _, c = O.rank_cache(csr, r)
    ring_n = int(c * frac)
    rng = np.random.default_rng(9)
    hot = rng.choice(n, 80, replace=False)
    batches = []
    for _ in range(12):
        ids = np.concatenate([rng.choice(hot, 40), rng.integers(0, n, 60)]).astype(np.int32)
        if not repeats:
            ids = np.unique(ids)
        ids = rng.permutation(ids)
        ids[rng.integers(0, ids.size, 2)] = [-1, n]
        batches.append(ids)
    feats = W.features(n, 3, "f32", seed=6)
    cache = O.LruCache(csr, r, ring_n)
    got = []
    for ids in batches:
        rows, counts = cache.gather(feats, ids)
        got.append((int(counts[0]), int(counts[1])))
    hist, final, recency, ring_hits = _list_lru(rank, c, ring_n, batches, n)
    assert got == hist
    assert (ring_hits > 0) == (frac > 0)    # the recency reorder is exercised
    assert {int(x) for x in np.nonzero(cache.slot_map >= 0)[0]} == final
    assert cache.recency().tolist() == recency
    for x in np.nonzero(cache.slot_map >= 0)[0]:
        assert cache.owner[cache.slot_map[x]] == x


def test_lru_without_ring_hits_is_fifo():
    """Batches of vertices never cached before, so no request hits the ring:
    LRU then admits exactly as FIFO does."""
    n, u, v = W.random_graph(n=500, m=4000, seed=36)
    csr = O.build_csr(n, u, v)
    f, l = O.FifoCache(csr, 0.2, 60), O.LruCache(csr, 0.2, 60)
    cold = np.random.default_rng(4).permutation(np.nonzero(f.slot_map < 0)[0]).astype(np.int32)
    feats = W.features(n, 2, "f32", seed=3)
    for ids in np.array_split(cold[:350], 7):   # 50 a batch: older admissions are gone before reuse
        _, cf = f.gather(feats, ids)
        _, cl = l.gather(feats, ids)
        assert cf.tolist() == cl.tolist() == [0, ids.size, 0]
        assert f.owner.tolist() == l.owner.tolist()
        assert f.slot_map.tolist() == l.slot_map.tolist()


# ------------------------------------------- loss, backward, update ---

def _loss_of(blocks, H0, Ws, y):
    logits = O.sage_forward(blocks, H0, Ws)
    return O.softmax_xent(logits, y)[0]


def test_softmax_xent_closed_forms():
    """Uniform logits give log C; the gradient rows sum to zero and equal
    (1/C - onehot)/n; a shift of every logit in a row changes nothing."""
    C, n = 7, 5
    y = np.array([0, 6, 3, 3, 1])
    loss, dZ = O.softmax_xent(np.zeros((n, C)), y)
    assert loss == pytest.approx(math.log(C), abs=1e-15)
    want = np.full((n, C), 1.0 / C)
    want[np.arange(n), y] -= 1.0
    assert np.allclose(dZ, want / n, atol=1e-15)
    rng = np.random.default_rng(0)
    Z = rng.normal(size=(n, C)) * 4
    l1, g1 = O.softmax_xent(Z, y)
    l2, g2 = O.softmax_xent(Z + rng.normal(size=(n, 1)) * 50, y)
    assert l1 == pytest.approx(l2, rel=1e-12)
    assert np.allclose(g1, g2, atol=1e-14)
    assert np.allclose(g1.sum(axis=1), 0, atol=1e-15)
    # a one-row, two-class case by hand: loss = log(1 + e^(z1 - z0))
    l, g = O.softmax_xent(np.array([[0.3, -1.2]]), [0])
    assert l == pytest.approx(math.log1p(math.exp(-1.5)), rel=1e-14)
    assert g[0, 1] == pytest.approx(1 / (1 + math.exp(1.5)), rel=1e-14)


def test_softmax_xent_finite_difference():
    rng = np.random.default_rng(1)
    Z = rng.normal(size=(6, 5)) * 3
    y = rng.integers(0, 5, 6)
    _, g = O.softmax_xent(Z, y)
    eps = 1e-6
    for i, c in itertools.product(range(6), range(5)):
        Zp, Zm = Z.copy(), Z.copy()
        Zp[i, c] += eps
        Zm[i, c] -= eps
        fd = (O.softmax_xent(Zp, y)[0] - O.softmax_xent(Zm, y)[0]) / (2 * eps)
        assert fd == pytest.approx(g[i, c], abs=1e-9)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_aggregate_mean_t_is_the_adjoint(seed):
    """<agg(X), G> = <X, agg^T(G)>, with agg taken from the C forward
    (the W = [0; I] pass-through of sage_layer)."""
    n, u, v = W.random_graph(300, 1500, seed)
    csr = O.build_csr(n, u, v)
    seeds = np.arange(0, n, 7, dtype=np.int32)
    blk = O.sample_blocks(csr, seeds, [4], 11 + seed)
    ip, ix = blk.indptr[0], blk.indices[0]
    rng = np.random.default_rng(seed)
    d = 5
    X = rng.normal(size=(blk.sizes[1], d))
    G = rng.normal(size=(blk.sizes[0], d))
    Wpass = np.concatenate([np.zeros((d, d)), np.eye(d)])
    agg = O.sage_layer(ip, ix, X, Wpass, relu=False, bf16=False, round_out=False)
    lhs = float((agg * G).sum())
    rhs = float((X * O.aggregate_mean_t(ip, ix, X.shape[0], G)).sum())
    assert lhs == pytest.approx(rhs, rel=1e-12)
    # isolated destination rows (no edges) send nothing back
    dX = O.aggregate_mean_t([0, 0, 2], [1, 1], 3, np.ones((2, 1)))
    assert dX.ravel().tolist() == [0.0, 1.0, 0.0]


@pytest.mark.parametrize("fanouts,dims", [([3, 2], [4, 6, 3]), ([2, 3, 2], [3, 5, 4, 4])])
def test_sage_backward_finite_difference(fanouts, dims):
    """Every weight gradient against central differences of the loss of the
    full forward (float64, ReLU kinks are measure-zero for random data)."""
    n, u, v = W.random_graph(80, 300, 5)
    csr = O.build_csr(n, u, v)
    seeds = np.array([3, 17, 40, 41, 77], np.int32)
    blk = O.sample_blocks(csr, seeds, fanouts, 99)
    rng = np.random.default_rng(7)
    H0 = rng.normal(size=(blk.sizes[-1], dims[0]))
    Ws = [rng.normal(size=(2 * dims[l], dims[l + 1])) * 0.7 for l in range(len(fanouts))]
    y = rng.integers(0, dims[-1], blk.sizes[0])
    logits, trace = O.sage_forward(blk, H0, Ws, keep=True)
    _, dZ = O.softmax_xent(logits, y)
    dWs = O.sage_backward(blk, H0, Ws, trace, dZ)
    eps = 1e-6
    for l, Wl in enumerate(Ws):
        assert dWs[l].shape == Wl.shape
        for a, o in itertools.product(range(Wl.shape[0]), range(Wl.shape[1])):
            Wp = [w.copy() for w in Ws]
            Wm = [w.copy() for w in Ws]
            Wp[l][a, o] += eps
            Wm[l][a, o] -= eps
            fd = (_loss_of(blk, H0, Wp, y) - _loss_of(blk, H0, Wm, y)) / (2 * eps)
            assert fd == pytest.approx(dWs[l][a, o], abs=1e-7), (l, a, o)


def test_train_step_decreases_loss_and_applies_sgd():
    n, u, v = W.random_graph(200, 900, 3)
    csr = O.build_csr(n, u, v)
    blk = O.sample_blocks(csr, np.arange(0, 200, 9, dtype=np.int32), [4, 3], 5)
    rng = np.random.default_rng(2)
    dims = [6, 8, 4]
    H0 = rng.normal(size=(blk.sizes[-1], dims[0]))
    Ws = [rng.normal(size=(2 * dims[l], dims[l + 1])) * 0.5 for l in range(2)]
    y = rng.integers(0, 4, blk.sizes[0])
    lr = 0.05
    loss, _, dWs, new = O.train_step(blk, H0, Ws, y, lr)
    for w, g, w2 in zip(Ws, dWs, new):
        assert np.array_equal(w2, w - lr * g)
    # a small step along the negative gradient lowers the loss
    assert _loss_of(blk, H0, new, y) < loss


# ------------------------------------------- locality-biased selection ---

def _exact_successive(weights, k):
    """Probability of every k-subset under successive sampling without
    replacement (each pick proportional to weight among those left), by
    enumerating the ordered pick sequences."""
    idx = range(len(weights))
    probs = {}
    for seq in itertools.permutations(idx, k):
        p, left = 1.0, float(sum(weights))
        for i in seq:
            p *= weights[i] / left
            left -= weights[i]
        key = frozenset(seq)
        probs[key] = probs.get(key, 0.0) + p
    return probs


def _chi2_against(csr, hub, slot, eta, k, probs, trials, hop=0):
    counts = {s: 0 for s in probs}
    for t in range(trials):
        s = O.sample_node_biased(csr, hub, k, (321 << 32) | t, hop, slot, eta)
        counts[frozenset(s.tolist())] += 1
    return sum((counts[s] - trials * p) ** 2 / (trials * p) for s, p in probs.items())


@pytest.mark.parametrize("eta,k,cached", [(1, 3, {1, 4}), (3, 2, {2, 5}), (5, 3, {1, 2, 3}), (40, 2, {6})])
def test_biased_selection_is_weighted_successive_sampling(eta, k, cached):
    """Subset frequencies of the biased selector against the exact
    probabilities of successive weighted sampling (eta = 1: uniform)."""
    csr = _star(7)                               # hub 0, neighbours 1..6
    slot = np.full(7, -1, np.int32)
    for v in cached:
        slot[v] = 0
    weights = [eta if v in cached else 1 for v in range(1, 7)]
    probs = {frozenset(v + 1 for v in s): p for s, p in _exact_successive(weights, k).items()}
    trials = 30000
    chi2 = _chi2_against(csr, 0, slot, eta, k, probs, trials)
    dof = len(probs) - 1
    # P(chi2 > dof + 6 sqrt(2 dof) + 10) is below 1e-4 for these dof
    assert chi2 < dof + 6 * math.sqrt(2 * dof) + 10, (chi2, dof)
    if eta == 1:
        assert all(abs(p - 1 / len(probs)) < 1e-12 for p in probs.values())


def test_biased_selection_properties():
    n, u, v = W.random_graph(n=80, m=900, seed=3)
    csr = O.build_csr(n, u, v)
    _, slot, _ = O.rank_cache(csr, 0.3)
    for node in range(n):
        row = csr.col[csr.row_ptr[node]:csr.row_ptr[node + 1]]
        for k, eta in itertools.product([0, 1, 4, 9, 64, -1], [1, 7, 65536]):
            s = O.sample_node_biased(csr, node, k, 55, 2, slot, eta)
            want = len(row) if k < 0 else min(len(row), k)
            assert s.size == want
            assert len(set(s.tolist())) == s.size
            assert set(s.tolist()) <= set(row.tolist())
            if k < 0 or len(row) <= k:
                assert s.tolist() == row.tolist()
            else:
                flags = (slot[s] >= 0).tolist()
                assert flags == sorted(flags, reverse=True), "cached picks come first"
            assert np.array_equal(s, O.sample_node_biased(csr, node, k, 55, 2, slot, eta))


def test_biased_selection_strong_bias_takes_cached():
    """With eta = 65536 and at least k cached neighbours, an uncached pick
    needs a class draw below u / (eta c + u): rare."""
    csr = _star(101)
    slot = np.full(101, -1, np.int32)
    slot[1:31] = np.arange(30)                   # 30 of 100 neighbours cached
    k, trials, uncached = 10, 2000, 0
    for t in range(trials):
        s = O.sample_node_biased(csr, 0, k, t, 1, slot, 65536)
        uncached += int((slot[s] < 0).sum())
    # expected uncached picks per trial is about k * 70 / (65536 * 21) ~ 5e-4
    assert uncached <= 10


def test_below64_exact():
    rng = np.random.default_rng(4)
    for _ in range(2000):
        x = int(rng.integers(0, 2 ** 32))
        b = int(rng.integers(1, 2 ** 63))
        assert O.below64(x, b) == (x * b) >> 32
    assert O.below64(2 ** 32 - 1, 2 ** 48) == ((2 ** 32 - 1) * 2 ** 48) >> 32


def test_biased_blocks_consistent():
    n, u, v = W.random_graph(n=400, m=5000, seed=6)
    csr = O.build_csr(n, u, v)
    _, slot, _ = O.rank_cache(csr, 0.25)
    seeds = W.epoch_permutation(n)[:40]
    blk = O.sample_blocks(csr, seeds, [5, 4], 9, bias_slot_map=slot, eta=8)
    for h in range(2):
        ip, nb, ix = blk.indptr[h], blk.nbrs[h], blk.indices[h]
        assert np.array_equal(blk.nodes[ix], nb)
        for i in range(blk.sizes[h]):
            node = blk.nodes[i]
            want = O.sample_node_biased(csr, int(node), [5, 4][h], 9, h, slot, 8)
            assert np.array_equal(nb[ip[i]:ip[i + 1]], want)
    # the bias raises the share of sampled edges that land on cached vertices
    plain = O.sample_blocks(csr, seeds, [5, 4], 9)
    share = lambda b: np.mean(np.concatenate([slot[x] >= 0 for x in b.nbrs]))
    assert share(blk) > share(plain)
