"""Python face of the CPU oracle (TEST INFRASTRUCTURE ONLY).

The oracle is the plain, slow, single-threaded C definition in oracle.c of
what the sampled mini-batch step computes (Algorithm 1's forward, Eq. 1,
Eq. 2 and the static device cache of Section 3.2 of GNNavigator).  Only
``tests/``, ``__graft_entry__.smoke()`` and the bench's ``cpu_baseline`` leg
may import this package.  The HIP library never imports it, and it never
imports the HIP library: the two share no code.

All functions take and return numpy arrays.  Floating-point results are
float64.  Feature / weight inputs in bfloat16 are passed as uint16 bit
patterns and widened exactly to float64 here.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into oracle/liboracle.so with gcc."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-Wall", "-fPIC", "-shared", "-o", tmp,
                               os.path.join(_HERE, "oracle.c"), "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    src = os.path.join(_HERE, "oracle.c")
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(src) > os.path.getmtime(_LIB_PATH):
        build(force=True)
    lib = C.CDLL(_LIB_PATH)
    P, i64, i32, u32, u64, f64 = C.c_void_p, C.c_int64, C.c_int32, C.c_uint32, C.c_uint64, C.c_double
    lib.oracle_build_csr.argtypes = [i64, i64, P, P, i32, P, P]
    lib.oracle_build_csr.restype = i64
    lib.oracle_rank_cache.argtypes = [i64, P, f64, P, P]
    lib.oracle_rank_cache.restype = i64
    lib.oracle_philox4x32_10.argtypes = [P, P, P]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_draw.argtypes = [u64, u32, i64, u32]
    lib.oracle_draw.restype = u32
    lib.oracle_below.argtypes = [u32, u32]
    lib.oracle_below.restype = u32
    lib.oracle_sample_node.argtypes = [P, P, i64, i32, u64, u32, P]
    lib.oracle_sample_node.restype = i64
    lib.oracle_sample_blocks.argtypes = [i64, P, P, P, i64, P, i32, u64, P, u32, P, P, P, P, P]
    lib.oracle_sample_node_biased.argtypes = [P, P, i64, i32, u64, u32, P, u32, P]
    lib.oracle_sample_node_biased.restype = i64
    lib.oracle_below64.argtypes = [u32, u64]
    lib.oracle_below64.restype = u64
    lib.oracle_sample_blocks.restype = i32
    lib.oracle_gather.argtypes = [i64, P, i64, P, P, i64, P, P, P]
    lib.oracle_gather.restype = None
    lib.oracle_cache_fifo_admit.argtypes = [P, P, i64, i64, P, P, i64]
    lib.oracle_cache_fifo_admit.restype = None
    lib.oracle_cache_lru_update.argtypes = [P, P, i64, i64, P, P, P, i64, P, i64]
    lib.oracle_cache_lru_update.restype = None
    lib.oracle_round_bf16.argtypes = [f64]
    lib.oracle_round_bf16.restype = f64
    lib.oracle_round_bf16_array.argtypes = [P, P, i64]
    lib.oracle_round_bf16_array.restype = None
    lib.oracle_sage_layer.argtypes = [i64, P, P, P, i64, i64, P, i64, i32, i32, i32, P, i64, P, P]
    lib.oracle_sage_layer.restype = None
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data if a is not None else None


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


# ------------------------------------------------------------------- O1 ---
class CSR:
    def __init__(self, n: int, row_ptr: np.ndarray, col: np.ndarray):
        self.n = n
        self.row_ptr = row_ptr   # int64[n+1]
        self.col = col           # int32[nnz]

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.row_ptr)


def build_csr(n: int, src, dst, symmetrize: bool = True) -> CSR:
    src, dst = _i32(src), _i32(dst)
    m = src.size
    row_ptr = np.zeros(n + 1, np.int64)
    col = np.empty(max(1, 2 * m), np.int32)
    nnz = _load().oracle_build_csr(n, m, _ptr(src), _ptr(dst), int(symmetrize),
                                   _ptr(row_ptr), _ptr(col))
    if nnz == -1:
        raise ValueError("edge endpoint outside [0, n)")
    if nnz < 0:
        raise MemoryError("oracle_build_csr")
    return CSR(n, row_ptr, col[:nnz].copy())


# ------------------------------------------------------------------- O2 ---
def rank_cache(csr: CSR, r: float):
    """(rank int32[n], slot_map int32[n], C) of the degree-ranked cache."""
    rank = np.empty(max(csr.n, 1), np.int32)
    slot = np.empty(max(csr.n, 1), np.int32)
    c = _load().oracle_rank_cache(csr.n, _ptr(csr.row_ptr), float(r), _ptr(rank), _ptr(slot))
    return rank[:csr.n], slot[:csr.n], int(c)


# --------------------------------------------------------------- O3, O4 ---
def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, np.uint32)
    _load().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def draw(rng_seed: int, hop: int, v: int, j: int) -> int:
    return int(_load().oracle_draw(rng_seed, hop, v, j))


def below(x: int, b: int) -> int:
    return int(_load().oracle_below(x, b))


# ------------------------------------------------------------------- O5 ---
def sample_node(csr: CSR, v: int, k: int, rng_seed: int, hop: int) -> np.ndarray:
    deg = int(csr.row_ptr[v + 1] - csr.row_ptr[v])
    out = np.empty(max(1, deg), np.int32)
    c = _load().oracle_sample_node(_ptr(csr.row_ptr), _ptr(csr.col), v, k, rng_seed, hop, _ptr(out))
    return out[:c].copy()


# ------------------------------------------------------------------- O6 ---
class Blocks:
    """Sampled frontiers and per-hop blocks (see oracle.c, O6)."""

    def __init__(self, nodes, sizes, indptr, nbrs, indices):
        self.nodes = nodes        # int32[|F_L|]
        self.sizes = sizes        # [|F_0|, ..., |F_L|]
        self.indptr = indptr      # per hop h=1..L: int32[|F_(h-1)|+1]
        self.nbrs = nbrs          # per hop: int32[E_h] global ids (N_h)
        self.indices = indices    # per hop: int32[E_h] local ids in F_h

    @property
    def n_hops(self) -> int:
        return len(self.indptr)


def hop_bounds(n: int, n_seeds: int, fanouts, max_degree: int):
    """Per-hop capacity (E_h, |F_h|) from Eq. 12 with tau = 1, no overlap."""
    nb = [min(n, n_seeds)]
    eb = []
    for k in fanouts:
        kk = max_degree if k < 0 else min(k, max_degree)
        eb.append(nb[-1] * kk)
        nb.append(min(n, nb[-1] + eb[-1]))
    return eb, nb


def sample_node_biased(csr: CSR, v: int, k: int, rng_seed: int, hop: int, slot_map, eta: int) -> np.ndarray:
    """O5b: locality-biased selection (cached neighbours weighted eta)."""
    deg = int(csr.row_ptr[v + 1] - csr.row_ptr[v])
    out = np.empty(max(1, deg), np.int32)
    sm = _i32(slot_map)
    c = _load().oracle_sample_node_biased(_ptr(csr.row_ptr), _ptr(csr.col), v, k, rng_seed, hop, _ptr(sm),
                                          int(eta), _ptr(out))
    return out[:c].copy()


def below64(x: int, b: int) -> int:
    return int(_load().oracle_below64(x, b))


def sample_blocks(csr: CSR, seeds, fanouts, rng_seed: int, bias_slot_map=None, eta: int = 1) -> Blocks:
    """O6 expansion; with bias_slot_map every hop uses O5b with that map."""
    seeds = _i32(seeds)
    bias = None if bias_slot_map is None else _i32(bias_slot_map)
    fan = _i32(fanouts)
    L = len(fanouts)
    maxdeg = int(csr.degrees().max()) if csr.n > 0 else 0
    eb, nb = hop_bounds(csr.n, seeds.size, fanouts, maxdeg)
    nodes = np.empty(max(1, nb[-1]), np.int32)
    sizes = np.zeros(L + 1, np.int64)
    indptr = [np.empty(nb[h] + 1, np.int32) for h in range(L)]
    nbrs = [np.empty(max(1, eb[h]), np.int32) for h in range(L)]
    indices = [np.empty(max(1, eb[h]), np.int32) for h in range(L)]
    PP = C.c_void_p * max(1, L)
    rc = _load().oracle_sample_blocks(
        csr.n, _ptr(csr.row_ptr), _ptr(csr.col), _ptr(seeds), seeds.size, _ptr(fan), L,
        rng_seed, _ptr(bias), int(eta), _ptr(nodes), _ptr(sizes), PP(*[_ptr(a) for a in indptr]),
        PP(*[_ptr(a) for a in nbrs]), PP(*[_ptr(a) for a in indices]))
    if rc != 0:
        raise ValueError("seed outside [0, n)")
    sizes = [int(s) for s in sizes]
    ip = [indptr[h][:sizes[h] + 1].copy() for h in range(L)]
    e = [int(ip[h][-1]) for h in range(L)]
    return Blocks(nodes[:sizes[-1]].copy(), sizes, ip,
                  [nbrs[h][:e[h]].copy() for h in range(L)],
                  [indices[h][:e[h]].copy() for h in range(L)])


# ------------------------------------------------------------------- O7 ---
def gather(features: np.ndarray, slot_map: np.ndarray, ids, want_misses: bool = False):
    """(rows [n_ids, d] same dtype as features, counts int64[3][, missed ids])."""
    feats = np.ascontiguousarray(features)
    n = feats.shape[0]
    ids = _i32(ids)
    row_bytes = feats.shape[1] * feats.itemsize
    out = np.empty((ids.size, feats.shape[1]), feats.dtype)
    counts = np.zeros(3, np.int64)
    sm = _i32(slot_map)
    misses = np.empty(max(ids.size, 1), np.int32)
    _load().oracle_gather(n, _ptr(feats), row_bytes, _ptr(sm), _ptr(ids), ids.size,
                          _ptr(out), _ptr(counts), _ptr(misses))
    if want_misses:
        return out, counts, misses[:counts[1]].copy()
    return out, counts


class FifoCache:
    """Oracle state of a cache with a FIFO ring over its last `ring_n` slots.

    Starts from the degree-ranked static cache (rank_cache); after each
    gather the batch's misses are admitted in request order (see
    oracle_cache_fifo_admit in oracle.c).
    """

    def __init__(self, csr: "CSR", r: float, ring_n: int):
        rank, slot, c = rank_cache(csr, r)
        self.n, self.c = csr.n, c
        self.slot_map = slot.copy()
        self.owner = np.full(max(c, 1), -1, np.int32)[:c].copy()
        self.owner[:c] = rank[:c]
        if not 0 <= ring_n <= c:
            raise ValueError("ring larger than the cache")
        self.ring_n, self.ring_lo = ring_n, c - ring_n
        self.ptr = np.zeros(1, np.int64)

    def gather(self, features, ids):
        rows, counts, misses = gather(features, self.slot_map, ids, want_misses=True)
        if self.ring_n > 0 and misses.size:
            _load().oracle_cache_fifo_admit(_ptr(self.slot_map), _ptr(self.owner), self.ring_lo,
                                            self.ring_n, _ptr(self.ptr), _ptr(misses), misses.size)
        return rows, counts


class LruCache(FifoCache):
    """Oracle state of a cache with an LRU policy over its last `ring_n` slots.

    Starts from the degree-ranked static cache with the ring's slots in
    index order as the initial recency (lowest slot least recent); after each
    gather the ring slots the batch hit become the most recent and the
    misses are admitted into the least recently used slots (see
    oracle_cache_lru_update in oracle.c).
    """

    def __init__(self, csr: "CSR", r: float, ring_n: int):
        super().__init__(csr, r, ring_n)
        self.order = np.arange(self.ring_lo, self.c, dtype=np.int32)
        self.head = np.zeros(1, np.int64)

    def gather(self, features, ids):
        ids = _i32(ids)
        ok = (ids >= 0) & (ids < self.n)
        slots = self.slot_map[ids[ok]]
        hit_slots = np.ascontiguousarray(slots[slots >= 0], dtype=np.int32)
        rows, counts, misses = gather(features, self.slot_map, ids, want_misses=True)
        if self.ring_n > 0:
            _load().oracle_cache_lru_update(_ptr(self.slot_map), _ptr(self.owner), self.ring_lo, self.ring_n,
                                            _ptr(self.order), _ptr(self.head), _ptr(hit_slots),
                                            hit_slots.size, _ptr(misses), misses.size)
        return rows, counts

    def recency(self) -> np.ndarray:
        """Ring slots from least to most recently used."""
        return np.roll(self.order, -int(self.head[0]))


# ------------------------------------------------------------ bf16, O8 ---
def round_bf16(x: float) -> float:
    return float(_load().oracle_round_bf16(float(x)))


def round_bf16_array(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    _load().oracle_round_bf16_array(_ptr(x), _ptr(y), x.size)
    return y


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 view of float32 values or of bf16 bit patterns."""
    if dtype == "bf16":
        return (np.asarray(a).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def sage_layer(indptr, indices, X: np.ndarray, W: np.ndarray, relu: bool, bf16: bool,
               round_out: bool, rows=None, want_agg: bool = False):
    """One SAGE layer in float64.  X: [n_src, d_in], W: [2*d_in, d_out]."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    W = np.ascontiguousarray(W, dtype=np.float64)
    indptr, indices = _i32(indptr), _i32(indices)
    n_dst = indptr.size - 1
    d_in, d_out = X.shape[1], W.shape[1]
    assert W.shape[0] == 2 * d_in
    rws = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    n_rows = n_dst if rws is None else rws.size
    out = np.zeros((n_rows, d_out), np.float64)
    agg = np.zeros((n_rows, d_in), np.float64) if want_agg else None
    _load().oracle_sage_layer(n_dst, _ptr(indptr), _ptr(indices), _ptr(X), d_in, d_in, _ptr(W),
                              d_out, int(relu), int(bf16), int(round_out), _ptr(rws), n_rows,
                              _ptr(out), _ptr(agg) if agg is not None else None)
    return (out, agg) if want_agg else out


def sage_forward(blocks: Blocks, H0: np.ndarray, Ws, bf16: bool = False, keep=False):
    """L-layer forward (Algorithm 1, its per-layer aggregate/combine loop, forward only).

    Layer l (1-based) uses block b = L-l+1: destinations F_(b-1), sources
    F_b; hidden layers apply ReLU (and bf16 rounding in bf16 mode); the last
    layer's output is returned unrounded.  ``keep`` also returns the list of
    every layer's (agg, H) pair.
    """
    L = blocks.n_hops
    X = np.asarray(H0, dtype=np.float64)
    trace = []
    for l in range(1, L + 1):
        b = L - l + 1
        last = l == L
        H, agg = sage_layer(blocks.indptr[b - 1], blocks.indices[b - 1], X, Ws[l - 1],
                            relu=not last, bf16=bf16, round_out=not last, want_agg=True)
        trace.append((agg, H))
        X = H
    return (X, trace) if keep else X


def sage_forward_rows(blocks: Blocks, H0: np.ndarray, Ws, out_rows, bf16: bool = False):
    """Logits of the destination rows ``out_rows`` of F_0 only.

    Same arithmetic as ``sage_forward``, restricted to the receptive field
    of the requested rows: layer l is evaluated only at the rows that layer
    l+1 reads (its own destination rows and their sampled neighbours).
    Rows outside the receptive field are never read, so they stay zero.
    """
    L = blocks.n_hops
    need = [None] * (L + 1)          # need[l]: rows of H^l that must be computed
    need[L] = np.unique(np.asarray(out_rows, dtype=np.int64))
    for l in range(L, 1, -1):
        b = L - l + 1                # layer l reads block b
        ip, ix = blocks.indptr[b - 1], blocks.indices[b - 1]
        rows = need[l]
        nb = [ix[ip[i]:ip[i + 1]] for i in rows]
        cat = np.concatenate([rows] + [x.astype(np.int64) for x in nb]) if len(rows) else rows
        need[l - 1] = np.unique(cat)
    X = np.asarray(H0, dtype=np.float64)
    for l in range(1, L + 1):
        b = L - l + 1
        last = l == L
        rows = need[l]
        part = sage_layer(blocks.indptr[b - 1], blocks.indices[b - 1], X, Ws[l - 1],
                          relu=not last, bf16=bf16, round_out=not last, rows=rows)
        if last:
            order = np.searchsorted(rows, np.asarray(out_rows, dtype=np.int64))
            return part[order]
        full = np.zeros((blocks.sizes[b - 1], Ws[l - 1].shape[1]), np.float64)
        full[rows] = part
        X = full


# ------------------------------------------------- O9: loss, backward ---
# The training half of Algorithm 1's iteration (loss, backward, update),
# written with numpy in float64.  Forward activations come from
# sage_forward(..., keep=True).

def softmax_xent(Z: np.ndarray, y) -> tuple:
    """Mean softmax cross-entropy over the rows of Z [n, C] with labels y.

    Returns (loss, dZ) where dZ = (softmax(Z) - onehot(y)) / n is the
    gradient of the mean loss with respect to Z.
    """
    Z = np.asarray(Z, dtype=np.float64)
    y = np.asarray(y, dtype=np.int64)
    n = Z.shape[0]
    if n == 0:
        return 0.0, np.zeros_like(Z)
    zmax = Z.max(axis=1, keepdims=True)
    e = np.exp(Z - zmax)
    s = e.sum(axis=1, keepdims=True)
    logp = Z - zmax - np.log(s)
    loss = -logp[np.arange(n), y].mean()
    dZ = e / s
    dZ[np.arange(n), y] -= 1.0
    return float(loss), dZ / n


def aggregate_mean_t(indptr, indices, n_src: int, G: np.ndarray) -> np.ndarray:
    """Adjoint of the mean aggregation of one block (Eq. 1 Aggregate).

    The forward sets agg[i] = (1/cnt_i) * sum of X[indices[p]] over the
    row's edges p; so dX[j] = sum over edges p with indices[p] = j of
    G[i] / cnt_i, where i is the row that holds p.
    """
    indptr = np.asarray(indptr, dtype=np.int64)
    indices = np.asarray(indices, dtype=np.int64)
    G = np.asarray(G, dtype=np.float64)
    cnt = np.diff(indptr)
    row_of_edge = np.repeat(np.arange(cnt.size), cnt)
    dX = np.zeros((n_src, G.shape[1]), np.float64)
    if indices.size:
        np.add.at(dX, indices, G[row_of_edge] / cnt[row_of_edge, None])
    return dX


def sage_backward(blocks: Blocks, H0: np.ndarray, Ws, trace, dZ: np.ndarray, abs_scale: bool = False):
    """Weight gradients of the L-layer SAGE for the output gradient dZ.

    Layer l (block b = L-l+1) computed Z_l = [X[0:n_dst] | agg] W_l from
    its input X = H^(l-1); hence dW_l = [X[0:n_dst] | agg]^T dZ_l.  Below
    the first layer the gradient flows back: d[X[0:n_dst]] = dZ_l W_top^T,
    d(agg) = dZ_l W_bot^T, dX = self part + aggregate_mean_t(d(agg)), and
    through the ReLU of layer l-1: dZ_(l-1) = dX * [H^(l-1) > 0].
    Returns [dW_1, ..., dW_L].  abs_scale: the same recursion over absolute
    values (|X|, |agg|, |W|, |dZ|), the scale of each sum's rounding error.
    """
    if abs_scale:
        H0 = np.abs(np.asarray(H0, dtype=np.float64))
        Ws = [np.abs(np.asarray(w, dtype=np.float64)) for w in Ws]
        trace = [(np.abs(a), np.abs(h)) for a, h in trace]
        dZ = np.abs(np.asarray(dZ, dtype=np.float64))
    L = blocks.n_hops
    dWs = [None] * L
    G = np.asarray(dZ, dtype=np.float64)
    for l in range(L, 0, -1):
        b = L - l + 1
        X = np.asarray(H0, dtype=np.float64) if l == 1 else trace[l - 2][1]
        agg = trace[l - 1][0]
        n_dst = blocks.sizes[b - 1]
        W = np.asarray(Ws[l - 1], dtype=np.float64)
        d_in = X.shape[1]
        dWs[l - 1] = np.concatenate([X[:n_dst], agg], axis=1).T @ G
        if l == 1:
            break
        dX = aggregate_mean_t(blocks.indptr[b - 1], blocks.indices[b - 1], X.shape[0], G @ W[d_in:].T)
        dX[:n_dst] += G @ W[:d_in].T
        G = dX * (X > 0)
    return dWs


def train_step(blocks: Blocks, H0: np.ndarray, Ws, y, lr: float):
    """One iteration: forward, mean softmax-CE over F_0 with labels y,
    backward, and plain SGD W_l <- W_l - lr * dW_l.

    Returns (loss, logits, [dW_l], [updated W_l]).
    """
    Wd = [np.asarray(w, dtype=np.float64) for w in Ws]
    logits, trace = sage_forward(blocks, H0, Wd, keep=True)
    loss, dZ = softmax_xent(logits, y)
    dWs = sage_backward(blocks, H0, Wd, trace, dZ)
    return loss, logits, dWs, [w - lr * g for w, g in zip(Wd, dWs)]
