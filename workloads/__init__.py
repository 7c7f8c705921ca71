"""Seeded synthetic inputs shared by the oracle, the tests and the bench.

This module only *makes inputs*: edge lists, node features, seed batches and
layer weights.  It contains none of the method's arithmetic (no CSR build, no
sampling, no dedup, no gather, no aggregation); those live separately in the
oracle and in the HIP library, and neither imports the other.

Graph shapes follow the paper's node-classification workloads (Section 4.1
names ogbn-arxiv, ogbn-products and Reddit2; Section 4.1 also augments its
estimator with random power-law graphs).  None of those datasets is used:
every graph here is a synthetic power-law graph of the same node count,
density and feature width.

* Chung-Lu graphs: expected-degree weights w_i ~ (i+1)^(-1/(gamma-1)), capped
  at sqrt(n * avg_deg) and rescaled to sum n * avg_deg; endpoints drawn i.i.d.
  proportional to w; self pairs dropped; pairs deduplicated; draws topped up
  until the number of distinct undirected pairs reaches n * avg_deg / 2; node
  ids finally permuted so degree is not correlated with id.
* R-MAT graphs (Chakrabarti, Zhan, Faloutsos 2004): scale-s recursive
  quadrant choice with probabilities (a, b, c, d); endpoints >= n rejected;
  self pairs dropped; pairs deduplicated and topped up; ids permuted.
* Features: i.i.d. N(0, 1) float32, or their bfloat16 rounding.
* Seeds: batch b of an epoch is P[b*B:(b+1)*B] of a seeded permutation P.
* Weights: Glorot-uniform U(-a, a), a = sqrt(6 / (2*d_in + d_out)), shaped
  [2*d_in, d_out] (self half on top, neighbour half below).

Edge lists come from the C generator in gen.c (xoshiro256**, fixed seed);
features, seed permutations and weights from numpy's Philox bit generator
with fixed seeds.  A workload is therefore a pure function of its name.
Generated arrays are cached as .npz files under $GNNAV_WORKLOAD_CACHE
(default /tmp/gnnav_workloads).
"""
from __future__ import annotations

import hashlib
import json
import os
import time

import numpy as np

GRAPH_SEED = 1
FEAT_SEED = 2
PERM_SEED = 3
WEIGHT_SEED = 4
RNG_BASE = 5
LABEL_SEED = 6

# The five workloads.  ``cache`` is the fraction r of nodes held in the
# device cache; ``store_on_device`` keeps the full feature store in HBM.
CONFIGS = {
    "chunglu-10k-d64": dict(
        gen="chunglu", n=10_000, avg_deg=10, gamma=2.1, d=64, dtype="f32",
        fanouts=[5, 5], batch=256, hidden=64, classes=16, cache=0.0,
        store_on_device=True, offsets_i64=False),
    "chunglu-169k-d128": dict(
        gen="chunglu", n=169_000, avg_deg=14, gamma=2.1, d=128, dtype="f32",
        fanouts=[25, 10], batch=1024, hidden=256, classes=40, cache=0.20,
        store_on_device=False, offsets_i64=False),
    "chunglu-233k-d602": dict(
        gen="chunglu", n=233_000, avg_deg=490, gamma=2.1, d=602, dtype="f32",
        fanouts=[25, 10], batch=1024, hidden=256, classes=41, cache=0.50,
        store_on_device=False, offsets_i64=False),
    "chunglu-2450k-d100": dict(
        gen="chunglu", n=2_450_000, avg_deg=50, gamma=2.1, d=100, dtype="f32",
        fanouts=[15, 10, 5], batch=1024, hidden=256, classes=47, cache=0.10,
        store_on_device=False, offsets_i64=False),
    "rmat-10m-d128": dict(
        gen="rmat", n=10_000_000, scale=24, abcd=(0.57, 0.19, 0.19, 0.05),
        nnz=250_000_000, d=128, dtype="bf16", fanouts=[15, 10, 5],
        batch=4096, hidden=256, classes=64, cache=0.25,
        cache_sweep=[0.0, 0.25, 1.0], store_on_device=False,
        offsets_i64=True),
}
CONFIG_ORDER = list(CONFIGS)


def _cache_dir() -> str:
    d = os.environ.get("GNNAV_WORKLOAD_CACHE", "/tmp/gnnav_workloads")
    os.makedirs(d, exist_ok=True)
    return d


def _cached(key: str, make):
    """Return the arrays made by ``make()``, memoised on disk under ``key``."""
    h = hashlib.sha1(key.encode()).hexdigest()[:16]
    path = os.path.join(_cache_dir(), f"{h}.npz")
    if os.path.exists(path):
        with np.load(path) as z:
            return tuple(z[f"a{i}"] for i in range(len(z.files)))
    arrs = make()
    tmp = path + f".tmp{os.getpid()}.npz"
    np.savez(tmp, **{f"a{i}": a for i, a in enumerate(arrs)})
    os.replace(tmp, path)
    return arrs


# ---------------------------------------------------------------- graphs ---

_HERE = os.path.dirname(os.path.abspath(__file__))
_GEN_LIB = None


def build_generator(force: bool = False) -> str:
    """Compile workloads/gen.c into workloads/libgen.so (gcc)."""
    import subprocess
    out = os.path.join(_HERE, "libgen.so")
    if force or not os.path.exists(out):
        tmp = out + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-o", tmp,
                               os.path.join(_HERE, "gen.c"), "-lm"])
        os.replace(tmp, out)
    return out


def _gen():
    global _GEN_LIB
    if _GEN_LIB is None:
        import ctypes as C
        lib = C.CDLL(build_generator())
        i64, f64, u64, p32 = C.c_int64, C.c_double, C.c_uint64, C.c_void_p
        lib.gen_chung_lu.argtypes = [i64, f64, f64, u64, p32, p32, i64]
        lib.gen_chung_lu.restype = i64
        lib.gen_rmat.argtypes = [C.c_int32, i64, f64, f64, f64, f64, u64, p32, p32, i64]
        lib.gen_rmat.restype = i64
        lib.gen_chung_lu_weights.argtypes = [i64, f64, f64, p32]
        lib.gen_chung_lu_weights.restype = i64
        _GEN_LIB = lib
    return _GEN_LIB


def chung_lu_edges(n: int, avg_deg: float, gamma: float, seed: int = GRAPH_SEED):
    """Undirected Chung-Lu pairs (src, dst), each pair listed once, u != v."""
    target = int(round(n * avg_deg / 2))
    src = np.empty(target, np.int32)
    dst = np.empty(target, np.int32)
    got = _gen().gen_chung_lu(n, float(avg_deg), float(gamma), seed,
                              src.ctypes.data, dst.ctypes.data, target)
    if got != target:
        raise RuntimeError(f"Chung-Lu generator failed ({got})")
    return src, dst


def rmat_edges(scale: int, n: int, nnz: int, abcd, seed: int = GRAPH_SEED):
    """Undirected R-MAT pairs over ids [0, n), n <= 2**scale, nnz/2 pairs."""
    target = nnz // 2
    src = np.empty(target, np.int32)
    dst = np.empty(target, np.int32)
    a, b, c, d = (float(x) for x in abcd)
    got = _gen().gen_rmat(scale, n, a, b, c, d, seed, src.ctypes.data,
                          dst.ctypes.data, target)
    if got != target:
        raise RuntimeError(f"R-MAT generator failed ({got})")
    return src, dst


# ------------------------------------------------------- features, seeds ---

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 values, via torch's cast."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def features(n: int, d: int, dtype: str = "f32", seed: int = FEAT_SEED) -> np.ndarray:
    """Row-major [n, d] N(0,1) features: float32, or uint16 bf16 bit patterns."""
    rng = np.random.Generator(np.random.Philox(seed))
    if dtype == "f32":
        return rng.standard_normal((n, d), dtype=np.float32)
    out = np.empty((n, d), np.uint16)
    step = max(1, (1 << 24) // max(d, 1))
    for s in range(0, n, step):
        e = min(n, s + step)
        out[s:e] = f32_to_bf16_bits(rng.standard_normal((e - s, d), dtype=np.float32))
    return out


def epoch_permutation(n: int, seed: int = PERM_SEED) -> np.ndarray:
    rng = np.random.Generator(np.random.Philox(seed))
    return rng.permutation(n).astype(np.int32)


def glorot(d_in: int, d_out: int, dtype: str, seed: int) -> np.ndarray:
    """[2*d_in, d_out] Glorot-uniform weights (float32 or bf16 bits)."""
    rng = np.random.Generator(np.random.Philox(seed))
    a = np.sqrt(6.0 / (2 * d_in + d_out))
    w = rng.uniform(-a, a, size=(2 * d_in, d_out)).astype(np.float32)
    return w if dtype == "f32" else f32_to_bf16_bits(w)


def labels(n: int, classes: int, seed: int = LABEL_SEED) -> np.ndarray:
    """Synthetic class label of every node: int32[n], uniform over [0, classes)."""
    rng = np.random.Generator(np.random.Philox(seed))
    return rng.integers(0, classes, size=n, dtype=np.int32)


def rng_seed_for_batch(b: int) -> int:
    """Sampler key of batch b: (5 << 32) | b."""
    return (RNG_BASE << 32) | int(b)


# --------------------------------------------------------------- workload ---

class Workload:
    """One named configuration; arrays are generated lazily and memoised."""

    def __init__(self, name: str, **overrides):
        if name not in CONFIGS:
            raise KeyError(f"unknown workload {name!r}; known: {CONFIG_ORDER}")
        self.name = name
        self.cfg = dict(CONFIGS[name])
        self.cfg.update(overrides)
        c = self.cfg
        self.n = int(c["n"])
        self.d = int(c["d"])
        self.dtype = c["dtype"]
        self.fanouts = list(c["fanouts"])
        self.L = len(self.fanouts)
        self.batch = int(c["batch"])
        self.dims = [self.d] + [int(c["hidden"])] * (self.L - 1) + [int(c["classes"])]
        self._edges = self._feats = self._perm = self._weights = None

    def _key(self, what: str) -> str:
        keys = ["gen", "n", "avg_deg", "gamma", "scale", "abcd", "nnz"]
        spec = {k: self.cfg.get(k) for k in keys}
        if what != "edges":
            spec.update(d=self.d, dtype=self.dtype, hidden=self.cfg["hidden"],
                        classes=self.cfg["classes"], L=self.L)
        return what + json.dumps(spec, sort_keys=True, default=str)

    def edges(self):
        if self._edges is None:
            c = self.cfg
            if c["gen"] == "chunglu":
                make = lambda: chung_lu_edges(self.n, c["avg_deg"], c["gamma"])
            else:
                make = lambda: rmat_edges(c["scale"], self.n, c["nnz"], c["abcd"])
            self._edges = _cached(self._key("edges"), make)
        return self._edges

    def features(self) -> np.ndarray:
        if self._feats is None:
            self._feats = _cached(self._key("feats"),
                                  lambda: (features(self.n, self.d, self.dtype),))[0]
        return self._feats

    def permutation(self) -> np.ndarray:
        if self._perm is None:
            self._perm = epoch_permutation(self.n)
        return self._perm

    def n_batches(self) -> int:
        return self.n // self.batch

    def seeds(self, b: int) -> np.ndarray:
        p = self.permutation()
        nb = max(1, self.n_batches())
        b = b % nb
        return np.ascontiguousarray(p[b * self.batch:(b + 1) * self.batch])

    def weights(self):
        if self._weights is None:
            self._weights = [glorot(self.dims[l], self.dims[l + 1], self.dtype,
                                    WEIGHT_SEED * 1000 + l) for l in range(self.L)]
        return self._weights

    def rng_seed(self, b: int) -> int:
        return rng_seed_for_batch(b)

    def labels(self) -> np.ndarray:
        if getattr(self, "_labels", None) is None:
            self._labels = labels(self.n, self.dims[-1])
        return self._labels


def tiny_graph(kind: str):
    """Hand-built edge lists (n, src, dst) for edge-case tests."""
    if kind == "empty":
        return 5, np.zeros(0, np.int32), np.zeros(0, np.int32)
    if kind == "one_edge":
        return 2, np.array([0], np.int32), np.array([1], np.int32)
    if kind == "path":
        n = 12
        return n, np.arange(n - 1, dtype=np.int32), np.arange(1, n, dtype=np.int32)
    if kind == "star":
        n = 200
        return n, np.zeros(n - 1, np.int32), np.arange(1, n, dtype=np.int32)
    if kind == "clique":
        n = 9
        u, v = np.triu_indices(n, 1)
        return n, u.astype(np.int32), v.astype(np.int32)
    if kind == "isolated":
        # nodes 0..9 form a cycle; 10..19 have no edges; plus self loops and
        # duplicate pairs that the CSR build must drop.
        u = np.array(list(range(10)) + [3, 4, 4], np.int32)
        v = np.array([(i + 1) % 10 for i in range(10)] + [3, 5, 5], np.int32)
        return 20, u, v
    if kind == "deg_k":
        # hub 0 has degree exactly 5; hub 6 has degree exactly 6.
        u = np.array([0] * 5 + [6] * 6, np.int32)
        v = np.array([1, 2, 3, 4, 5] + [7, 8, 9, 10, 11, 12], np.int32)
        return 13, u, v
    raise KeyError(kind)


def random_graph(n: int, m: int, seed: int):
    """Small Erdos-Renyi-like multigraph edge list (duplicates, self loops allowed)."""
    rng = np.random.Generator(np.random.Philox(1000 + seed))
    u = rng.integers(0, n, m).astype(np.int32)
    v = rng.integers(0, n, m).astype(np.int32)
    return n, u, v


def timed(label: str, fn, *a, **kw):
    t = time.perf_counter()
    r = fn(*a, **kw)
    print(f"[workloads] {label}: {time.perf_counter() - t:.1f}s", flush=True)
    return r
