"""Python binding of libgnnav.so (the C ABI declared in include/gnnav.h).

Argument marshalling only: every step of the sampled mini-batch path runs in
the HIP kernels of the library.  torch supplies device memory (tensors) and
the stream (``torch.cuda.current_stream()``); nothing else is used from it.
If the library is not built this module raises on import: there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgnnav.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python paper_2404_09544_amd/build.py`")

# torch first: its wheel carries its own HIP runtime, which it loads by a
# file name that differs from the runtime's soname.  Loaded after torch, the
# library's libamdhip64.so.7 dependency resolves to that same copy; loaded
# before, the process would end up with two runtimes (two sets of device
# state), and allocations made through one fail in the other.
import torch  # noqa: E402,F401

_lib = C.CDLL(LIB_PATH)

F32, BF16 = 0, 1
SYMMETRIZE, OFFSETS_I64 = 0x1, 0x2
STORE_ON_DEVICE = 0x1
STATUS = {0: "OK", 1: "E_INVALID", 2: "E_RANGE", 3: "E_NOMEM", 4: "E_CAPACITY", 5: "E_DEVICE"}
EXPORTS = [
    "gnnav_last_error", "gnnav_abi_version", "gnnav_build_csr", "gnnav_graph_info",
    "gnnav_graph_csr_host", "gnnav_graph_free", "gnnav_build_cache", "gnnav_cache_info",
    "gnnav_cache_slot_map_host", "gnnav_cache_contents_host", "gnnav_cache_set_policy",
    "gnnav_cache_set_link_workgroups", "gnnav_cache_free", "gnnav_blocks_create", "gnnav_blocks_free",
    "gnnav_sample", "gnnav_sample_async", "gnnav_sample_biased", "gnnav_blocks_sync", "gnnav_blocks_device_sizes",
    "gnnav_blocks_hop", "gnnav_blocks_nodes", "gnnav_gather", "gnnav_gather_n", "gnnav_gather_n_after",
    "gnnav_aggregate_mean", "gnnav_combine", "gnnav_combine_kernel", "gnnav_sage_forward", "gnnav_sage_train_step",
    "gnnav_softmax_xent", "gnnav_aggregate_mean_backward", "gnnav_weight_grad", "gnnav_profile_start",
    "gnnav_profile_stop", "gnnav_profile_count", "gnnav_profile_get", "gnnav_profile_samples",
    "gnnav_sync", "gnnav_debug_set_spin_limit", "gnnav_debug_fail_allocations", "gnnav_gather_noalloc",
    "gnnav_stream_create", "gnnav_stream_destroy",
]


class GnnavError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class BlockView(C.Structure):
    _fields_ = [("n_dst", C.c_int64), ("n_src", C.c_int64), ("nnz", C.c_int64),
                ("indptr", C.c_void_p), ("indices", C.c_void_p), ("neighbors", C.c_void_p),
                ("src_ids", C.c_void_p)]


P, i64, i32, u32, u64, f64 = C.c_void_p, C.c_int64, C.c_int32, C.c_uint32, C.c_uint64, C.c_double
_sig = {
    "gnnav_last_error": ([], C.c_char_p),
    "gnnav_abi_version": ([], i32),
    "gnnav_build_csr": ([i64, i64, P, P, u32, P], i32),
    "gnnav_graph_info": ([P, P, P, P, P], i32),
    "gnnav_graph_csr_host": ([P, P, P], i32),
    "gnnav_graph_free": ([P], None),
    "gnnav_build_cache": ([P, P, i64, i32, f64, u32, P], i32),
    "gnnav_cache_info": ([P, P, P, P, P, P], i32),
    "gnnav_cache_slot_map_host": ([P, P], i32),
    "gnnav_cache_contents_host": ([P, P, P], i32),
    "gnnav_cache_set_policy": ([P, i32, i64], i32),
    "gnnav_cache_set_link_workgroups": ([P, i32], i32),
    "gnnav_cache_free": ([P], None),
    "gnnav_blocks_create": ([P], i32),
    "gnnav_blocks_free": ([P], None),
    "gnnav_sample": ([P, P, i64, P, i32, u64, P, P], i32),
    "gnnav_sample_async": ([P, P, i64, P, i32, u64, P, P], i32),
    "gnnav_sample_biased": ([P, P, u32, P, i64, P, i32, u64, P, i32, P], i32),
    "gnnav_blocks_sync": ([P, P], i32),
    "gnnav_blocks_device_sizes": ([P, P, P], i32),
    "gnnav_gather_n": ([P, P, P, i64, P, i64, P, P], i32),
    "gnnav_gather_n_after": ([P, P, P, i64, P, i64, P, P, P], i32),
    "gnnav_blocks_hop": ([P, i32, C.POINTER(BlockView)], i32),
    "gnnav_blocks_nodes": ([P, P, P, P], i32),
    "gnnav_gather": ([P, P, i64, P, i64, P, P], i32),
    "gnnav_aggregate_mean": ([P, P, i64, P, i64, i64, i32, P, i64, P], i32),
    "gnnav_combine": ([P, i64, P, i64, i64, i64, P, i64, i32, i32, i32, P, i64, P], i32),
    "gnnav_combine_kernel": ([i64, i64, i32], i32),
    "gnnav_sage_forward": ([P, P, i64, P, P, i32, i32, P, i64, P], i32),
    "gnnav_sage_train_step": ([P, P, i64, P, P, i32, P, C.c_float, P, i64, P, P, P], i32),
    "gnnav_softmax_xent": ([P, i64, i64, i64, P, P, i64, P, P], i32),
    "gnnav_aggregate_mean_backward": ([P, P, i64, i64, P, i64, P, i64, P, i64, i64, P, i64, P], i32),
    "gnnav_weight_grad": ([P, i64, P, i64, i64, i64, P, i64, i64, P, P], i32),
    "gnnav_profile_start": ([], i32),
    "gnnav_profile_stop": ([], i32),
    "gnnav_profile_count": ([], i32),
    "gnnav_profile_get": ([i32, P, i32, P, P], i32),
    "gnnav_profile_samples": ([i32, P, i64, P], i32),
    "gnnav_sync": ([P], i32),
    "gnnav_debug_set_spin_limit": ([u32], i32),
    "gnnav_debug_fail_allocations": ([i64], i32),
    "gnnav_gather_noalloc": ([P, P, i64, P, i64, P, P], i32),
    "gnnav_stream_create": ([i32, i32, P], i32),
    "gnnav_stream_destroy": ([P], i32),
}
for _name, (_args, _res) in _sig.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res


def _check(st: int):
    if st != 0:
        raise GnnavError(st, _lib.gnnav_last_error().decode())


def abi_version() -> int:
    return int(_lib.gnnav_abi_version())


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def sync(stream=None):
    """gnnav_sync: wait for `stream`; raises E_DEVICE if device-side work has
    reported a failure (a scan whose look-back wait gave up) since the last
    report."""
    _check(_lib.gnnav_sync(_stream(stream)))


def stream_create(part: int, parts: int):
    """gnnav_stream_create: a stream on share `part` of `parts` of the
    compute units, as a torch.cuda.ExternalStream.  The library's stream
    outlives the wrapper; release it with stream_destroy."""
    import torch
    h = C.c_void_p()
    _check(_lib.gnnav_stream_create(int(part), int(parts), C.byref(h)))
    return torch.cuda.ExternalStream(h.value)


def stream_destroy(stream):
    """gnnav_stream_destroy: waits for the stream, then releases it."""
    _check(_lib.gnnav_stream_destroy(_stream(stream)))


def debug_set_spin_limit(polls: int):
    """Testing hook: look-back polls before a scan's wait gives up (0: at once)."""
    _check(_lib.gnnav_debug_set_spin_limit(int(polls)))


def debug_fail_allocations(after: int):
    """Testing hook: allocations after the next `after` fail (negative: off)."""
    _check(_lib.gnnav_debug_fail_allocations(int(after)))


def _dev_ptr(t):
    return None if t is None else t.data_ptr()


def _np_ptr(a: np.ndarray):
    return a.ctypes.data


def dtype_code(dtype: str) -> int:
    return {"f32": F32, "bf16": BF16}[dtype]


def padded_ld(d: int, dtype: str) -> int:
    elt = 2 if dtype == "bf16" else 4
    return (d * elt + 15) // 16 * 16 // elt


# ------------------------------------------------------------------ graph
class Graph:
    """CSR of G(V, E) in HBM (gnnav_build_csr)."""

    def __init__(self, n_nodes: int, src, dst, symmetrize: bool = True, offsets_i64: bool = False):
        src = np.ascontiguousarray(src, dtype=np.int32)
        dst = np.ascontiguousarray(dst, dtype=np.int32)
        if src.shape != dst.shape:
            raise ValueError("src and dst differ in length")
        flags = (SYMMETRIZE if symmetrize else 0) | (OFFSETS_I64 if offsets_i64 else 0)
        h = P()
        _check(_lib.gnnav_build_csr(n_nodes, src.size, _np_ptr(src), _np_ptr(dst), flags, C.byref(h)))
        self._h = h
        n, nnz, md, o64 = i64(), i64(), i64(), i32()
        _check(_lib.gnnav_graph_info(h, C.byref(n), C.byref(nnz), C.byref(md), C.byref(o64)))
        self.n, self.nnz, self.max_degree, self.offsets_i64 = n.value, nnz.value, md.value, bool(o64.value)

    def csr_host(self, with_col: bool = True):
        rp = np.empty(self.n + 1, np.int64)
        col = np.empty(max(self.nnz, 1), np.int32) if with_col else None
        _check(_lib.gnnav_graph_csr_host(self._h, _np_ptr(rp), _np_ptr(col) if with_col else None))
        return rp, (col[:self.nnz] if with_col else None)

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.gnnav_graph_free(self._h)
            self._h = None

    __del__ = close


# ------------------------------------------------------------------ cache
class Cache:
    """Degree-ranked HBM cache + pinned host store (gnnav_build_cache)."""

    def __init__(self, graph: Graph, feats: np.ndarray, dtype: str, cache_fraction: float,
                 store_on_device: bool = False):
        feats = np.ascontiguousarray(feats)
        if feats.ndim != 2 or feats.shape[0] != graph.n:
            raise ValueError("features must be [n_nodes, d]")
        want = np.uint16 if dtype == "bf16" else np.float32
        if feats.dtype != want:
            raise ValueError(f"features must be {want} for dtype {dtype}")
        h = P()
        _check(_lib.gnnav_build_cache(graph._h, _np_ptr(feats), feats.shape[1], dtype_code(dtype),
                                      float(cache_fraction), STORE_ON_DEVICE if store_on_device else 0,
                                      C.byref(h)))
        self._h = h
        self.dtype = dtype
        nc, d, ld, dt, sod = i64(), i64(), i64(), i32(), i32()
        _check(_lib.gnnav_cache_info(h, C.byref(nc), C.byref(d), C.byref(ld), C.byref(dt), C.byref(sod)))
        self.n_cached, self.d, self.ld = nc.value, d.value, ld.value
        self.store_on_device = bool(sod.value)
        self.n = graph.n

    def set_policy(self, policy: str, dynamic_slots: int = 0):
        """'static', or 'fifo' / 'lru' over the last `dynamic_slots` cache slots."""
        code = {"static": 0, "fifo": 1, "lru": 2}[policy]
        _check(_lib.gnnav_cache_set_policy(self._h, code, int(dynamic_slots)))

    def set_link_workgroups(self, workgroups: int):
        """Workgroups of later gathers that copy misses over the host link."""
        _check(_lib.gnnav_cache_set_link_workgroups(self._h, int(workgroups)))

    def contents(self):
        """(owners int32[n_cached], rows [n_cached, ld]) currently in the cache."""
        owners = np.empty(max(self.n_cached, 1), np.int32)
        rows = np.empty((max(self.n_cached, 1), self.ld), np.uint16 if self.dtype == "bf16" else np.float32)
        _check(_lib.gnnav_cache_contents_host(self._h, _np_ptr(owners), _np_ptr(rows)))
        return owners[:self.n_cached], rows[:self.n_cached]

    def slot_map(self) -> np.ndarray:
        out = np.empty(max(self.n, 1), np.int32)
        _check(_lib.gnnav_cache_slot_map_host(self._h, _np_ptr(out)))
        return out[:self.n]

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.gnnav_cache_free(self._h)
            self._h = None

    __del__ = close


# ----------------------------------------------------------------- blocks
class Blocks:
    """Device workspace holding one batch's frontiers and hops."""

    def __init__(self):
        h = P()
        _check(_lib.gnnav_blocks_create(C.byref(h)))
        self._h = h

    def hop(self, h: int) -> BlockView:
        v = BlockView()
        _check(_lib.gnnav_blocks_hop(self._h, h, C.byref(v)))
        return v

    def sizes(self):
        L = i32()
        _check(_lib.gnnav_blocks_nodes(self._h, None, None, C.byref(L)))
        n = np.zeros(L.value + 1, np.int64)
        ptr = P()
        _check(_lib.gnnav_blocks_nodes(self._h, C.byref(ptr), _np_ptr(n), None))
        return [int(x) for x in n], ptr.value

    def sync(self, stream=None):
        """Publish the last (async) sample's sizes to the host."""
        _check(_lib.gnnav_blocks_sync(self._h, _stream(stream)))

    def device_sizes(self, n_hops: int):
        """(device pointer to the int32 size array, host Eq. 12 bounds [L+1])."""
        ptr = P()
        bounds = np.zeros(n_hops + 1, np.int64)
        _check(_lib.gnnav_blocks_device_sizes(self._h, C.byref(ptr), _np_ptr(bounds)))
        return ptr.value, [int(x) for x in bounds]

    def nodes_ptr(self) -> int:
        ptr = P()
        _check(_lib.gnnav_blocks_nodes(self._h, C.byref(ptr), None, None))
        return ptr.value

    def to_host(self):
        """Host copies: (nodes, sizes, [indptr], [neighbors], [indices])."""
        import torch
        torch.cuda.synchronize()
        sizes, nodes_ptr = self.sizes()
        L = len(sizes) - 1

        def fetch(ptr, count):
            out = np.empty(max(count, 1), np.int32)
            if count > 0:
                _hip_memcpy_d2h(out, ptr, count * 4)
            return out[:count]
        nodes = fetch(nodes_ptr, sizes[-1])
        ip, nb, ix = [], [], []
        for h in range(1, L + 1):
            v = self.hop(h)
            ip.append(fetch(v.indptr, v.n_dst + 1))
            nb.append(fetch(v.neighbors, v.nnz))
            ix.append(fetch(v.indices, v.nnz))
        return nodes, sizes, ip, nb, ix

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.gnnav_blocks_free(self._h)
            self._h = None

    __del__ = close


_hip = None


def _hip_memcpy_d2h(dst: np.ndarray, src_ptr: int, nbytes: int):
    """Synchronous device-to-host copy through the HIP runtime (test/tooling use)."""
    global _hip
    if _hip is None:
        _hip = C.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [P, P, C.c_size_t, C.c_int]
        _hip.hipMemcpy.restype = C.c_int
    rc = _hip.hipMemcpy(dst.ctypes.data, src_ptr, nbytes, 2)  # hipMemcpyDeviceToHost
    if rc != 0:
        raise GnnavError(5, f"hipMemcpy failed ({rc})")


def _copy_device_i32(dst, src_ptr: int, count: int):
    """Enqueue a device-to-device copy of `count` int32 from src_ptr into the
    torch tensor dst on torch's current stream (bookkeeping, not the path)."""
    global _hip
    if _hip is None:
        _hip = C.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [P, P, C.c_size_t, C.c_int]
        _hip.hipMemcpy.restype = C.c_int
    fn = _hip.hipMemcpyAsync
    fn.argtypes = [P, P, C.c_size_t, C.c_int, P]
    fn.restype = C.c_int
    import torch
    rc = fn(dst.data_ptr(), src_ptr, count * 4, 3, torch.cuda.current_stream().cuda_stream)
    if rc != 0:
        raise GnnavError(5, f"hipMemcpyAsync failed ({rc})")


# --------------------------------------------------------------- the path
def sample(graph: Graph, seeds, fanouts, rng_seed: int, blocks: Blocks, stream=None):
    """gnnav_sample: seeds is a device int32 tensor."""
    fan = np.ascontiguousarray(fanouts, dtype=np.int32)
    _check(_lib.gnnav_sample(graph._h, _dev_ptr(seeds), seeds.numel(), _np_ptr(fan), fan.size,
                             int(rng_seed) & 0xFFFFFFFFFFFFFFFF, blocks._h, _stream(stream)))
    return blocks


def sample_async(graph: Graph, seeds, fanouts, rng_seed: int, blocks: Blocks, stream=None):
    """gnnav_sample_async: enqueue only; sizes stay on the device."""
    fan = np.ascontiguousarray(fanouts, dtype=np.int32)
    _check(_lib.gnnav_sample_async(graph._h, _dev_ptr(seeds), seeds.numel(), _np_ptr(fan), fan.size,
                                   int(rng_seed) & 0xFFFFFFFFFFFFFFFF, blocks._h, _stream(stream)))
    return blocks


def sample_biased(graph: Graph, cache: Cache, eta: int, seeds, fanouts, rng_seed: int, blocks: Blocks,
                  async_: bool = False, stream=None):
    """gnnav_sample_biased: cached neighbours weigh eta (eta = 1: uniform weights)."""
    fan = np.ascontiguousarray(fanouts, dtype=np.int32)
    _check(_lib.gnnav_sample_biased(graph._h, cache._h, int(eta), _dev_ptr(seeds), seeds.numel(), _np_ptr(fan),
                                    fan.size, int(rng_seed) & 0xFFFFFFFFFFFFFFFF, blocks._h, int(bool(async_)),
                                    _stream(stream)))
    return blocks


def gather_n(cache: Cache, ids_ptr: int, n_ids_dev_ptr: int, n_ids_max: int, out, counts, stream=None,
             copy_after=None):
    """gnnav_gather_n: the request count is read from device memory.
    copy_after: a recorded torch.cuda.Event the row copies wait for."""
    if copy_after is None:
        _check(_lib.gnnav_gather_n(cache._h, ids_ptr, n_ids_dev_ptr, n_ids_max, _dev_ptr(out), out.stride(0),
                                   _dev_ptr(counts), _stream(stream)))
    else:
        _check(_lib.gnnav_gather_n_after(cache._h, ids_ptr, n_ids_dev_ptr, n_ids_max, _dev_ptr(out),
                                         out.stride(0), _dev_ptr(counts), copy_after.cuda_event, _stream(stream)))


def gather(cache: Cache, ids_ptr: int, n_ids: int, out, counts, stream=None):
    """gnnav_gather into a device tensor `out` [>= n_ids, ld] and int64 counts[3]."""
    ld = out.stride(0)
    _check(_lib.gnnav_gather(cache._h, ids_ptr, n_ids, _dev_ptr(out), ld, _dev_ptr(counts),
                             _stream(stream)))


def gather_noalloc(cache: Cache, ids_ptr: int, n_ids: int, out, counts, stream=None):
    """gnnav_gather_noalloc: gnnav_gather with its workspace in static device
    memory (at most 2**20 ids; calls overlapping on one device race)."""
    _check(_lib.gnnav_gather_noalloc(cache._h, ids_ptr, n_ids, _dev_ptr(out), out.stride(0), _dev_ptr(counts),
                                     _stream(stream)))


def aggregate_mean(indptr_ptr: int, indices_ptr: int, n_dst: int, x, d: int, dtype: str, out,
                   stream=None):
    _check(_lib.gnnav_aggregate_mean(indptr_ptr, indices_ptr, n_dst, _dev_ptr(x), x.stride(0), d,
                                     dtype_code(dtype), _dev_ptr(out), out.stride(0), _stream(stream)))


def combine(self_x, agg, m: int, d_in: int, w, d_out: int, dtype: str, relu: bool, out_bf16: bool,
            out, stream=None):
    _check(_lib.gnnav_combine(_dev_ptr(self_x), self_x.stride(0), _dev_ptr(agg), agg.stride(0), m, d_in,
                              _dev_ptr(w), d_out, dtype_code(dtype), int(relu), int(out_bf16),
                              _dev_ptr(out), out.stride(0), _stream(stream)))



COMBINE_KERNELS = {0: "skinny", 1: "ring", 2: "split"}


def combine_kernel(m: int, d_out: int, dtype: str) -> str:
    """gnnav_combine_kernel: which kernel a combine of m rows runs."""
    k = _lib.gnnav_combine_kernel(int(m), int(d_out), dtype_code(dtype))
    if k < 0:
        raise GnnavError(1, "bad combine_kernel arguments")
    return COMBINE_KERNELS[k]

def sage_train_step(blocks: Blocks, x, weights, dims, labels, lr: float, logits, loss, grads=None,
                    stream=None):
    """gnnav_sage_train_step: fp32; `weights` (device tensors) are updated in place."""
    L = len(weights)
    wp = (P * L)(*[w.data_ptr() for w in weights])
    gp = (P * L)(*[g.data_ptr() for g in grads]) if grads is not None else None
    dm = np.ascontiguousarray(dims, dtype=np.int32)
    _check(_lib.gnnav_sage_train_step(blocks._h, _dev_ptr(x), x.stride(0), wp, _np_ptr(dm), L,
                                      _dev_ptr(labels), float(lr), _dev_ptr(logits), logits.stride(0),
                                      _dev_ptr(loss), gp, _stream(stream)))


def softmax_xent(logits, n: int, n_classes: int, labels, dz, loss, stream=None):
    _check(_lib.gnnav_softmax_xent(_dev_ptr(logits), logits.stride(0), n, n_classes, _dev_ptr(labels),
                                   _dev_ptr(dz), dz.stride(0), _dev_ptr(loss), _stream(stream)))


def aggregate_mean_backward(indptr_ptr: int, indices_ptr: int, n_dst: int, n_src: int, dagg, d: int, out,
                            dself=None, mask=None, stream=None):
    _check(_lib.gnnav_aggregate_mean_backward(
        indptr_ptr, indices_ptr, n_dst, n_src, _dev_ptr(dagg), dagg.stride(0),
        _dev_ptr(dself) if dself is not None else None, dself.stride(0) if dself is not None else 0,
        _dev_ptr(mask) if mask is not None else None, mask.stride(0) if mask is not None else 0,
        d, _dev_ptr(out), out.stride(0), _stream(stream)))


def weight_grad(self_x, agg, m: int, d_in: int, dz, d_out: int, dw, stream=None):
    _check(_lib.gnnav_weight_grad(_dev_ptr(self_x), self_x.stride(0), _dev_ptr(agg), agg.stride(0), m, d_in,
                                  _dev_ptr(dz), dz.stride(0), d_out, _dev_ptr(dw), _stream(stream)))


def sage_forward(blocks: Blocks, x, weights, dims, dtype: str, logits, stream=None):
    L = len(weights)
    wp = (P * L)(*[w.data_ptr() for w in weights])
    dm = np.ascontiguousarray(dims, dtype=np.int32)
    _check(_lib.gnnav_sage_forward(blocks._h, _dev_ptr(x), x.stride(0), wp, _np_ptr(dm), L,
                                   dtype_code(dtype), _dev_ptr(logits), logits.stride(0),
                                   _stream(stream)))


# -------------------------------------------------------------- profiling
def profile_start():
    _check(_lib.gnnav_profile_start())


def profile_samples() -> dict:
    """After profile_stop: {kernel name: float32 array of per-launch ms}."""
    out = {}
    buf = C.create_string_buffer(128)
    for i in range(_lib.gnnav_profile_count()):
        n = i64()
        _check(_lib.gnnav_profile_get(i, buf, 128, None, None))
        _check(_lib.gnnav_profile_samples(i, None, 0, C.byref(n)))
        ms = np.empty(max(n.value, 1), np.float32)
        _check(_lib.gnnav_profile_samples(i, _np_ptr(ms), n.value, None))
        out[buf.value.decode()] = ms[:n.value]
    return out


def profile_stop() -> dict:
    """Stop recording; {kernel name: (launches, total ms)}."""
    _check(_lib.gnnav_profile_stop())
    out = {}
    buf = C.create_string_buffer(128)
    for i in range(_lib.gnnav_profile_count()):
        n, ms = i64(), f64()
        _check(_lib.gnnav_profile_get(i, buf, 128, C.byref(n), C.byref(ms)))
        out[buf.value.decode()] = (n.value, ms.value)
    return out
