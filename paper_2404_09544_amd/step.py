"""One sampled mini-batch step through the C ABI (Algorithm 1's forward).

``MiniBatchStep.run`` is the synchronous form: gnnav_sample (which publishes
the frontier sizes to the host) -> gnnav_gather(F_L) -> gnnav_sage_forward.

``MiniBatchStep.enqueue`` is the asynchronous form: gnnav_sample_async ->
gnnav_gather_n (row count read on the device) -> gnnav_sage_forward, all on
one stream with no host synchronisation; ``finish`` waits and returns the
logits.  Buffers are sized once from the Eq. 12 capacity bounds.

``MiniBatchStep.train`` is a training iteration (fp32): the same sampling
and gather, then gnnav_sage_train_step (forward, softmax cross-entropy over
F_0, backward, SGD on the step's weights in place).

``Pipeline`` runs consecutive batches on alternating streams, each with its
own step (blocks, gathered rows, logits), so batch b+1's sampling and
host-link gather overlap batch b's aggregation and combine: the overlap
Eq. 4 assumes when it takes the epoch time as n_iter times the larger of
(t_sample + t_transfer) and (t_replace + t_compute).  Gathers take the host
link one batch at a time, in batch order (each waits for the previous
batch's gather): two gathers sharing the link would finish together and
leave it idle while both batches compute.

Device buffers are torch tensors that only grow.
"""
from __future__ import annotations

import atexit

import numpy as np
import torch

from . import (Blocks, Cache, Graph, gather, gather_n, sage_forward, sage_train_step, sample, sample_async,
               sample_biased, stream_create, stream_destroy, sync)


def to_device_weights(ws, dtype: str):
    out = []
    for w in ws:
        a = np.ascontiguousarray(w)
        t = torch.from_numpy(a.view(np.int16) if dtype == "bf16" else a)
        out.append(t.to("cuda").contiguous())
    return out


class MiniBatchStep:
    """One batch's sampling, gather and model step.  eta: when set, sampling
    is locality-biased toward the cache's vertices (gnnav_sample_biased)."""

    def __init__(self, graph: Graph, cache: Cache, weights_dev, dims, fanouts, dtype: str, eta=None):
        self.graph, self.cache = graph, cache
        self.weights = list(weights_dev)
        self.dims = list(dims)
        self.fanouts = list(fanouts)
        self.L = len(self.fanouts)
        self.dtype = dtype
        self.blocks = Blocks()
        self.ld = cache.ld
        self._tdt = torch.int16 if dtype == "bf16" else torch.float32
        self.h0 = torch.empty((0, self.ld), dtype=self._tdt, device="cuda")
        self.logits = torch.empty((0, self.dims[-1]), dtype=torch.float32, device="cuda")
        self.counts = torch.zeros(3, dtype=torch.int64, device="cuda")
        self.loss = torch.zeros(1, dtype=torch.float32, device="cuda")
        self.gathered = torch.cuda.Event()       # recorded after each gather
        self.sizes = None
        self._seeds = None
        self._stream = None
        self.eta = eta

    def _sample(self, seeds_dev, rng_seed: int, async_: bool, st):
        if self.eta is None:
            (sample_async if async_ else sample)(self.graph, seeds_dev, self.fanouts, rng_seed, self.blocks, st)
        else:
            sample_biased(self.graph, self.cache, self.eta, seeds_dev, self.fanouts, rng_seed, self.blocks,
                          async_=async_, stream=st)

    def _grow(self, n_l: int, n_0: int, stream=None):
        if self.h0.shape[0] >= n_l and self.logits.shape[0] >= n_0:
            return
        if stream is not None:
            stream.synchronize()        # old buffers may still be read by enqueued work
        if self.h0.shape[0] < n_l:
            self.h0 = torch.empty((n_l + 16, self.ld), dtype=self._tdt, device="cuda")
        if self.logits.shape[0] < n_0:
            self.logits = torch.empty((n_0 + 16, self.dims[-1]), dtype=torch.float32, device="cuda")

    # -------------------------------------------------------------- sync
    def run(self, seeds_dev, rng_seed: int, stream=None):
        """Sample, gather and forward one batch; returns the logits view [|F_0|, classes]."""
        self._sample(seeds_dev, rng_seed, False, stream)
        sizes, nodes_ptr = self.blocks.sizes()
        self.sizes = sizes
        self._grow(sizes[-1], sizes[0])
        gather(self.cache, nodes_ptr, sizes[-1], self.h0, self.counts, stream)
        sage_forward(self.blocks, self.h0, self.weights, self.dims, self.dtype, self.logits, stream)
        return self.logits[:sizes[0]]

    # ------------------------------------------------------------- async
    def enqueue(self, seeds_dev, rng_seed: int, stream=None, gather_after=None, record_gather: bool = True):
        """Enqueue one batch on `stream` without waiting for it; the gather's
        row copies wait for the event `gather_after` when given, and
        `self.gathered` is recorded after them unless record_gather is off."""
        st = stream if stream is not None else torch.cuda.current_stream()
        self._seeds = seeds_dev            # keep alive until the work has run
        self._stream = st
        self._sample(seeds_dev, rng_seed, True, st)
        sizes_ptr, bounds = self.blocks.device_sizes(self.L)
        self._grow(bounds[-1], bounds[0], st)
        gather_n(self.cache, self.blocks.nodes_ptr(), sizes_ptr + 4 * self.L, bounds[-1], self.h0,
                 self.counts, st, copy_after=gather_after)
        if record_gather:
            self.gathered.record(st)
        sage_forward(self.blocks, self.h0, self.weights, self.dims, self.dtype, self.logits, st)
        self.sizes = None

    # ------------------------------------------------------------ train
    def _inputs(self, seeds_dev, rng_seed: int, async_mode: bool, st, gather_after=None):
        """Sample and gather F_L's rows into h0 (on stream st)."""
        if async_mode:
            self._seeds = seeds_dev
            self._stream = st
            self._sample(seeds_dev, rng_seed, True, st)
            sizes_ptr, bounds = self.blocks.device_sizes(self.L)
            self._grow(bounds[-1], bounds[0], st)
            gather_n(self.cache, self.blocks.nodes_ptr(), sizes_ptr + 4 * self.L, bounds[-1], self.h0,
                     self.counts, st, copy_after=gather_after)
            self.gathered.record(st)
            self.sizes = None
        else:
            self._sample(seeds_dev, rng_seed, False, st)
            sizes, nodes_ptr = self.blocks.sizes()
            self.sizes = sizes
            self._grow(sizes[-1], sizes[0])
            gather(self.cache, nodes_ptr, sizes[-1], self.h0, self.counts, st)

    def _train_tail(self, labels_dev, lr: float, grads, st):
        sage_train_step(self.blocks, self.h0, self.weights, self.dims, labels_dev, lr, self.logits, self.loss,
                        grads, st)

    def train(self, seeds_dev, rng_seed: int, labels_dev, lr: float, grads=None, async_mode: bool = False,
              stream=None):
        """One training iteration; labels_dev: device int32 label of every vertex.

        Sync mode returns the logits view [|F_0|, classes]; async mode
        returns None (call ``finish`` for the view).  The loss lands in
        ``self.loss``; ``grads`` (optional device tensors) receive dW_l.
        """
        if self.dtype != "f32":
            raise ValueError("training runs in fp32")
        st = stream if stream is not None else torch.cuda.current_stream()
        self._inputs(seeds_dev, rng_seed, async_mode, st)
        self._train_tail(labels_dev, lr, grads, st)
        return None if async_mode else self.logits[:self.sizes[0]]

    def finish(self):
        """Wait for the enqueued batch; returns its logits view [|F_0|, classes]."""
        self.blocks.sync(self._stream)
        self.sizes, _ = self.blocks.sizes()
        return self.logits[:self.sizes[0]]

    def h0_view(self):
        return self.h0[:self.sizes[-1]]


_STREAMS = []
_PART_STREAMS = {}


@atexit.register
def _release_part_streams():
    """The library's compute-unit-share streams, released at exit after their
    work (a failure here has already been reported by the work itself)."""
    for streams in _PART_STREAMS.values():
        for st in streams:
            try:
                stream_destroy(st)
            except Exception:
                pass
    _PART_STREAMS.clear()


def pipeline_streams(n: int, cu_partition: bool = False):
    """The process's pipeline streams, created once and shared by every
    Pipeline.  HIP multiplexes streams onto a few hardware queues (four by
    default); two busy streams that land on one queue run one after the
    other, so the pipeline keeps its stream count at its depth.  With
    cu_partition, stream j runs on share j of n of the compute units
    (gnnav_stream_create), so the batches in flight never share a unit."""
    if cu_partition:
        if n not in _PART_STREAMS:
            _PART_STREAMS[n] = [stream_create(j, n) for j in range(n)]
        return _PART_STREAMS[n]
    while len(_STREAMS) < n:
        _STREAMS.append(torch.cuda.Stream())
    return _STREAMS[:n]


class Pipeline:
    """Batches b, b+1, ... on `depth` streams in turn (slot b % depth)."""

    def __init__(self, graph: Graph, cache: Cache, weights_dev, dims, fanouts, dtype: str, depth: int = 2,
                 eta=None, link_workgroups=None, cu_partition: bool = False):
        """link_workgroups: host-link workgroups of this pipeline's gathers
        (None keeps the cache's setting); fewer slow the batches computing
        alongside a gather less, at a small cost in link rate.
        cu_partition: each slot's stream runs on its own 1/depth share of
        the compute units, which speeds up steps whose host-link transfer
        dominates and slows down the others."""
        self.slots = [MiniBatchStep(graph, cache, weights_dev, dims, fanouts, dtype, eta=eta) for _ in range(depth)]
        self.streams = pipeline_streams(depth, cu_partition)
        self.depth = depth
        self.count = 0
        self._updated = None
        self.cache = cache
        self.link_workgroups = link_workgroups

    def _link(self):
        if self.link_workgroups is not None:
            self.cache.set_link_workgroups(self.link_workgroups)

    def _previous_gather(self):
        return self.slots[(self.count - 1) % self.depth].gathered if self.count > 0 else None

    def enqueue(self, seeds_dev, rng_seed: int):
        """Enqueue the next batch; returns the slot it runs in.  With the
        whole feature store in HBM no gather crosses the host link, so the
        gathers are not ordered (no event per batch)."""
        k = self.count % self.depth
        self._link()
        if self.cache.store_on_device:
            self.slots[k].enqueue(seeds_dev, rng_seed, self.streams[k], record_gather=False)
        else:
            self.slots[k].enqueue(seeds_dev, rng_seed, self.streams[k], gather_after=self._previous_gather())
        self.count += 1
        return self.slots[k]

    def enqueue_train(self, seeds_dev, rng_seed: int, labels_dev, lr: float):
        """Enqueue the next training iteration.  Its sampling and gather may
        run alongside the previous batch; its forward waits for the previous
        batch's weight update (the weights are shared)."""
        k = self.count % self.depth
        slot, st = self.slots[k], self.streams[k]
        if slot.dtype != "f32":
            raise ValueError("training runs in fp32")
        self._link()
        slot._inputs(seeds_dev, rng_seed, True, st, gather_after=self._previous_gather())
        if self._updated is not None:
            st.wait_event(self._updated)
        slot._train_tail(labels_dev, lr, None, st)
        self._updated = torch.cuda.Event()
        self._updated.record(st)
        self.count += 1
        return slot

    def synchronize(self):
        """Wait for every slot's stream; raises if device-side work reported
        a failure (gnnav_sync)."""
        for s in self.streams:
            sync(s)
