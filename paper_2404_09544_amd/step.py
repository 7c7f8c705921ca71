"""One sampled mini-batch step through the C ABI (Algorithm 1's forward).

``MiniBatchStep.run`` enqueues gnnav_sample -> gnnav_gather(F_L) ->
gnnav_sage_forward on one stream.  Device buffers (gathered features,
logits, hit/miss counts) are torch tensors that only grow, so a steady run
allocates nothing per batch.
"""
from __future__ import annotations

import numpy as np
import torch

from . import BF16, Blocks, Cache, Graph, gather, padded_ld, sage_forward, sample


def to_device_weights(ws, dtype: str):
    out = []
    for w in ws:
        a = np.ascontiguousarray(w)
        t = torch.from_numpy(a.view(np.int16) if dtype == "bf16" else a)
        out.append(t.to("cuda").contiguous())
    return out


class MiniBatchStep:
    def __init__(self, graph: Graph, cache: Cache, weights_dev, dims, fanouts, dtype: str):
        self.graph, self.cache = graph, cache
        self.weights = list(weights_dev)
        self.dims = list(dims)
        self.fanouts = list(fanouts)
        self.dtype = dtype
        self.blocks = Blocks()
        self.ld = cache.ld
        tdt = torch.int16 if dtype == "bf16" else torch.float32
        self._tdt = tdt
        self.h0 = torch.empty((0, self.ld), dtype=tdt, device="cuda")
        self.logits = torch.empty((0, self.dims[-1]), dtype=torch.float32, device="cuda")
        self.counts = torch.zeros(3, dtype=torch.int64, device="cuda")
        self.sizes = None

    def _grow(self, n_l: int, n_0: int):
        if self.h0.shape[0] < n_l:
            self.h0 = torch.empty((int(n_l * 1.25) + 16, self.ld), dtype=self._tdt, device="cuda")
        if self.logits.shape[0] < n_0:
            self.logits = torch.empty((int(n_0 * 1.25) + 16, self.dims[-1]), dtype=torch.float32,
                                      device="cuda")

    def run(self, seeds_dev, rng_seed: int, stream=None):
        """Sample, gather and forward one batch; returns the logits view [|F_0|, classes]."""
        sample(self.graph, seeds_dev, self.fanouts, rng_seed, self.blocks, stream)
        sizes, nodes_ptr = self.blocks.sizes()
        self.sizes = sizes
        self._grow(sizes[-1], sizes[0])
        gather(self.cache, nodes_ptr, sizes[-1], self.h0, self.counts, stream)
        sage_forward(self.blocks, self.h0, self.weights, self.dims, self.dtype, self.logits, stream)
        return self.logits[:sizes[0]]

    def h0_view(self):
        return self.h0[:self.sizes[-1]]
