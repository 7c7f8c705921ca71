"""Throughput of the sampled mini-batch step on one MI355X.

A step is one mini-batch through the whole path: Eq. 2 fanout sampling with
per-hop dedup/relabel, the cache gather of F_L's feature rows (hits from
HBM, misses from the pinned host store), and the L-layer SAGE forward
(mean aggregation + combine GEMM).  Seeds for every batch are staged in HBM
before the timed region; graph, cache and weights are built once.

Prints one JSON line: seeds/s over the timed steps; a roofline entry for the
kernel with the largest share of the step, whatever bounds it (host link,
HBM or matrix cores), and one for the largest device-bound kernel (each the
algorithmic bytes or flops of its launches over their HIP-event durations,
measured inside the timed region); per-kernel figures, the sampling chain
included; the same batches with every row cached (r = 1, where the gather
is the HBM-bound hit copy alone); and the CPU oracle timed on a bounded
sample of the same batches.  Every leg ends at a synchronisation point that
fails the run if device-side work reported an error.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sampled seed nodes/sec through sample+gather+2-layer SAGE fwd; gather/SpMM GB/s"
DEFAULT_WORKLOAD = "chunglu-233k-d602"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
HOST_LINK_PEAK_GBS = 64.0      # PCIe 5.0 x16, one direction
MFMA_PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def _code_only(text: str) -> str:
    """Source text without comments and blank lines (a comment edit leaves
    the kernel, and the counters taken on it, unchanged)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = (re.sub(r"//.*$", "", ln).rstrip() for ln in text.splitlines())
    return "\n".join(ln for ln in lines if ln)


def kernel_source_hash(files) -> str:
    h = hashlib.sha1()
    for f in files:
        with open(os.path.join(ROOT, "paper_2404_09544_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:12]


KERNEL_SOURCES = {"aggregate_mean": ["spmm.hip", "common.hpp"],
                  "gather_rows": ["gather.hip", "common.hpp"],
                  "cache_admit": ["cache_update.hip", "scan.hpp", "common.hpp"],
                  "classify": ["gather.hip", "scan.hpp", "common.hpp"],
                  "combine_gemm": ["gemm.hip", "common.hpp", "dma.hpp", "bf16split.hpp"],
                  "sample_hop": ["sample.hip", "common.hpp"],
                  "dedup_first": ["sample.hip", "common.hpp"],
                  "dedup_scan": ["sample.hip", "scan.hpp", "common.hpp"],
                  "count_scan": ["sample.hip", "scan.hpp", "common.hpp"],
                  "relabel": ["sample.hip", "common.hpp"]}


def cpu_model() -> str:
    """The host CPU's model name as /proc/cpuinfo gives it."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def traffic_for(kernel: str, trace: str):
    """Counted bytes per launch of `kernel` from the committed rocprofv3
    counter runs of the run named `trace` (profiles/*_traffic.json), if they
    were taken on the current kernel source; else None.  The record holds
    bytes_per_launch (FETCH_SIZE and WRITE_SIZE scaled by a plain copy's
    readings) and, where collected, the requests the L2 sent to the memory
    side (dram_*) and to the host link (io_*), in bytes per launch."""
    src = KERNEL_SOURCES.get(kernel.split(".")[0])
    path = os.path.join(ROOT, "profiles", f"{kernel}_{trace}_traffic.json")
    if src is None or not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_hash") != kernel_source_hash(src):
        return None
    return rec


def link_calibration(G, cache, wl, torch):
    """Achievable host-link rates on this machine: a DMA copy from pinned memory,
    and the library's zero-copy miss path over uncached rows in id order."""
    out = {}
    nbytes = 256 << 20
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst.copy_(src, non_blocking=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        dst.copy_(src, non_blocking=True)
    e1.record()
    torch.cuda.synchronize()
    out["dma_h2d_gbs"] = round(5 * nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9, 2)
    del src, dst
    slot = cache.slot_map()
    ids = np.nonzero(slot < 0)[0].astype(np.int32)[:100_000]
    if ids.size and not cache.store_on_device:
        ids_d = torch.from_numpy(ids).cuda()
        rows = torch.empty((ids.size, cache.ld), dtype=torch.int16 if wl.dtype == "bf16" else torch.float32,
                           device="cuda")
        counts = torch.zeros(3, dtype=torch.int64, device="cuda")
        G.gather(cache, ids_d.data_ptr(), ids.size, rows, counts)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(3):
            G.gather(cache, ids_d.data_ptr(), ids.size, rows, counts)
        e1.record()
        torch.cuda.synchronize()
        elt = 2 if wl.dtype == "bf16" else 4
        out["zero_copy_gather_gbs"] = round(3 * ids.size * wl.d * elt / (e0.elapsed_time(e1) * 1e-3) / 1e9, 2)
    else:
        out["zero_copy_gather_gbs"] = None
    return out


def device_calibration(torch, m: int, k: int, n: int, dtype: str):
    """Context for the roofline fractions on this machine: a plain 1 GiB HBM
    copy, and the vendor library's GEMM (torch.mm, hipBLASLt; fp32 without
    reduced-precision shortcuts) on the layer-1 combine shape [m, k] x [k, n]."""
    out = {}
    x = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    out["hbm_copy_gbs"] = round(5 * 2 * x.numel() * 4 / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del x, y
    if m > 0:
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        prev = torch.backends.cuda.matmul.allow_tf32
        torch.backends.cuda.matmul.allow_tf32 = False
        a = torch.randn((m, k), device="cuda").to(tdt)
        b = torch.randn((k, n), device="cuda").to(tdt)
        for _ in range(3):
            torch.mm(a, b)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(20):
            torch.mm(a, b)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / 20
        tf = 2.0 * m * k * n / (us * 1e-6) / 1e12
        out["library_gemm"] = {"shape": [m, k, n], "dtype": dtype, "us": round(us, 2), "tflops": round(tf, 2),
                               "frac": round(tf / MFMA_PEAK_TFLOPS[dtype], 4)}
        torch.backends.cuda.matmul.allow_tf32 = prev
        del a, b
    return out


def locality_report(args, G, g, c, wl, seeds_dev, torch, batches=5):
    """Biased against uniform sampling on the first timed batches (untimed):
    the hit rate of F_L and the share of sampled picks that land on cached
    vertices.  Within each class both samplers pick uniformly, so the
    difference of the two shares is the total-variation distance between the
    biased and the uniform distribution of a pick."""
    slot = c.slot_map()
    out = {"eta": args.eta}
    for label, eta in (("biased", args.eta), ("uniform", None)):
        hits = picks = cached = nodes_total = 0
        blk = G.Blocks()
        for b in range(args.warmup, args.warmup + batches):
            if eta is None:
                G.sample(g, seeds_dev[b], wl.fanouts, wl.rng_seed(b), blk)
            else:
                G.sample_biased(g, c, eta, seeds_dev[b], wl.fanouts, wl.rng_seed(b), blk)
            nodes, _, _, nbrs, _ = blk.to_host()
            hits += int((slot[nodes] >= 0).sum())
            nodes_total += nodes.size
            for nb in nbrs:
                picks += nb.size
                cached += int((slot[nb] >= 0).sum())
        blk.close()
        out[f"hit_rate_{label}"] = round(hits / max(nodes_total, 1), 4)
        out[f"cached_pick_share_{label}"] = round(cached / max(picks, 1), 4)
        out[f"frontier_{label}"] = round(nodes_total / batches, 1)
    out["pick_distribution_tv_shift"] = round(out["cached_pick_share_biased"] - out["cached_pick_share_uniform"], 4)
    log(f"locality eta={args.eta}: hit rate {out['hit_rate_uniform']} -> {out['hit_rate_biased']}, "
        f"cached share of picks {out['cached_pick_share_uniform']} -> {out['cached_pick_share_biased']}")
    return out


# Host-link workgroups of a pipelined leg.  With w workgroups copying
# misses, the transfer runs at LINK_RATE[w] of the 64-workgroup rate and
# kernels running alongside it slow down by LINK_SLOWDOWN[w] (both measured
# on MI355X: a zero-copy gather of 140k random 2416-byte rows next to an HBM
# stream kernel).  A pipelined step takes about max(transfer, the rest of the
# batch slowed down), so the count with the smaller estimate is used; the
# inputs are the sequential leg's per-batch stage times.
LINK_RATE = {64: 1.0, 32: 0.974}
LINK_SLOWDOWN = {64: 1.77, 32: 1.31}


def pick_link_workgroups(t_transfer_ms: float, t_rest_ms: float):
    est = {w: max(t_transfer_ms / LINK_RATE[w], t_rest_ms * LINK_SLOWDOWN[w]) for w in LINK_RATE}
    return min(est, key=lambda w: (est[w], -w)), {str(w): round(v, 4) for w, v in est.items()}


# (compute units partitioned, streams) a pipelined leg may take
PIPE_CANDIDATES = [(False, 3), (True, 2), (True, 3)]


def pick_pipeline(args, make, enqueue, n_b: int, torch, n_time: int = 12):
    """(cu_partition, streams, trial ms/step per candidate) of a pipelined
    leg.  With the partition each batch in flight runs on its own share of
    the compute units (gnnav_stream_create), so the host-link workgroups of
    one batch's gather never share a unit with another batch's kernels; that
    pays where the transfer dominates and costs where sampling and compute
    do.  auto times n_time batches through each candidate (after one untimed
    batch per stream) before the timed region and keeps the fastest.
    Measured on MI355X (ms/step; three streams on all units / two on halves
    / three on thirds): 233k/602-d r=0.5 1.364 / 1.320 / 1.349, 2.45M 1.798
    / 1.747 / 1.770, 169k 0.168-0.181 / 0.171-0.179 / 0.164-0.165, R-MAT
    r=0.25 0.233-0.240 / 0.270-0.276 / 0.276-0.278; training 169k 0.258-0.262
    / 0.228-0.231 / 0.264, 233k 1.343 / 1.310."""
    if args.cu_partition != "auto":
        part = args.cu_partition == "on"
        depth = args.depth if args.depth is not None else (2 if part else 3)
        return part, depth, None
    cands = PIPE_CANDIDATES if args.depth is None else [(False, args.depth), (True, args.depth)]
    trial = {}
    for part, depth in cands:
        pipe = make(depth, part)
        for i in range(depth):
            enqueue(pipe, i % n_b)
        pipe.synchronize()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(n_time):
            enqueue(pipe, i % n_b)
        pipe.synchronize()
        torch.cuda.synchronize()
        trial[(part, depth)] = (time.perf_counter() - t0) * 1e3 / n_time
        del pipe
    part, depth = min(trial, key=trial.get)
    return part, depth, {f"{'shares' if p else 'all_units'}_{d}": round(v, 4) for (p, d), v in trial.items()}


def train_leg(args, G, g, c, wl, ws, seeds_dev, sizes_hist, torch, to_device_weights, MiniBatchStep, Pipeline):
    """Training iterations on the same batches: one stream with every kernel
    timed, then the two-stream pipeline (each forward waits for the
    previous update).  Starts from the bench's initial weights."""
    labels = torch.from_numpy(wl.labels()).cuda()
    n_b = args.warmup + args.steps
    L = wl.L
    wtrain = to_device_weights(ws, "f32")
    step = MiniBatchStep(g, c, wtrain, wl.dims, wl.fanouts, "f32", eta=args.eta)
    stream = torch.cuda.current_stream()
    losses = []
    for b in range(args.warmup):
        step.train(seeds_dev[b], wl.rng_seed(b), labels, args.lr, async_mode=True, stream=stream)
    torch.cuda.synchronize()
    G.profile_start()
    loss_hist = torch.zeros(n_b, dtype=torch.float32, device="cuda")
    t0 = time.perf_counter()
    for b in range(args.warmup, n_b):
        step.train(seeds_dev[b], wl.rng_seed(b), labels, args.lr, async_mode=True, stream=stream)
        loss_hist[b].copy_(step.loss[0])
    torch.cuda.synchronize()
    seq = time.perf_counter() - t0
    prof = G.profile_stop()
    G.sync(stream)
    losses = loss_hist[args.warmup:].cpu().numpy()
    link_est = None
    t_tr = prof.get("gather_rows", (0, 0.0))[1] / args.steps
    if args.train_link_workgroups == "auto":
        link_wgs, link_est = pick_link_workgroups(t_tr, seq * 1e3 / args.steps - t_tr)
    else:
        link_wgs = int(args.train_link_workgroups)
    def make(depth, part):
        return Pipeline(g, c, wtrain, wl.dims, wl.fanouts, "f32", depth=depth, eta=args.eta,
                        link_workgroups=link_wgs, cu_partition=part)

    part, depth, trial = pick_pipeline(
        args, make, lambda p, b: p.enqueue_train(seeds_dev[b], wl.rng_seed(b), labels, args.lr), n_b, torch)
    pipe = make(depth, part)
    for b in range(args.warmup):
        pipe.enqueue_train(seeds_dev[b], wl.rng_seed(b), labels, args.lr)
    pipe.synchronize()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for b in range(args.warmup, n_b):
        pipe.enqueue_train(seeds_dev[b], wl.rng_seed(b), labels, args.lr)
    pipe.synchronize()          # raises if device-side work reported a failure
    torch.cuda.synchronize()
    piped = time.perf_counter() - t0
    G.sync()
    c.set_link_workgroups(64)
    log(f"train: sequential {seq * 1e3 / args.steps:.3f} ms/step, pipelined {piped * 1e3 / args.steps:.3f} ms/step, "
        f"loss {losses[0]:.4f} -> {losses[-1]:.4f}")
    # algorithmic work of the backward kernels from the measured sizes
    work = {}
    for sz in sizes_hist:
        for l in range(1, L + 1):
            hb = L - l + 1
            n_dst, n_src = sz[hb - 1], sz[hb]
            din, dout = wl.dims[l - 1], wl.dims[l]
            work[f"wgrad.l{l}"] = work.get(f"wgrad.l{l}", 0.0) + 2.0 * n_dst * (2 * din) * dout
            if l > 1:
                work[f"bwd_gemm.l{l}"] = work.get(f"bwd_gemm.l{l}", 0.0) + 2.0 * 2 * n_dst * dout * din
    kernels = {}
    for name, (launches, ms) in prof.items():
        k = {"launches": launches, "total_ms": round(ms, 4), "avg_us": round(ms * 1e3 / max(launches, 1), 3)}
        if name in work:
            tf = work[name] / (ms * 1e-3) / 1e12
            if name.startswith("wgrad.l"):
                # fp32 products computed on the bf16 matrix cores through the
                # three-way bf16 split (six executed bf16 MFMA products per fp32
                # product): the algorithmic rate against the fp32 peak, the
                # executed bf16 work beside it
                k.update({"bound": "mfma", "achieved": round(tf, 2), "peak": MFMA_PEAK_TFLOPS["f32"],
                          "unit": "TFLOP/s", "frac": round(tf / MFMA_PEAK_TFLOPS["f32"], 4),
                          "executed_bf16_tflops": round(6 * tf, 2),
                          "executed_frac_of_bf16_peak": round(6 * tf / MFMA_PEAK_TFLOPS["bf16"], 4)})
            else:
                k.update({"bound": "mfma", "achieved": round(tf, 2), "peak": MFMA_PEAK_TFLOPS["f32"],
                          "unit": "TFLOP/s", "frac": round(tf / MFMA_PEAK_TFLOPS["f32"], 4)})
        kernels[name] = k
    return {"metric": "trained seed nodes/sec (sample+gather+forward+softmax-CE+backward+SGD)",
            "value": round(wl.batch * args.steps / piped, 2), "unit": "seeds/s",
            "ms_per_step": round(piped * 1e3 / args.steps, 4),
            "value_sequential": round(wl.batch * args.steps / seq, 2), "lr": args.lr,
            "pipeline_link_workgroups": link_wgs, "link_workgroup_estimates_ms": link_est,
            "pipeline_streams": depth, "cu_partition": part, "pipeline_trial_ms": trial,
            "loss_first": round(float(losses[0]), 6), "loss_last": round(float(losses[-1]), 6),
            "kernels": kernels}


SIZE_SLOTS = 24      # device size array: |F_h| at [h], E_h at [17 + h] (L <= 3 fits in 24)


SEED_TILE = 2048     # seeds the library dedups in one workgroup (one scan tile)


def sampling_bytes(wl, n_h, e_h, off_bytes: int, max_deg: int) -> dict:
    """Algorithmic bytes of one batch's sampling-chain kernels (Eq. 2 and its
    union), by kernel label: each datum a kernel must read or write counted
    once at its own width -- 4-byte ids, counts and slots, `off_bytes` row
    offsets, 8-byte node-table entries (an atomic update counted as a read
    and a write).  A hop with 0 < k <= 64 samples into a slot list of
    min(k, max_deg) slots per row that its dedup scan compacts (no count
    scan); other hops count first.  These kernels make 4- to 8-byte random
    accesses, so they are bound by memory transactions, not by these bytes."""
    L = wl.L
    b0 = wl.batch
    slotted = [0 < k <= 64 and max_deg > 0 for k in wl.fanouts]
    # the seeds' dedup: ids, table, F_0; with hop 1's counts when hop 1 counts
    out = {"dedup_first": b0 * (4 + 16),
           "dedup_scan": b0 * (4 + 8) + n_h[0] * (4 + 8)
           + (0 if slotted[0] else n_h[0] * (2 * off_bytes + 4) + 4),
           "sample_hop": 0, "count_scan": 0, "relabel": 0}
    for h in range(1, L + 1):
        rows, e, new = n_h[h - 1], e_h[h], n_h[h] - n_h[h - 1]
        relabel_prev = e_h[h - 1] * (4 + 8 + 4) if h >= 2 else 0
        if slotted[h - 1]:
            slots = rows * min(wl.fanouts[h - 1], max_deg)
            # rows' ids and offsets, every slot written, picked columns read, first positions noted
            out["sample_hop"] += rows * (4 + 2 * off_bytes) + slots * 4 + e * (4 + 16)
            # slots read, table read for used slots, N_h and indptr written, new
            # ids appended; hop h-1's relabel riding along
            out["dedup_scan"] += slots * 4 + e * (8 + 4) + (rows + 1) * 4 + new * (4 + 8) + relabel_prev
        else:
            # rows' ids, offsets and indptr; picked columns read, neighbours written, first positions noted
            out["sample_hop"] += rows * (4 + 2 * off_bytes + 4) + e * (4 + 4 + 16)
            out["dedup_scan"] += e * (4 + 8) + new * (4 + 8)
            if h >= 2:   # this hop's counts plus hop h-1's relabel riding along
                out["count_scan"] += rows * (4 + 2 * off_bytes) + (rows + 1) * 4 + relabel_prev
    out["relabel"] = e_h[L] * (4 + 8 + 4)
    out["classify"] = n_h[L] * (4 + 4 + 8)
    if slotted[0] and b0 <= SEED_TILE:
        # seeds that fit one scan tile: first positions and their scan in one launch
        out["dedup_scan"] += out.pop("dedup_first")
    return out


def forward_legs(args, G, g, c, wl, wdev, seeds_dev, torch, MiniBatchStep, Pipeline, link_override=None):
    """The forward measurement on cache `c`: a sequential leg on one stream
    with every kernel timed by HIP events (the per-kernel figures), then the
    pipelined leg (the throughput).  Both end at a synchronisation point that
    raises if device-side work reported a failure."""
    L = wl.L
    n_b = args.warmup + args.steps
    step = MiniBatchStep(g, c, wdev, wl.dims, wl.fanouts, wl.dtype, eta=args.eta)
    counts_hist = torch.zeros((n_b, 3), dtype=torch.int64, device="cuda")
    seq_counts_hist = torch.zeros((n_b, 3), dtype=torch.int64, device="cuda")
    sizes_dev_hist = torch.zeros((n_b, SIZE_SLOTS), dtype=torch.int32, device="cuda")

    def record(slot, b, st, hist):
        """Copy this batch's counts and frontier/hop sizes aside on its own stream."""
        ptr, _ = slot.blocks.device_sizes(L)
        with torch.cuda.stream(st):
            hist[b].copy_(slot.counts)
            G._copy_device_i32(sizes_dev_hist[b], ptr, SIZE_SLOTS)

    # ---- sequential steps on one stream, every kernel timed --------------
    stream = torch.cuda.current_stream()
    for b in range(args.warmup):
        step.enqueue(seeds_dev[b], wl.rng_seed(b), stream)
        record(step, b, stream, seq_counts_hist)
    G.sync(stream)
    G.profile_start()
    torch.cuda.synchronize()
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t_start = time.perf_counter()
    marks[0].record(stream)
    for b in range(args.warmup, n_b):
        step.enqueue(seeds_dev[b], wl.rng_seed(b), stream)
        record(step, b, stream, seq_counts_hist)
        marks[b - args.warmup + 1].record(stream)
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    prof = G.profile_stop()
    G.sync(stream)
    prof_samples = G.profile_samples()
    batch_ms = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)])
    seq_elapsed = t_end - t_start
    seq_ms = seq_elapsed * 1e3 / args.steps
    log(f"r={c.n_cached / max(wl.n, 1):.3g} sequential {args.steps} steps: {seq_ms:.3f} ms/step, "
        f"{wl.batch * args.steps / seq_elapsed:,.0f} seeds/s")
    sizes_all = sizes_dev_hist[args.warmup:].cpu().numpy()

    # ---- the pipeline (batch b+1 overlaps batch b on another stream) -----
    link_est = None
    t_tr = prof.get("gather_rows", (0, 0.0))[1] / args.steps
    if link_override is not None:
        link_wgs = link_override
    elif args.link_workgroups == "auto":
        link_wgs, link_est = pick_link_workgroups(t_tr, seq_ms - t_tr)
    else:
        link_wgs = int(args.link_workgroups)
    def make(depth, part):
        return Pipeline(g, c, wdev, wl.dims, wl.fanouts, wl.dtype, depth=depth, eta=args.eta,
                        link_workgroups=link_wgs, cu_partition=part)

    part, depth, trial = pick_pipeline(args, make, lambda p, b: p.enqueue(seeds_dev[b], wl.rng_seed(b)), n_b,
                                       torch)
    pipe = make(depth, part)
    for b in range(args.warmup):
        pipe.enqueue(seeds_dev[b], wl.rng_seed(b))
    pipe.synchronize()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for b in range(args.warmup, n_b):
        pipe.enqueue(seeds_dev[b], wl.rng_seed(b))
    pipe.synchronize()          # raises if device-side work reported a failure
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    G.sync()
    # the timed pass's last batches, still in their slots, against the
    # sequential leg's frontier sizes
    for j in range(min(pipe.depth, args.steps)):
        st = pipe.slots[(pipe.count - 1 - j) % pipe.depth]
        st.finish()
        assert list(st.sizes) == sizes_all[args.steps - 1 - j, :L + 1].tolist(), "pipelined batch differs in size"
    # the same batches again, untimed, each one's counts and sizes copied
    # aside as it completes (the results are deterministic): the copies would
    # otherwise add two enqueues per batch to the timed host loop
    for b in range(args.warmup, n_b):
        slot = pipe.enqueue(seeds_dev[b], wl.rng_seed(b))
        record(slot, b, pipe.streams[(pipe.count - 1) % pipe.depth], counts_hist)
    pipe.synchronize()
    torch.cuda.synchronize()
    c.set_link_workgroups(64)
    elapsed = t_end - t_start
    log(f"r={c.n_cached / max(wl.n, 1):.3g} pipelined {args.steps} steps: {elapsed * 1e3 / args.steps:.3f} ms/step, "
        f"{wl.batch * args.steps / elapsed:,.0f} seeds/s")
    piped_sizes = sizes_dev_hist[args.warmup:].cpu().numpy()
    assert np.array_equal(piped_sizes[:, :L + 1], sizes_all[:, :L + 1]), "pipelined batches differ in size"
    return {"prof": prof, "prof_samples": prof_samples, "batch_ms": batch_ms, "seq_elapsed": seq_elapsed,
            "seq_ms": seq_ms, "elapsed": elapsed, "ms_per_step": elapsed * 1e3 / args.steps,
            "counts": counts_hist[args.warmup:].cpu().numpy(),
            "seq_counts": seq_counts_hist[args.warmup:].cpu().numpy(),
            "n_h": sizes_all[:, :L + 1].astype(np.int64), "e_h": sizes_all[:, 17:17 + L + 1].astype(np.int64),
            "link_workgroups": link_wgs, "link_est": link_est, "depth": depth, "cu_partition": part,
            "trial": trial}


def kernel_entries(args, G, g, c, wl, fwd, seeds_dev, ring, link, profiled_config, trace_name):
    """Per-kernel figures of a sequential leg: each kernel's algorithmic work
    over the timed batches (from their measured sizes) divided by its total
    HIP-event time, against the roofline that bounds it."""
    L = wl.L
    prof, prof_samples = fwd["prof"], fwd["prof_samples"]
    elt = 2 if wl.dtype == "bf16" else 4
    off = 8 if g.offsets_i64 else 4
    # gather_rows moves hits (HBM) and misses (host link) in one launch: it is
    # host-link bound when there are misses, HBM bound otherwise
    work = {"gather_rows": 0.0, "cache_admit": 0.0}
    hit_bytes = miss_bytes = 0.0
    edge, gemm_bytes, samp = {}, {}, {}
    probe = G.Blocks()
    for i, b in enumerate(range(args.warmup, args.warmup + args.steps)):
        n_h, e_h = fwd["n_h"][i], fwd["e_h"][i]
        hits, misses = int(fwd["seq_counts"][i][0]), int(fwd["seq_counts"][i][1])
        hit_bytes += hits * (2 * wl.d * elt + 8)
        miss_bytes += misses * wl.d * elt
        work["cache_admit"] += min(misses, ring) * (2 * wl.d * elt + 16)
        for k, v in sampling_bytes(wl, n_h, e_h, off, g.max_degree).items():
            samp[k] = samp.get(k, 0.0) + v
        # re-sampling a batch is deterministic: regenerate its blocks (untimed,
        # with the leg's own sampler) to count the distinct source rows of
        # each aggregation
        if args.eta is None:
            G.sample(g, seeds_dev[b], wl.fanouts, wl.rng_seed(b), probe)
        else:
            G.sample_biased(g, c, args.eta, seeds_dev[b], wl.fanouts, wl.rng_seed(b), probe)
        _, sz, ip, _, ix = probe.to_host()
        if sz != [int(x) for x in n_h]:
            # only a biased sampler over a cache that moved since (FIFO or LRU) can
            # do this; the distinct-row counts are then of a similar batch
            log(f"batch {b}: re-sampled sizes {sz} differ from the timed batch's {[int(x) for x in n_h]}")
        for l in range(1, L + 1):
            hb = L - l + 1
            n_dst, E = int(n_h[hb - 1]), int(ip[hb - 1][-1])
            u = np.unique(ix[hb - 1]).size
            din, dout = wl.dims[l - 1], wl.dims[l]
            ka, kg = f"aggregate_mean.l{l}", f"combine_gemm.l{l}"
            # compulsory bytes: each distinct source row once, each output row once, the CSR
            work[ka] = work.get(ka, 0.0) + u * din * elt + n_dst * din * elt + 4 * (E + n_dst + 1)
            edge[ka] = edge.get(ka, 0.0) + E * din * elt + n_dst * din * elt + 4 * (E + n_dst + 1)
            work[kg] = work.get(kg, 0.0) + 2.0 * n_dst * (2 * din) * dout
            out_elt = elt if l < L else 4
            gemm_bytes[kg] = gemm_bytes.get(kg, 0.0) + (n_dst * 2 * din + 2 * din * dout) * elt + n_dst * dout * out_elt
    probe.close()
    work.update(samp)
    gemm_kind = {}
    for l in range(1, L + 1):
        m_mean = max(1, int(round(float(np.mean(fwd["n_h"][:, L - l])))))
        gemm_kind[f"combine_gemm.l{l}"] = G.combine_kernel(m_mean, wl.dims[l], wl.dtype)
    link_bound = miss_bytes > 0
    work["gather_rows"] = miss_bytes if link_bound else hit_bytes

    kernels = {}
    for name, (launches, ms) in prof.items():
        kernels[name] = {"launches": launches, "total_ms": round(ms, 4),
                         "avg_us": round(ms * 1e3 / max(launches, 1), 3)}
        smp = prof_samples.get(name)
        if smp is not None and smp.size:
            q = np.percentile(smp.astype(np.float64) * 1e3, [10, 50, 90])
            kernels[name].update({"p10_us": round(q[0], 3), "median_us": round(q[1], 3), "p90_us": round(q[2], 3)})
    rows = []
    for name in work:
        if name not in prof or work[name] <= 0:
            continue
        launches, ms = prof[name]
        split = gemm_kind.get(name) == "split"
        if name == "gather_rows" and link_bound:
            bound, peak, unit, amount = "host_link", HOST_LINK_PEAK_GBS, "GB/s", work[name]
        elif name.startswith("combine_gemm"):
            # the algorithmic flops (2*M*K*N) against the peak of the precision
            # the result carries (the split kernel computes fp32 products on
            # the bf16 matrix cores; its executed bf16 work is a side figure);
            # HBM-bound below the ridge point of that peak
            ridge = MFMA_PEAK_TFLOPS[wl.dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
            if work[name] / max(gemm_bytes.get(name, 1.0), 1.0) >= ridge:
                bound, peak, unit, amount = "mfma", MFMA_PEAK_TFLOPS[wl.dtype], "TFLOP/s", work[name]
            else:
                bound, peak, unit, amount = "hbm", HBM_PEAK_GBS, "GB/s", gemm_bytes[name]
        else:
            bound, peak, unit, amount = "hbm", HBM_PEAK_GBS, "GB/s", work[name]
        achieved = amount / (ms * 1e-3) / (1e12 if unit == "TFLOP/s" else 1e9)
        ent = {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
               "frac": round(achieved / peak, 4), "per_launch": round(amount / max(launches, 1), 1)}
        if name in edge:
            ent["achieved_edge_effective"] = round(edge[name] / (ms * 1e-3) / 1e9, 2)
        if name in samp:
            ent["note"] = "4-8 byte random accesses: transaction-bound"
        rec = traffic_for(name, trace_name) if profiled_config else None
        if rec:
            counted = rec.get("bytes_per_launch")
            # a link-bound gather's counted traffic (the L2's fetches from
            # memory and from the host link, and its writes) against the
            # launch's algorithmic bytes: hit rows read and written, miss rows
            # read over the link and written, list entries
            byte_work = gemm_bytes.get(name) if name.startswith("combine_gemm") else (
                (hit_bytes + miss_bytes * (2 + 8 / (wl.d * elt)) if link_bound else hit_bytes)
                if name == "gather_rows" else work[name])
            ent["counted_bytes_per_launch"] = counted
            ent["counted_gbs"] = round(counted * launches / (ms * 1e-3) / 1e9, 2)
            if byte_work:
                ent["useful_byte_efficiency"] = round(byte_work / max(launches, 1) / counted, 4)
            if name == "gather_rows" and link_bound:
                ent["algorithmic_bytes_per_launch"] = round(byte_work / max(launches, 1), 1)
            for key in ("dram_read_bytes_per_launch", "dram_write_bytes_per_launch", "io_read_bytes_per_launch"):
                if rec.get(key) is not None:
                    ent[key] = rec[key]
            if rec.get("io_read_bytes_per_launch"):
                ent["io_read_gbs_counted"] = round(rec["io_read_bytes_per_launch"] * launches / (ms * 1e-3) / 1e9, 2)
        if name.startswith("combine_gemm"):
            ent["kernel"] = gemm_kind.get(name)
            ent["tflops"] = round(work[name] / (ms * 1e-3) / 1e12, 2)
            ent["flop_per_byte"] = round(work[name] / max(gemm_bytes.get(name, 1.0), 1.0), 1)
            if split:
                ex = 6 * work[name] / (ms * 1e-3) / 1e12
                ent["method"] = "fp32 products as six bf16 part products on the bf16 matrix cores"
                ent["executed_bf16_tflops"] = round(ex, 2)
                ent["executed_frac_of_bf16_peak"] = round(ex / MFMA_PEAK_TFLOPS["bf16"], 4)
        if name == "gather_rows":
            ent["hit_bytes_per_launch"] = round(hit_bytes / max(launches, 1), 1)
            if link_bound:
                if link.get("zero_copy_gather_gbs"):
                    ent["frac_of_measured_link"] = round(achieved / link["zero_copy_gather_gbs"], 4)
                ent["hit_hbm_gbs_alongside"] = round(hit_bytes / (ms * 1e-3) / 1e9, 2)
        kernels[name].update(ent)
        rows.append((ms, name))
    return kernels, rows, {"hit_bytes": hit_bytes, "miss_bytes": miss_bytes, "link_bound": link_bound,
                           "gemm_kind": gemm_kind}


def roofline_of(kernels, name, trace_name, profiled_config):
    k = kernels[name]
    rec = traffic_for(name, trace_name) if profiled_config else None
    out = {"kernel": name, "bound": k["bound"], "achieved": k["achieved"], "peak": k["peak"], "unit": k["unit"],
           "frac": k["frac"], "traffic": rec.get("bytes_per_launch") if rec else None}
    for key in ("method", "executed_bf16_tflops", "executed_frac_of_bf16_peak", "frac_of_measured_link",
                "hit_bytes_per_launch", "algorithmic_bytes_per_launch", "useful_byte_efficiency",
                "io_read_bytes_per_launch",
                "io_read_gbs_counted", "dram_read_bytes_per_launch", "dram_write_bytes_per_launch"):
        if key in k:
            out[key] = k[key]
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cache-fraction", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-batches", type=int, default=16,
                    help="most batches the single-core oracle baseline runs")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="the single-core oracle baseline runs batches until this much time has passed")
    ap.add_argument("--cpu-threads", type=int, default=16,
                    help="cap on the threads of the all-core oracle baseline")
    ap.add_argument("--depth", type=int, default=None,
                    help="streams in the pipelined pass (default: chosen with the partition; 3 without it: "
                         "a third batch in flight keeps the latency-bound sampling kernels busier, 4 measured "
                         "slower)")
    ap.add_argument("--cu-partition", choices=["auto", "on", "off"], default="auto",
                    help="run each pipelined batch on its own share of the compute units (auto: time a few "
                         "batches of three streams on all units, two on halves and three on thirds before "
                         "the timed region and keep the fastest)")
    ap.add_argument("--cache-policy", choices=["static", "fifo", "lru"], default="static",
                    help="fifo: admit each batch's misses into a ring over the last cache slots; lru: the same "
                         "ring, evicting the least recently used slots first")
    ap.add_argument("--dynamic-fraction", type=float, default=1.0,
                    help="share of the cache slots in the ring (with --cache-policy fifo or lru)")
    ap.add_argument("--eta", type=int, default=None,
                    help="locality-biased sampling: cached neighbours weigh eta (default: uniform)")
    ap.add_argument("--no-train", action="store_true", help="skip the training leg")
    ap.add_argument("--no-r1", action="store_true",
                    help="skip the extra forward leg with every row cached (r = 1: the hit gather alone)")
    ap.add_argument("--lr", type=float, default=0.01, help="SGD step of the training leg")
    ap.add_argument("--link-workgroups", default="auto",
                    help="host-link workgroups of the pipelined forward leg's gathers: a count, or auto "
                         "(estimated from the sequential leg's stage times)")
    ap.add_argument("--train-link-workgroups", default="auto",
                    help="the same for the pipelined training leg")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (scales rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = 256 * 1024 * 1024
        x = torch.ones(n, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path is single-GPU: no sharding, no collectives)", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    import paper_2404_09544_amd as G
    from paper_2404_09544_amd.step import MiniBatchStep, Pipeline, to_device_weights

    torch.cuda.set_device(0)
    wl = W.Workload(args.workload)
    r = wl.cfg["cache"] if args.cache_fraction is None else args.cache_fraction
    t0 = time.perf_counter()
    src, dst = wl.edges()
    feats = wl.features()
    log(f"inputs {wl.name}: n={wl.n} pairs={src.size} d={wl.d} {wl.dtype} ({time.perf_counter() - t0:.1f}s)")
    t0 = time.perf_counter()
    g = G.Graph(wl.n, src, dst, offsets_i64=wl.cfg["offsets_i64"])
    c = G.Cache(g, feats, wl.dtype, r, store_on_device=wl.cfg["store_on_device"])
    log(f"graph nnz={g.nnz} max_deg={g.max_degree}; cache C={c.n_cached} ld={c.ld} "
        f"({time.perf_counter() - t0:.1f}s)")
    rp, _ = g.csr_host(with_col=False)
    deg = np.diff(rp)
    top = np.sort(deg)[::-1][:c.n_cached].sum() if c.n_cached else 0
    graph_stats = {"n": wl.n, "nnz": g.nnz, "deg_min": int(deg.min()), "deg_mean": round(float(deg.mean()), 2),
                   "deg_max": int(deg.max()), "cached_rows": c.n_cached,
                   "nnz_share_of_cached_rows": round(float(top) / max(g.nnz, 1), 4)}
    del rp, deg
    link = link_calibration(G, c, wl, torch)
    log(f"host link: DMA {link['dma_h2d_gbs']} GB/s, zero-copy gather of uncached rows {link['zero_copy_gather_gbs']} GB/s")
    ring = 0
    if args.cache_policy != "static":
        ring = int(round(c.n_cached * min(max(args.dynamic_fraction, 0.0), 1.0)))
        c.set_policy(args.cache_policy, ring)
        log(f"{args.cache_policy.upper()} ring over the last {ring} of {c.n_cached} cache slots")
    ws = wl.weights()
    wdev = to_device_weights(ws, wl.dtype)
    n_b = args.warmup + args.steps
    seeds_dev = [torch.from_numpy(wl.seeds(b)).cuda() for b in range(n_b)]
    L = wl.L

    # ---- the forward step at the workload's cache fraction (the headline) --
    fwd = forward_legs(args, G, g, c, wl, wdev, seeds_dev, torch, MiniBatchStep, Pipeline)
    prof = fwd["prof"]
    # counter runs are committed per workload and cache fraction, with a
    # static cache and uniform sampling: their bytes apply only to such runs
    profiled_config = args.eta is None and args.cache_policy == "static"
    trace_name = wl.name if r == wl.cfg["cache"] else f"{wl.name}_r{r:g}"
    kernels, rows, fstats = kernel_entries(args, G, g, c, wl, fwd, seeds_dev, ring, link, profiled_config,
                                           trace_name)
    # the roofline entry: the kernel with the largest total time in the timed
    # sequential leg, whatever bounds it (the host link, HBM or the matrix
    # cores); the largest device-bound (HBM or MFMA) kernel is given beside it
    dom = max(rows)[1] if rows else None
    roofline = roofline_of(kernels, dom, trace_name, profiled_config) if dom else None
    device_rows = [(ms, n) for ms, n in rows if kernels[n]["bound"] in ("hbm", "mfma")]
    dom_dev = max(device_rows)[1] if device_rows else None
    roofline_device = roofline_of(kernels, dom_dev, trace_name, profiled_config) if dom_dev else None

    m1 = int(round(float(np.mean(fwd["n_h"][:, L - 1])))) if args.steps else 0
    device_cal = device_calibration(torch, m1, 2 * wl.dims[0], wl.dims[1], wl.dtype)
    for rl in (roofline, roofline_device):
        if rl is not None and rl["kernel"] == "combine_gemm.l1" and device_cal.get("library_gemm"):
            rl["library_frac_same_shape"] = device_cal["library_gemm"]["frac"]
            rl["library_tflops_same_shape"] = device_cal["library_gemm"]["tflops"]

    # ---- the same batches with every row cached: the hit gather alone ----
    r1 = None
    if not args.no_r1 and r < 1.0 and args.cache_policy == "static" and not wl.cfg["store_on_device"]:
        t0 = time.perf_counter()
        c1 = G.Cache(g, feats, wl.dtype, 1.0)
        log(f"cache r=1: C={c1.n_cached} ({time.perf_counter() - t0:.1f}s)")
        f1 = forward_legs(args, G, g, c1, wl, wdev, seeds_dev, torch, MiniBatchStep, Pipeline, link_override=64)
        k1, rows1, _ = kernel_entries(args, G, g, c1, wl, f1, seeds_dev, 0, link, args.eta is None,
                                      f"{wl.name}_r1")
        r1 = {"cache_fraction": 1.0, "value": round(wl.batch * args.steps / f1["elapsed"], 2), "unit": "seeds/s",
              "ms_per_step": round(f1["ms_per_step"], 4),
              "value_sequential": round(wl.batch * args.steps / f1["seq_elapsed"], 2),
              "pipeline_streams": f1["depth"], "cu_partition": f1["cu_partition"], "pipeline_trial_ms": f1["trial"],
              "roofline_gather": roofline_of(k1, "gather_rows", f"{wl.name}_r1", args.eta is None)
              if "gather_rows" in k1 and k1["gather_rows"].get("bound") else None,
              "roofline": roofline_of(k1, max(rows1)[1], f"{wl.name}_r1", args.eta is None) if rows1 else None,
              "kernels": k1}
        c1.close()
        if r1["roofline_gather"]:
            log(f"r=1 gather: {r1['roofline_gather']['achieved']} GB/s = {r1['roofline_gather']['frac']} of HBM")

    # ---- locality-biased sampling: hit rate against the shift it causes --
    locality = None
    if args.eta is not None:
        locality = locality_report(args, G, g, c, wl, seeds_dev, torch)

    # ---- training leg: sample + gather + forward + loss + backward + SGD ----
    train = None
    sizes_hist = fwd["n_h"].tolist()
    if not args.no_train and wl.dtype == "f32":
        train = train_leg(args, G, g, c, wl, ws, seeds_dev, sizes_hist, torch, to_device_weights, MiniBatchStep,
                          Pipeline)

    # ---- CPU baseline: the oracle on a bounded sample of the same batches --
    cpu = None
    cpu_all = None
    if not args.no_cpu_baseline:
        import oracle as O
        t0 = time.perf_counter()
        csr = O.build_csr(wl.n, src, dst)
        _, slot, _ = O.rank_cache(csr, r)
        dyn = ({"fifo": O.FifoCache, "lru": O.LruCache}[args.cache_policy](csr, r, ring) if ring else None)
        wd = [O.to_f64(w, wl.dtype) for w in ws]
        log(f"oracle set-up {time.perf_counter() - t0:.1f}s")
        # whole batches until --cpu-seconds have passed (at most --cpu-batches)
        nb = 0
        t0 = time.perf_counter()
        while nb < max(1, args.cpu_batches) and (nb == 0 or time.perf_counter() - t0 < args.cpu_seconds):
            b = args.warmup + nb
            bias = None if args.eta is None else (dyn.slot_map if dyn else slot)
            ob = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b), bias_slot_map=bias,
                                 eta=args.eta or 1)
            h0, _ = dyn.gather(feats, ob.nodes) if dyn else O.gather(feats, slot, ob.nodes)
            O.sage_forward(ob, O.to_f64(h0, wl.dtype), wd, bf16=wl.dtype == "bf16")
            nb += 1
        ct = time.perf_counter() - t0
        cpu = {"value": round(wl.batch * nb / ct, 2), "unit": "seeds/s", "cores": 1, "kind": "oracle",
               "cpu_model": cpu_model(),
               "sample": f"{nb} batch(es) of {wl.batch} seeds of {wl.name} (batches {args.warmup}.."
                         f"{args.warmup + nb - 1}), single-threaded C oracle, {ct:.1f}s"}
        log(f"oracle: {cpu['value']} seeds/s")
        # all host cores: independent batches on P threads (the C oracle
        # releases the interpreter lock), P = the cores this process may use
        P = max(1, min(len(os.sched_getaffinity(0)), args.cpu_threads))

        def one(b):
            bias = None if args.eta is None else (dyn.slot_map if dyn else slot)
            ob = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b), bias_slot_map=bias,
                                 eta=args.eta or 1)
            h0, _ = O.gather(feats, slot, ob.nodes)
            O.sage_forward(ob, O.to_f64(h0, wl.dtype), wd, bf16=wl.dtype == "bf16")

        if P > 1 and dyn is None:
            import concurrent.futures as cf
            t0 = time.perf_counter()
            with cf.ThreadPoolExecutor(max_workers=P) as ex:
                list(ex.map(one, [args.warmup + (i % args.steps) for i in range(P)]))
            ct = time.perf_counter() - t0
            cpu_all = {"value": round(wl.batch * P / ct, 2), "unit": "seeds/s", "cores": P, "kind": "oracle",
                       "cpu_model": cpu_model(),
                       "sample": f"{P} batches of {wl.batch} seeds of {wl.name}, one per thread, "
                                 f"single-threaded C oracle on each, {ct:.1f}s"}
            log(f"oracle on {P} threads: {cpu_all['value']} seeds/s")

    # Eq. 4 terms per batch from the sequential region: the host-link part
    # (t_transfer = miss copy), the sampling kernels, and the device compute.
    def per_batch(names):
        return sum(prof[n][1] for n in names if n in prof) / args.steps
    samp = ["dedup_first", "dedup_scan", "count_scan", "sample_hop", "relabel"]
    comp = [n for n in prof if n.startswith(("aggregate_mean", "combine_gemm"))] + ["classify", "weights_transpose"]
    repl = [n for n in prof if n.startswith("cache_")]   # every kernel of the update policy
    eq4 = {"t_sample_ms": round(per_batch(samp), 4), "t_transfer_ms": round(per_batch(["gather_rows"]), 4),
           "t_replace_ms": round(per_batch(repl), 4),
           "t_compute_ms": round(per_batch(comp), 4), "sequential_ms_per_step": round(fwd["seq_ms"], 4),
           "pipelined_ms_per_step": round(fwd["ms_per_step"], 4)}
    eq4["eq4_max_ms"] = round(max(eq4["t_sample_ms"] + eq4["t_transfer_ms"],
                                  eq4["t_replace_ms"] + eq4["t_compute_ms"]), 4)
    counts, seq_counts = fwd["counts"], fwd["seq_counts"]
    mean_sizes = np.mean(fwd["n_h"], axis=0).round(1).tolist()
    mean_edges = np.mean(fwd["e_h"][:, 1:], axis=0).round(1).tolist()
    hit_rate = float(counts[:, 0].sum() / max(counts[:, :2].sum(), 1))
    elt = 2 if wl.dtype == "bf16" else 4
    seeds_per_s = wl.batch * args.steps / fwd["elapsed"]
    batch_ms = fwd["batch_ms"]
    out = {
        "metric": METRIC, "value": round(seeds_per_s, 2), "unit": "seeds/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(fwd["ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name,
                   "seeds": {"graph": W.GRAPH_SEED, "features": W.FEAT_SEED, "permutation": W.PERM_SEED,
                             "weights": W.WEIGHT_SEED, "labels": W.LABEL_SEED,
                             "sampler_batch_b": f"({W.RNG_BASE} << 32) | b"},
                   "pipeline_streams": fwd["depth"], "cu_partition": fwd["cu_partition"],
                   "pipeline_trial_ms": fwd["trial"],
                   "link_workgroups": fwd["link_workgroups"],
                   "link_workgroup_estimates_ms": fwd["link_est"],
                   "n": wl.n, "nnz": g.nnz, "d": wl.d, "fanouts": wl.fanouts,
                   "batch": wl.batch, "layers": wl.L, "dims": wl.dims, "cache_fraction": r,
                   "store_on_device": wl.cfg["store_on_device"], "cache_policy": args.cache_policy,
                   "sampler": "uniform" if args.eta is None else f"locality-biased eta={args.eta}",
                   "dynamic_slots": ring, "global_batch": wl.batch},
        "value_sequential": round(wl.batch * args.steps / fwd["seq_elapsed"], 2),
        "roofline": roofline,
        "roofline_device": roofline_device,
        "cpu_baseline": cpu,
        "cpu_baseline_all_cores": cpu_all,
        "kernels": kernels,
        "r1": r1,
        "eq4": eq4,
        "locality": locality,
        "train": train,
        "host_link_calibration": link,
        "device_calibration": device_cal,
        "graph": graph_stats,
        "sequential_batch_ms": {"median": round(float(np.median(batch_ms)), 4),
                                "p10": round(float(np.percentile(batch_ms, 10)), 4),
                                "p90": round(float(np.percentile(batch_ms, 90)), 4)},
        "batch_stats": {"mean_frontier_sizes": mean_sizes, "mean_edges_per_hop": mean_edges,
                        "hit_rate": round(hit_rate, 4),
                        "hit_rate_sequential": round(float(seq_counts[:, 0].sum() / max(seq_counts[:, :2].sum(), 1)), 4),
                        "miss_bytes_per_batch": round(float(counts[:, 1].mean()) * wl.d * elt, 1)},
    }
    G.sync()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
