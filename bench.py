"""Throughput of the sampled mini-batch step on one MI355X.

A step is one mini-batch through the whole path: Eq. 2 fanout sampling with
per-hop dedup/relabel, the cache gather of F_L's feature rows (hits from
HBM, misses from the pinned host store), and the L-layer SAGE forward
(mean aggregation + combine GEMM).  Seeds for every batch are staged in HBM
before the timed region; graph, cache and weights are built once.

Prints one JSON line: seeds/s over the timed steps, a roofline entry for
the dominant device kernel (algorithmic bytes or flops per launch over its
average HIP-event duration, measured inside the timed region), per-kernel
figures, and the CPU oracle timed on a bounded sample of the same batches.

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
                  "combine_gemm": ["gemm.hip", "common.hpp", "dma.hpp", "bf16split.hpp"]}


def cpu_model() -> str:
    """The host CPU's model name as /proc/cpuinfo gives it."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def traffic_for(kernel: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if still current."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_hash") != kernel_source_hash(KERNEL_SOURCES[kernel.split(".")[0]]):
        return None
    return rec.get("bytes_per_launch")


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
    losses = loss_hist[args.warmup:].cpu().numpy()
    link_est = None
    if args.train_link_workgroups == "auto":
        t_tr = prof.get("gather_rows", (0, 0.0))[1] / args.steps
        link_wgs, link_est = pick_link_workgroups(t_tr, seq * 1e3 / args.steps - t_tr)
    else:
        link_wgs = int(args.train_link_workgroups)
    pipe = Pipeline(g, c, wtrain, wl.dims, wl.fanouts, "f32", depth=args.depth, eta=args.eta,
                    link_workgroups=link_wgs)
    for b in range(args.warmup):
        pipe.enqueue_train(seeds_dev[b], wl.rng_seed(b), labels, args.lr)
    pipe.synchronize()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for b in range(args.warmup, n_b):
        pipe.enqueue_train(seeds_dev[b], wl.rng_seed(b), labels, args.lr)
    pipe.synchronize()
    torch.cuda.synchronize()
    piped = time.perf_counter() - t0
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
                # the weight gradient runs on the bf16 matrix cores through the
                # three-way bf16 split: six executed bf16 MFMA flops per fp32 flop
                k.update({"bound": "mfma", "achieved": round(6 * tf, 2), "peak": MFMA_PEAK_TFLOPS["bf16"],
                          "unit": "TFLOP/s", "frac": round(6 * tf / MFMA_PEAK_TFLOPS["bf16"], 4),
                          "fp32_equivalent_tflops": round(tf, 2), "mfma_products_per_flop": 6})
            else:
                k.update({"bound": "mfma", "achieved": round(tf, 2), "peak": MFMA_PEAK_TFLOPS["f32"],
                          "unit": "TFLOP/s", "frac": round(tf / MFMA_PEAK_TFLOPS["f32"], 4)})
        kernels[name] = k
    return {"metric": "trained seed nodes/sec (sample+gather+forward+softmax-CE+backward+SGD)",
            "value": round(wl.batch * args.steps / piped, 2), "unit": "seeds/s",
            "ms_per_step": round(piped * 1e3 / args.steps, 4),
            "value_sequential": round(wl.batch * args.steps / seq, 2), "lr": args.lr,
            "pipeline_link_workgroups": link_wgs, "link_workgroup_estimates_ms": link_est,
            "loss_first": round(float(losses[0]), 6), "loss_last": round(float(losses[-1]), 6),
            "kernels": kernels}


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
    ap.add_argument("--depth", type=int, default=3,
                    help="streams in the pipelined pass (3: a third batch in flight keeps the latency-bound "
                         "sampling kernels busier; 4 measured slower)")
    ap.add_argument("--cache-policy", choices=["static", "fifo"], default="static",
                    help="fifo: admit each batch's misses into a ring over the last cache slots")
    ap.add_argument("--dynamic-fraction", type=float, default=1.0,
                    help="share of the cache slots in the FIFO ring (with --cache-policy fifo)")
    ap.add_argument("--eta", type=int, default=None,
                    help="locality-biased sampling: cached neighbours weigh eta (default: uniform)")
    ap.add_argument("--no-train", action="store_true", help="skip the training leg")
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
    if args.cache_policy == "fifo":
        ring = int(round(c.n_cached * min(max(args.dynamic_fraction, 0.0), 1.0)))
        c.set_policy("fifo", ring)
        log(f"FIFO ring over the last {ring} of {c.n_cached} cache slots")
    ws = wl.weights()
    wdev = to_device_weights(ws, wl.dtype)
    step = MiniBatchStep(g, c, wdev, wl.dims, wl.fanouts, wl.dtype, eta=args.eta)
    n_b = args.warmup + args.steps
    seeds_dev = [torch.from_numpy(wl.seeds(b)).cuda() for b in range(n_b)]
    L = wl.L
    counts_hist = torch.zeros((n_b, 3), dtype=torch.int64, device="cuda")
    seq_counts_hist = torch.zeros((n_b, 3), dtype=torch.int64, device="cuda")
    sizes_dev_hist = torch.zeros((n_b, L + 1), dtype=torch.int32, device="cuda")

    def record(slot, b, st, hist=counts_hist):
        """Copy this batch's counts and frontier sizes aside on its own stream."""
        ptr, _ = slot.blocks.device_sizes(L)
        with torch.cuda.stream(st):
            hist[b].copy_(slot.counts)
            G._copy_device_i32(sizes_dev_hist[b], ptr, L + 1)

    # ---- phase 1: sequential steps on one stream, every kernel timed -----
    # One batch after another with no host synchronisation between batches;
    # the library records HIP events around each kernel (per-kernel figures
    # and the roofline come from this region).
    stream = torch.cuda.current_stream()
    for b in range(args.warmup):
        step.enqueue(seeds_dev[b], wl.rng_seed(b), stream)
        record(step, b, stream, seq_counts_hist)
    torch.cuda.synchronize()
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
    prof_samples = G.profile_samples()
    batch_ms = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)])
    seq_elapsed = t_end - t_start
    seq_ms = seq_elapsed * 1e3 / args.steps
    log(f"sequential {args.steps} steps: {seq_ms:.3f} ms/step, {wl.batch * args.steps / seq_elapsed:,.0f} seeds/s")

    # ---- phase 2: the pipeline (batch b+1 overlaps batch b on another stream)
    fwd_link_est = None
    if args.link_workgroups == "auto":
        t_tr = prof.get("gather_rows", (0, 0.0))[1] / args.steps
        fwd_link, fwd_link_est = pick_link_workgroups(t_tr, seq_ms - t_tr)
    else:
        fwd_link = int(args.link_workgroups)
    pipe = Pipeline(g, c, wdev, wl.dims, wl.fanouts, wl.dtype, depth=args.depth, eta=args.eta,
                    link_workgroups=fwd_link)
    for b in range(args.warmup):
        slot = pipe.enqueue(seeds_dev[b], wl.rng_seed(b))
    pipe.synchronize()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for b in range(args.warmup, n_b):
        slot = pipe.enqueue(seeds_dev[b], wl.rng_seed(b))
        record(slot, b, pipe.streams[(pipe.count - 1) % pipe.depth])
    pipe.synchronize()
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    c.set_link_workgroups(64)
    elapsed = t_end - t_start
    ms_per_step = elapsed * 1e3 / args.steps
    seeds_per_s = wl.batch * args.steps / elapsed
    counts = counts_hist[args.warmup:].cpu().numpy()
    seq_counts = seq_counts_hist[args.warmup:].cpu().numpy()
    sizes_hist = sizes_dev_hist[args.warmup:].cpu().numpy().tolist()
    log(f"pipelined {args.steps} steps: {ms_per_step:.3f} ms/step, {seeds_per_s:,.0f} seeds/s")

    # ---- algorithmic work per timed batch, from the measured sizes -------
    # Re-sampling a batch is deterministic, so the blocks of each timed batch
    # are regenerated here (untimed) to count distinct source rows.
    elt = 2 if wl.dtype == "bf16" else 4
    # (the per-kernel figures come from the sequential region, so its counts)
    # gather_rows moves hits (HBM) and misses (host link) in one launch: it is
    # host-link bound when there are misses, HBM bound otherwise
    work = {"gather_rows": 0.0, "cache_admit": 0.0}
    hit_bytes = miss_bytes = 0.0
    edge = {}
    gemm_bytes = {}
    probe = G.Blocks()
    for i, b in enumerate(range(args.warmup, n_b)):
        sz = sizes_hist[i]
        hits, misses = int(seq_counts[i][0]), int(seq_counts[i][1])
        hit_bytes += hits * (2 * wl.d * elt + 8)
        miss_bytes += misses * wl.d * elt
        # admitted rows: read from the gathered batch, written to the cache, plus owner/slot-map entries
        work["cache_admit"] += min(misses, ring) * (2 * wl.d * elt + 16)
        G.sample(g, seeds_dev[b], wl.fanouts, wl.rng_seed(b), probe)
        _, _, ip, _, ix = probe.to_host()
        for l in range(1, L + 1):
            hb = L - l + 1
            n_dst, E = sz[hb - 1], int(ip[hb - 1][-1])
            u = np.unique(ix[hb - 1]).size
            din, dout = wl.dims[l - 1], wl.dims[l]
            ka, kg = f"aggregate_mean.l{l}", f"combine_gemm.l{l}"
            # compulsory bytes: each distinct source row once, each output row once, the CSR
            work[ka] = work.get(ka, 0.0) + u * din * elt + n_dst * din * elt + 4 * (E + n_dst + 1)
            edge[ka] = edge.get(ka, 0.0) + E * din * elt + n_dst * din * elt + 4 * (E + n_dst + 1)
            work[kg] = work.get(kg, 0.0) + 2.0 * n_dst * (2 * din) * dout
            # the GEMM's compulsory bytes: both A segments, W, the output (hidden
            # layers in the compute dtype, logits in fp32)
            out_elt = elt if l < L else 4
            gemm_bytes[kg] = gemm_bytes.get(kg, 0.0) + (n_dst * 2 * din + 2 * din * dout) * elt + n_dst * dout * out_elt
    probe.close()
    # which combine kernel each layer ran: the split-bf16 kernel executes six
    # bf16 MFMA products per fp32 product, so its roofline is the bf16 peak
    # over the executed flops (the fp32-equivalent rate is reported beside it)
    gemm_kind = {}
    for l in range(1, L + 1):
        m_mean = max(1, int(round(float(np.mean([sz[L - l] for sz in sizes_hist])))))
        gemm_kind[f"combine_gemm.l{l}"] = G.combine_kernel(m_mean, wl.dims[l], wl.dtype)
    link_bound = miss_bytes > 0
    work["gather_rows"] = miss_bytes if link_bound else hit_bytes
    # the committed counter runs used the workload's default cache, a static
    # policy and uniform sampling: their bytes apply only to such runs
    profiled_config = ((args.cache_fraction is None or args.cache_fraction == wl.cfg["cache"])
                       and args.eta is None and args.cache_policy == "static")

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
        if name not in prof:
            continue
        if name == "gather_rows" and link_bound:
            bound, peak, unit = "host_link", HOST_LINK_PEAK_GBS, "GB/s"
        elif name.startswith("combine_gemm"):
            # MFMA-bound when its executed flops per compulsory byte exceed
            # the ridge point peak_flops / HBM bandwidth, else HBM-bound
            split = gemm_kind.get(name) == "split"
            mfma_dtype = "bf16" if split else wl.dtype
            executed = work[name] * (6 if split else 1)
            ridge = MFMA_PEAK_TFLOPS[mfma_dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
            if executed / max(gemm_bytes.get(name, 1.0), 1.0) >= ridge:
                bound, peak, unit = "mfma", MFMA_PEAK_TFLOPS[mfma_dtype], "TFLOP/s"
            else:
                bound, peak, unit = "hbm", HBM_PEAK_GBS, "GB/s"
        else:
            bound, peak, unit = "hbm", HBM_PEAK_GBS, "GB/s"
        launches, ms = prof[name]
        amount = work[name]
        if name.startswith("combine_gemm"):
            amount = gemm_bytes[name] if bound == "hbm" else work[name] * (6 if gemm_kind.get(name) == "split" else 1)
        achieved = amount / (ms * 1e-3) / (1e12 if unit == "TFLOP/s" else 1e9)
        ent = {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
               "frac": round(achieved / peak, 4), "per_launch": round(amount / max(launches, 1), 1)}
        if name in edge:
            ent["achieved_edge_effective"] = round(edge[name] / (ms * 1e-3) / 1e9, 2)
        counted = traffic_for(name, wl.name) if profiled_config else None
        if counted:
            # rocprofv3-counted HBM bytes per launch (committed summary, same
            # kernel source): the counted rate, and compulsory / counted bytes
            byte_work = gemm_bytes.get(name) if name.startswith("combine_gemm") else (
                hit_bytes if name == "gather_rows" else work[name])
            ent["counted_bytes_per_launch"] = counted
            ent["counted_gbs"] = round(counted * launches / (ms * 1e-3) / 1e9, 2)
            if byte_work and not (name == "gather_rows" and link_bound):
                ent["useful_byte_efficiency"] = round(byte_work / max(launches, 1) / counted, 4)
        if name.startswith("combine_gemm"):
            ent["kernel"] = gemm_kind.get(name)
            ent["tflops"] = round(work[name] / (ms * 1e-3) / 1e12, 2)   # algorithmic (fp32-equivalent) rate
            ent["flop_per_byte"] = round(work[name] / max(gemm_bytes.get(name, 1.0), 1.0), 1)
            if gemm_kind.get(name) == "split":
                ent["mfma_products_per_flop"] = 6
        if name == "gather_rows" and link_bound:
            if link.get("zero_copy_gather_gbs"):
                ent["frac_of_measured_link"] = round(achieved / link["zero_copy_gather_gbs"], 4)
            # the hit rows move in the same launch, alongside the misses
            ent["hit_bytes_per_launch"] = round(hit_bytes / max(launches, 1), 1)
            ent["hit_hbm_gbs_alongside"] = round(hit_bytes / (ms * 1e-3) / 1e9, 2)
        kernels[name].update(ent)
        rows.append((ms, name))
    device_rows = [(ms, n) for ms, n in rows if kernels[n]["bound"] in ("hbm", "mfma")]
    dom = max(device_rows)[1] if device_rows else None
    roofline = None
    if dom:
        k = kernels[dom]
        roofline = {"kernel": dom, "bound": k["bound"], "achieved": k["achieved"], "peak": k["peak"],
                    "unit": k["unit"], "frac": k["frac"],
                    "traffic": traffic_for(dom, wl.name) if profiled_config else None}
        if dom.startswith("combine_gemm") and k.get("kernel") == "split":
            roofline["method"] = "fp32 through a three-way bf16 split: 6 bf16 MFMA products per fp32 product"
            roofline["fp32_equivalent_tflops"] = k["tflops"]
            # context: the same fp32 work against the fp32 matrix-core peak
            roofline["fp32_equivalent_frac_of_f32_peak"] = round(k["tflops"] / MFMA_PEAK_TFLOPS["f32"], 4)

    m1 = int(round(float(np.mean([sz[L - 1] for sz in sizes_hist])))) if sizes_hist else 0
    device_cal = device_calibration(torch, m1, 2 * wl.dims[0], wl.dims[1], wl.dtype)
    if roofline is not None and roofline["kernel"] == "combine_gemm.l1" and device_cal.get("library_gemm"):
        roofline["library_frac_same_shape"] = device_cal["library_gemm"]["frac"]
        roofline["library_tflops_same_shape"] = device_cal["library_gemm"]["tflops"]

    # ---- locality-biased sampling: hit rate against the shift it causes --
    locality = None
    if args.eta is not None:
        locality = locality_report(args, G, g, c, wl, seeds_dev, torch)

    # ---- training leg: sample + gather + forward + loss + backward + SGD ----
    train = None
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
        fifo = O.FifoCache(csr, r, ring) if ring else None
        wd = [O.to_f64(w, wl.dtype) for w in ws]
        log(f"oracle set-up {time.perf_counter() - t0:.1f}s")
        # whole batches until --cpu-seconds have passed (at most --cpu-batches)
        nb = 0
        t0 = time.perf_counter()
        while nb < max(1, args.cpu_batches) and (nb == 0 or time.perf_counter() - t0 < args.cpu_seconds):
            b = args.warmup + nb
            bias = None if args.eta is None else (fifo.slot_map if fifo else slot)
            ob = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b), bias_slot_map=bias,
                                 eta=args.eta or 1)
            h0, _ = fifo.gather(feats, ob.nodes) if fifo else O.gather(feats, slot, ob.nodes)
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
            bias = None if args.eta is None else (fifo.slot_map if fifo else slot)
            ob = O.sample_blocks(csr, wl.seeds(b), wl.fanouts, wl.rng_seed(b), bias_slot_map=bias,
                                 eta=args.eta or 1)
            h0, _ = O.gather(feats, slot, ob.nodes)
            O.sage_forward(ob, O.to_f64(h0, wl.dtype), wd, bf16=wl.dtype == "bf16")

        if P > 1 and fifo is None:
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
    repl = ["cache_evict", "cache_admit", "cache_advance"]
    eq4 = {"t_sample_ms": round(per_batch(samp), 4), "t_transfer_ms": round(per_batch(["gather_rows"]), 4),
           "t_replace_ms": round(per_batch(repl), 4),
           "t_compute_ms": round(per_batch(comp), 4), "sequential_ms_per_step": round(seq_ms, 4),
           "pipelined_ms_per_step": round(ms_per_step, 4)}
    eq4["eq4_max_ms"] = round(max(eq4["t_sample_ms"] + eq4["t_transfer_ms"],
                                  eq4["t_replace_ms"] + eq4["t_compute_ms"]), 4)
    mean_sizes = np.mean(np.array(sizes_hist), axis=0).round(1).tolist()
    hit_rate = float(counts[:, 0].sum() / max(counts[:, :2].sum(), 1))
    out = {
        "metric": METRIC, "value": round(seeds_per_s, 2), "unit": "seeds/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name,
                   "seeds": {"graph": W.GRAPH_SEED, "features": W.FEAT_SEED, "permutation": W.PERM_SEED,
                             "weights": W.WEIGHT_SEED, "labels": W.LABEL_SEED,
                             "sampler_batch_b": f"({W.RNG_BASE} << 32) | b"},
                   "pipeline_streams": args.depth, "link_workgroups": fwd_link, "link_workgroup_estimates_ms": fwd_link_est,
                   "n": wl.n, "nnz": g.nnz, "d": wl.d, "fanouts": wl.fanouts,
                   "batch": wl.batch, "layers": wl.L, "dims": wl.dims, "cache_fraction": r,
                   "store_on_device": wl.cfg["store_on_device"], "cache_policy": args.cache_policy,
                   "sampler": "uniform" if args.eta is None else f"locality-biased eta={args.eta}",
                   "fifo_slots": ring, "global_batch": wl.batch},
        "value_sequential": round(wl.batch * args.steps / seq_elapsed, 2),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "cpu_baseline_all_cores": cpu_all,
        "kernels": kernels,
        "eq4": eq4,
        "locality": locality,
        "train": train,
        "host_link_calibration": link,
        "device_calibration": device_cal,
        "graph": graph_stats,
        "sequential_batch_ms": {"median": round(float(np.median(batch_ms)), 4),
                                "p10": round(float(np.percentile(batch_ms, 10)), 4),
                                "p90": round(float(np.percentile(batch_ms, 90)), 4)},
        "batch_stats": {"mean_frontier_sizes": mean_sizes, "hit_rate": round(hit_rate, 4),
                        "hit_rate_sequential": round(float(seq_counts[:, 0].sum() / max(seq_counts[:, :2].sum(), 1)), 4),
                        "miss_bytes_per_batch": round(float(counts[:, 1].mean()) * wl.d * elt, 1)},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
