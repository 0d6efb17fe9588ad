#!/usr/bin/env python3
"""Benchmark: paged-KV gather / scatter / staged restore on one MI355X.

Default workload (--workload 8b-80k): Llama-3-8B-shaped KV cache (32 layers,
K and V each [20000 blocks, 16 tokens, 8 KV heads, head dim 128] bf16, N(0,1)
from a seed), an 80,000-token prefix = 5,000 blocks at seeded random block
ids, 256-token transfer chunks (all layers per chunk, layer-major).

One step = the whole hot path once over that prefix:
  1. gather the 5,000 blocks into packed chunks (HBM -> HBM),
  2. scatter the packed chunks into 5,000 fresh blocks (HBM -> HBM),
  3. staged restore of an 80k-token packed image from pinned host memory
     through a 4 x 64 MiB pinned staging ring (fill -> H2D on a side stream ->
     scatter kernel, overlapped through HIP events) into another 5,000 blocks.
Inputs are resident (cache in HBM, image in pinned host memory) before the
timed region starts. Prints ONE JSON line. `value` is the gather/scatter HBM
throughput (bytes read plus bytes written by the two kernels, per second of
their event-timed device time); the restore time is reported next to it.

Other workloads print one JSON line each with their own metric:
  --workload 8b-32k-sweep  32,768-token prefix, chunks of 16/64/256/1024
                           tokens (gather, scatter) and rings of 2/4/8 slots
                           (staged restore), 20,000-block pool;
  --workload 70b-batch     64 requests on a seeded prefix tree over a
                           70B-shaped cache (80 layers): the distinct missing
                           chunks restored through one ring while the new
                           blocks are offloaded through another;
  --workload 8b-placements the default gather and scatter on every pair of
                           several caches and packed buffers alive at once
                           (--caches, --packed): how much of a run-to-run
                           spread is where the allocations land in memory.
  --workload 8b-layouts    the default gather and scatter with the cache read
                           as each of the three layouts, on the same
                           allocations (--caches x --packed pairs): what a
                           layout costs, with placement held fixed.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, vendor figure
# The copy kernels' sources: the kernels, the store they issue, the walk
# selection and the launch constants they share.
KERNELS_SRC = [os.path.join(ROOT, "paper_2609_11744_amd", "csrc", f)
               for f in ("kvx_kernels.hip", "kvx_store.h", "kvx_walk.cpp", "kvx_internal.h")]

# HBM bytes of one gather launch on the 80k workload, from two rocprofv3 --pmc
# runs (FETCH_SIZE, then WRITE_SIZE; profiles/copy_units_8b_80k_pmc.md), each
# scaled by what the same counter reads for a 4 GiB plain device copy. Valid
# only for the kernel code they were taken on (kernels_sha256 below); otherwise the
# bench reports traffic as null.
GATHER_TRAFFIC = {
    "kernels_sha256": "96ab12857d16c71ee4cd3fc6458b23157b570131f84e23a98ea96daadf762bfa",
    # cache layout -> (fetched, written) HBM bytes of the timed gather launch
    # at the default 80k-token workload: FETCH_SIZE KiB x 1.999988 (copy
    # calibration), WRITE_SIZE KiB x 1.0
    "nhd": (10488814621, 10485760000),         # 5,121,521.1 / 10,240,000.0 KiB
    "paged_attn": (10488986766, 10485760000),  # 5,121,604.9 / 10,240,000.0 KiB
    "hnd": (10488843210, 10485760000),         # 5,121,536.0 / 10,240,000.0 KiB
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="8b-80k",
                    choices=["8b-80k", "8b-32k-sweep", "70b-batch", "8b-files", "8b-preload",
                             "8b-placements", "8b-layouts"])
    ap.add_argument("--caches", type=int, default=4,
                    help="8b-placements: caches allocated (8b-layouts: at most 2)")
    ap.add_argument("--packed", type=int, default=3,
                    help="8b-placements: packed buffers allocated")
    ap.add_argument("--num-blocks", type=int, default=20000)
    ap.add_argument("--prefix-blocks", type=int, default=5000)
    ap.add_argument("--kv-heads", type=int, default=8,
                    help="default workload: KV heads held by this GPU (8: the whole 8B-shaped "
                         "cache; 1: one tensor-parallel shard at tp = 8)")
    ap.add_argument("--chunk-tokens", type=int, default=256)
    ap.add_argument("--slots", type=int, default=4)
    ap.add_argument("--slot-mib", type=int, default=64)
    ap.add_argument("--fill-threads", type=int, default=8)
    ap.add_argument("--seed", type=int, default=3)
    ap.add_argument("--layout", default="nhd", choices=["nhd", "hnd", "paged_attn"],
                    help="cache tensor layout (8b-80k workload)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-blocks", type=int, default=1250)
    ap.add_argument("--probe-reps", type=int, default=10)
    ap.add_argument("--tier-dir", default="_tier_bench",
                    help="8b-files: directory for the chunk files (created, removed after)")
    ap.add_argument("--io-depth", type=int, default=8, help="8b-files: storage I/O depth")
    ap.add_argument("--offload-reps", type=int, default=3,
                    help="reps of the staged offload leg (8b-80k), timed after the steps")
    ap.add_argument("--trace-out", default="",
                    help="8b-80k: write the traced restore's timeline (run after the timed "
                         "steps) as Chrome trace-event JSON to this path")
    ap.add_argument("--sweep-reps", type=int, default=5,
                    help="reps of the 32k-token gather / scatter sweep (8b-80k), timed after "
                         "the steps; 0 skips it")
    return ap.parse_args()


def kernels_sha256(texts=None) -> str:
    """Fingerprint of the copy kernels' code: their sources with comments and
    runs of blank space removed, so that editing a comment does not void the
    recorded traffic."""
    import re

    if texts is None:
        texts = []
        for path in KERNELS_SRC:
            with open(path, encoding="utf-8") as f:
                texts.append(f.read())
    h = hashlib.sha256()
    for text in texts:
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(re.sub(r"\s+", " ", text).strip().encode())
    return h.hexdigest()


def copies_desc(stats):
    """How a ring's last transfer moved its host-link copies."""
    if stats.get("dma"):
        return "DMA engine (id bit %d)" % stats["dma_engine"]
    return "HIP runtime"


def probes(dev, reps):
    """Same-run link and copy probes: 1 GiB pinned H2D / D2H, 4 GiB D2D, and
    the HBM read / write / copy rates of a kernel shaped like the slab mover."""
    import torch

    def timed_copy(dst, src, n):
        out = []
        for _ in range(n):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            dst.copy_(src, non_blocking=True)
            b.record()
            b.synchronize()
            out.append(a.elapsed_time(b))
        return statistics.median(out)

    p = {}
    h = torch.empty(1 << 30, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    p["h2d_GBps"] = (1 << 30) / timed_copy(d, h, reps) / 1e6
    p["d2h_GBps"] = (1 << 30) / timed_copy(h, d, reps) / 1e6
    del h, d
    dd = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
    ds = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
    # HBM moves all-zero data measurably faster than random data on this part
    # (an 80k gather of zeroed blocks: ~6 % faster), so the probe source holds
    # the same seeded N(0,1) bf16 stream the KV cache does.
    import kvsynth
    kvsynth.fill_device(ds, 1, kvsynth.image_stream(9))
    torch.cuda.synchronize()
    p["d2d_copy_GBps_rw"] = 2 * (4 << 30) / timed_copy(dd, ds, 5) / 1e6

    # The slab mover's own shape on contiguous memory: reading only, writing
    # only (a fixed pattern), copying (kvx_probe_stream), 4 GiB each, median of 5.
    import paper_2609_11744_amd as kvx

    def timed_probe(mode, n):
        out = []
        for _ in range(n):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            kvx.kvx_probe_stream(ds if mode != 1 else None, dd if mode != 0 else None, 4 << 30, mode)
            b.record()
            b.synchronize()
            out.append(a.elapsed_time(b))
        return statistics.median(out)

    p["hbm_read_GBps"] = (4 << 30) / timed_probe(0, 5) / 1e6
    p["hbm_write_GBps"] = (4 << 30) / timed_probe(1, 5) / 1e6
    p["hbm_copy_GBps_rw"] = 2 * (4 << 30) / timed_probe(2, 5) / 1e6
    del dd, ds
    torch.cuda.empty_cache()
    log(f"probes: {p}")
    return p


_HOLD = {"cycles": None}
HOLD_US = 200.0


def hold_stream():
    """Keep the current stream busy for about HOLD_US microseconds (a spin
    kernel), so that the host-side launch of the call enqueued next overlaps
    it and events recorded around that call time its device execution only.
    With the GPU idle when a timed call starts, its events also count the
    call's host-side launch: about 1 % of a 3.3 ms kernel, 4 % of the
    0.46 ms one-head shard gather."""
    import torch

    sleep = getattr(torch.cuda, "_sleep", None)
    if sleep is None:  # no spin kernel in this torch: calls are timed from idle
        _HOLD["cycles"] = 0
        return
    if _HOLD["cycles"] is None:
        torch.cuda._sleep(1000)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = 4_000_000
        a.record()
        torch.cuda._sleep(n)
        b.record()
        b.synchronize()
        per_us = n / max(a.elapsed_time(b) * 1e3, 1.0)
        _HOLD["cycles"] = max(int(per_us * HOLD_US), 1)
    torch.cuda._sleep(_HOLD["cycles"])


def event_ms(fn, reps, hold=True):
    """Device time of fn() per call (ms), HIP events on the current stream;
    with hold, the stream is busy while fn is enqueued (hold_stream)."""
    import torch

    out = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if hold:
            hold_stream()
        a.record()
        fn()
        b.record()
        b.synchronize()
        out.append(a.elapsed_time(b))
    return out


def fill_cache(cache, seed, role):
    import kvsynth

    for l in range(cache.num_layers):
        kvsynth.fill_device(cache.k[l], seed, kvsynth.cache_stream(role, l, 0))
        kvsynth.fill_device(cache.v[l], seed, kvsynth.cache_stream(role, l, 1))


def base_record(args, metric, unit, value, ms_per_step, config, higher=True):
    return {"metric": metric, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": higher,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded N(0,1) bf16 KV, seeded random block ids)",
            "config": config}


# ---- default: 8B-shaped cache, 80,000-token prefix ------------------------------------

def run_80k(args):
    import numpy as np
    import torch

    import kvsynth
    import paper_2609_11744_amd as kvx

    dev = torch.device("cuda:0")
    L, BS, H, D, E = 32, 16, args.kv_heads, 128, 2
    if H < 1 or 8 % H:
        raise SystemExit("--kv-heads must divide the 8B shape's 8 KV heads")
    NB, n, ct = args.num_blocks, args.prefix_blocks, args.chunk_tokens
    if 3 * n > NB:
        raise SystemExit("pool too small for three disjoint prefixes")
    slab = BS * H * D * E
    payload = n * L * 2 * slab
    log(f"workload: 8B-shaped cache {NB} blocks ({NB * L * 2 * slab / 1e9:.1f} GB), "
        f"prefix {n} blocks = {n * BS} tokens, payload {payload / 1e9:.3f} GB")

    layout = {"nhd": kvx.KVX_LAYOUT_NHD, "hnd": kvx.KVX_LAYOUT_HND,
              "paged_attn": kvx.KVX_LAYOUT_PAGED_ATTN}[args.layout]
    cache = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev, layout=layout)
    fill_cache(cache, args.seed, kvsynth.ROLE_SRC)
    perm = np.random.default_rng(args.seed).permutation(NB).astype(np.int32)
    bt_src = torch.from_numpy(perm[:n].copy()).to(dev)
    bt_dst = torch.from_numpy(perm[n:2 * n].copy()).to(dev)
    bt_rst = torch.from_numpy(perm[2 * n:3 * n].copy()).to(dev)
    packed = torch.empty(payload, dtype=torch.uint8, device=dev)
    t0 = time.time()
    image = kvx.PinnedBuffer(payload)
    kvsynth.fill_host(image.array, args.seed, kvsynth.image_stream(1), threads=16)
    log(f"pinned image {payload / 1e9:.2f} GB ready in {time.time() - t0:.1f} s")
    ring = kvx.StagingRing(dev, args.slots, args.slot_mib << 20)
    ring.bind(cache, 0, L, n, ct, image, fill_threads=args.fill_threads)
    torch.cuda.synchronize()
    probe = probes(dev, args.probe_reps)

    def step(record):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        # the gather is enqueued while the stream is busy, so the events time
        # the device work of both calls (the scatter is enqueued while the
        # gather runs)
        hold_stream()
        e[0].record()
        kvx.kvx_gather_blocks(cache, 0, L, bt_src, n, ct, packed)
        e[1].record()
        kvx.kvx_scatter_blocks(cache, 0, L, bt_dst, n, ct, packed)
        e[2].record()
        # The restore is timed as its own phase, from its first fill to its last
        # scatter: the gather and scatter above finish first, so its pipeline
        # does not queue behind them.
        e[2].synchronize()
        t_r = time.perf_counter()
        kvx.kvx_restore_from_staging(ring, bt_rst)
        e[3].record()
        e[3].synchronize()
        restore_ms = (time.perf_counter() - t_r) * 1e3
        if record is not None:
            record["gather_ms"].append(e[0].elapsed_time(e[1]))
            record["scatter_ms"].append(e[1].elapsed_time(e[2]))
            record["restore_ms"].append(restore_ms)
            record["restore_dev_ms"].append(e[2].elapsed_time(e[3]))
            st = ring.stats()
            record["fill_ms"].append(st["fill_ms"])
            record["wait_fill_ms"].append(st["wait_fill_ms"])

    for _ in range(args.warmup):
        step(None)
    kvx.kvx_check()
    rec = {k: [] for k in ("gather_ms", "scatter_ms", "restore_ms", "restore_dev_ms", "fill_ms",
                           "wait_fill_ms")}
    torch.cuda.synchronize()
    t_begin = time.perf_counter()
    for _ in range(args.steps):
        step(rec)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_begin) * 1e3
    kvx.kvx_check()
    log("timed steps done")
    # the same calls timed from an idle GPU: the events then also count each
    # call's host-side launch
    launch_g = event_ms(lambda: kvx.kvx_gather_blocks(cache, 0, L, bt_src, n, ct, packed), 3,
                        hold=False)
    launch_s = event_ms(lambda: kvx.kvx_scatter_blocks(cache, 0, L, bt_dst, n, ct, packed), 3,
                        hold=False)
    kvx.kvx_check()
    timeline = restore_timeline(args, ring, bt_rst)
    offload = offload_leg(args, dev, cache, L, ct, n, bt_src, image, probe)
    sweep = sweep_32k(args, cache, L, perm, packed, slab, args.sweep_reps) \
        if H == 8 and args.sweep_reps > 0 else None

    med = {k: statistics.median(v) for k, v in rec.items()}
    mean_g = statistics.mean(rec["gather_ms"])
    mean_s = statistics.mean(rec["scatter_ms"])
    rw = 2 * payload
    gs_GBps = 2 * rw / ((sum(rec["gather_ms"]) + sum(rec["scatter_ms"])) / args.steps) / 1e6
    gather_GBps = rw / mean_g / 1e6
    scatter_GBps = rw / mean_s / 1e6
    restore_GBps = payload / med["restore_ms"] / 1e6
    gate = gate_from_rate(restore_GBps, L, H, D, E) if H == 8 else None
    cpu = None if args.no_cpu_baseline else cpu_baseline(args, L, BS, H, D, E, perm)
    traffic = None
    if GATHER_TRAFFIC["kernels_sha256"] == kernels_sha256() and args.layout in GATHER_TRAFFIC and \
            (args.num_blocks, args.prefix_blocks, args.chunk_tokens, H) == (20000, 5000, 256, 8):
        traffic = sum(GATHER_TRAFFIC[args.layout])

    out = base_record(
        args, "KV gather/scatter GB/s & % HBM peak; 80k-token prefix restore ms",
        "GB/s", round(gs_GBps, 1), round(wall_ms / args.steps, 3),
        {"workload": "llama-3-8b-shaped paged KV, 80k-token prefix (5000 blocks), "
                     "256-token chunks, 4 x 64 MiB pinned staging ring" +
                     ("" if H == 8 else f"; one GPU's share under tensor parallelism over KV "
                                        f"heads: {H} of 8 heads (tp = {8 // H})"),
         "num_blocks": NB, "prefix_tokens": n * BS, "chunk_tokens": ct, "kv_heads": H,
         "cache_layout": args.layout, "slots": args.slots, "slot_mib": args.slot_mib,
         "fill_threads": args.fill_threads, "parallelism": "single GPU"})
    out.update({
        "pct_hbm_peak": round(100 * gs_GBps / HBM_PEAK_GBPS, 2),
        "gather_GBps_rw": round(gather_GBps, 1),
        "scatter_GBps_rw": round(scatter_GBps, 1),
        "gather_ms": round(mean_g, 4),
        "scatter_ms": round(mean_s, 4),
        "gather_ms_stats": ms_stats(rec["gather_ms"]),
        "scatter_ms_stats": ms_stats(rec["scatter_ms"]),
        "timing": (f"device time of each call: HIP events on its stream, the call enqueued "
                   f"behind a {HOLD_US:.0f} us spin kernel so that its host-side launch is "
                   f"not counted; launch_inclusive: the same calls timed from an idle GPU"
                   if _HOLD["cycles"] else "HIP events on each call's stream from an idle GPU "
                   "(no spin kernel in this torch): the host-side launch is counted"),
        "launch_inclusive": {"gather_ms": ms_stats(launch_g), "scatter_ms": ms_stats(launch_s)},
        "walks": {"gather": kvx.kvx_copy_walk(cache, 0, L, n, ct, True),
                  "scatter": kvx.kvx_copy_walk(cache, 0, L, n, ct, False)},
        "restore_ms": round(med["restore_ms"], 3),
        "restore_GBps": round(restore_GBps, 2),
        "restore_frac_of_h2d": round(restore_GBps / probe["h2d_GBps"], 4),
        "h2d_copies": copies_desc(ring.stats()),
        "restore_breakdown_ms": {"fill_thread_sum": round(med["fill_ms"], 2),
                                 "enqueue_wait_for_fill": round(med["wait_fill_ms"], 2),
                                 "device_span": round(med["restore_dev_ms"], 2)},
        "restore_timeline": timeline,
        "offload": offload,
        "sweep_32k": sweep,
        "gate": gate,
        "probes": {k: round(v, 2) for k, v in probe.items()},
        "roofline": {"bound": "hbm",
                     "kernel": "gather (copy_units_kernel<true, false, layout %s>)" % args.layout,
                     "achieved": round(gather_GBps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(gather_GBps / HBM_PEAK_GBPS, 4),
                     "traffic": traffic, "algorithmic_bytes": rw,
                     "copy_ceiling_GBps": round(probe["hbm_copy_GBps_rw"], 1),
                     "frac_of_copy_ceiling": round(gather_GBps / probe["hbm_copy_GBps_rw"], 4)},
        "cpu_baseline": cpu,
    })
    print(json.dumps(out), flush=True)
    ring.close()
    image.free()


def restore_timeline(args, ring, bt_rst):
    """One more restore, outside the timed steps, with the ring's timeline on
    (kvx_ring_set_trace): the counters it yields (host-to-device busy time
    and gaps, per-piece fill, copy and scatter times), and with --trace-out
    the timeline itself as Chrome trace-event JSON."""
    import torch

    import paper_2609_11744_amd as kvx

    ring.set_trace(True)
    try:
        t0 = time.perf_counter()
        kvx.kvx_restore_from_staging(ring, bt_rst)
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t0) * 1e3
        ev = ring.trace()
    finally:
        ring.set_trace(False)
    if args.trace_out:
        with open(args.trace_out, "w") as f:
            json.dump(kvx.trace_chrome(ev, name="restore, 80k-token prefix"), f)
    summary = timeline_summary(ev)
    summary["restore_ms_traced"] = round(wall_ms, 3)
    log(f"restore timeline: {summary}")
    return summary


def timeline_summary(ev):
    """Counters of a restore timeline: pieces, the host-to-device copies' busy
    time (union of their intervals), span and idle gaps, their rate while
    busy, the median piece's fill (first fill start to last fill end), copy
    and scatter times, and how long the first copy waited from the first fill
    and the last scatter ran past the last copy."""
    by = {}
    for e in ev:
        by.setdefault(e["kind"], []).append(e)
    h2d = sorted(by.get("h2d", []), key=lambda e: e["t0_ns"])
    if not h2d:
        return {"pieces": 0}
    busy, end, gaps = 0, None, []
    for e in h2d:
        if end is None or e["t0_ns"] >= end:
            if end is not None:
                gaps.append(e["t0_ns"] - end)
            busy += e["t1_ns"] - e["t0_ns"]
            end = e["t1_ns"]
        elif e["t1_ns"] > end:
            busy += e["t1_ns"] - end
            end = e["t1_ns"]
    fills = {}
    for e in by.get("fill", []):
        a, b = fills.get(e["piece"], (e["t0_ns"], e["t1_ns"]))
        fills[e["piece"]] = (min(a, e["t0_ns"]), max(b, e["t1_ns"]))
    scat = sorted(by.get("scatter", []), key=lambda e: e["t0_ns"])
    first = min((a for a, _ in fills.values()), default=h2d[0]["t0_ns"])
    return {
        "pieces": len(h2d),
        "h2d_busy_ms": round(busy / 1e6, 3),
        "h2d_span_ms": round((h2d[-1]["t1_ns"] - h2d[0]["t0_ns"]) / 1e6, 3),
        "h2d_idle_ms": round(sum(gaps) / 1e6, 3),
        "h2d_max_gap_us": round(max(gaps, default=0) / 1e3, 1),
        "h2d_GBps_while_busy": round(sum(e["bytes"] for e in h2d) / busy, 2) if busy else None,
        "piece_fill_ms_median": round(statistics.median(b - a for a, b in fills.values()) / 1e6,
                                      3) if fills else None,
        "piece_h2d_ms_median": round(statistics.median(e["t1_ns"] - e["t0_ns"] for e in h2d)
                                     / 1e6, 3),
        "piece_scatter_us_median": round(statistics.median(e["t1_ns"] - e["t0_ns"] for e in scat)
                                         / 1e3, 1) if scat else None,
        "first_h2d_after_first_fill_ms": round((h2d[0]["t0_ns"] - first) / 1e6, 3),
        "last_scatter_after_last_h2d_us": round((scat[-1]["t1_ns"] - h2d[-1]["t1_ns"]) / 1e3, 1)
        if scat else None,
    }


def ms_stats(v):
    """Median, min and mean of event-timed milliseconds, and how many."""
    return {"median": round(statistics.median(v), 4), "min": round(min(v), 4),
            "mean": round(statistics.mean(v), 4), "n": len(v)}


def sweep_32k(args, cache, L, perm, packed, slab, reps=5):
    """The granularity sweep's gather and scatter on the same cache, outside
    the timed steps: a 32,768-token prefix (the first 2,048 of the seeded
    block permutation; scatter into the next 2,048) in chunks of 16, 64, 256
    and 1,024 tokens, each timed with events (median of reps)."""
    import torch

    import paper_2609_11744_amd as kvx

    n = 2048
    payload = n * L * 2 * slab
    src = torch.from_numpy(perm[:n].copy()).to(cache.device)
    dst = torch.from_numpy(perm[n:2 * n].copy()).to(cache.device)
    rows = []
    for ct in (16, 64, 256, 1024):
        g = event_ms(lambda: kvx.kvx_gather_blocks(cache, 0, L, src, n, ct, packed), reps + 1)[1:]
        sc = event_ms(lambda: kvx.kvx_scatter_blocks(cache, 0, L, dst, n, ct, packed), reps + 1)[1:]
        rows.append({"chunk_tokens": ct,
                     "gather_GBps_rw": round(2 * payload / statistics.median(g) / 1e6, 1),
                     "scatter_GBps_rw": round(2 * payload / statistics.median(sc) / 1e6, 1),
                     "gather_pct_hbm_peak": round(100 * 2 * payload / statistics.median(g) / 1e6
                                                  / HBM_PEAK_GBPS, 2),
                     "scatter_pct_hbm_peak": round(100 * 2 * payload / statistics.median(sc) / 1e6
                                                   / HBM_PEAK_GBPS, 2),
                     "gather_ms": ms_stats(g), "scatter_ms": ms_stats(sc),
                     "walks": {"gather": kvx.kvx_copy_walk(cache, 0, L, n, ct, True),
                               "scatter": kvx.kvx_copy_walk(cache, 0, L, n, ct, False)}})
    kvx.kvx_check()
    log(f"32k sweep: {[(r['chunk_tokens'], r['gather_pct_hbm_peak'], r['scatter_pct_hbm_peak']) for r in rows]}")
    return {"prefix_tokens": n * 16, "payload_bytes": payload, "reps": reps, "rows": rows}


# A stated synthetic calibration for the gate of an 8B-shaped model (no model
# runs here): cold TTFT 0.012 + 1.4e-5 x + 2.2e-10 x^2 s and the cache-hit
# path's non-transfer part 0.010 + 1.0e-7 x s, at knots from 1k to 128k tokens.
GATE_KNOTS = [1024.0, 4096.0, 8192.0, 16384.0, 32768.0, 65536.0, 131072.0]
GATE_COLD = [0.012 + 1.4e-5 * x + 2.2e-10 * x * x for x in GATE_KNOTS]
GATE_BASE = [0.010 + 1.0e-7 * x for x in GATE_KNOTS]


def gate_from_rate(restore_GBps, L, H, D, E):
    """The break-even gate of the pinned-host staging tier fed by the restore
    rate this run measured (Secs. 5.2, 6.6), on the synthetic curves above:
    the tier's threshold and the bandwidth a path must sustain at 1k, 8k and
    80k tokens; also for a tier ten and a hundred times slower."""
    from paper_2609_11744_amd import breakeven as be
    import paper_2609_11744_amd as kvx

    bpt = kvx.kvx_bytes_per_token(L, H, D, E)
    cold, base = be.Curve(GATE_KNOTS, GATE_COLD), be.Curve(GATE_KNOTS, GATE_BASE)
    # the required bandwidth depends on the curves only (the transfer the hit
    # path adds is credited back), so it is computed once, at the measured rate
    hit = be.hit_curve_from_restore(base, bpt, restore_GBps)
    copy = be.Curve(GATE_KNOTS, [x * bpt / (restore_GBps * 1e9) for x in GATE_KNOTS])
    need = {d: be.required_GBps(cold, hit, copy, d, bpt) for d in (1024, 8192, 81920)}
    out = {"curves": "synthetic: cold 0.012 + 1.4e-5 x + 2.2e-10 x^2 s, hit non-transfer "
                     "0.010 + 1.0e-7 x s (x tokens), knots 1k..128k",
           "bytes_per_token": bpt, "granularity_tokens": 256,
           "required_GBps": {str(d): round(v, 3) for d, v in need.items()}, "tiers": []}
    for name, rate in (("staging (measured)", restore_GBps), ("10x slower", restore_GBps / 10),
                       ("100x slower", restore_GBps / 100)):
        out["tiers"].append({
            "tier": name, "restore_GBps": round(rate, 3),
            "threshold_tokens": be.tier_threshold(cold, base, bpt, rate, 131072, 256),
            "sustains_required_at": [d for d, v in need.items() if rate >= v]})
    return out


def offload_leg(args, dev, cache, L, ct, n, bt_src, image, probe):
    """The store direction at the same size: gather of the prefix blocks into
    ring slots and D2H into host chunks (the pinned restore image is reused as
    the sink once the timed steps are done), timed separately after them."""
    import torch

    import paper_2609_11744_amd as kvx

    if args.offload_reps <= 0:
        return None
    BS = cache.block_size
    bpc = ct // BS
    per_block = image.nbytes // n
    sinks = [(image.array[b * per_block:min(n, b + bpc) * per_block], b, min(bpc, n - b))
             for b in range(0, n, bpc)]
    ring = kvx.StagingRing(dev, args.slots, args.slot_mib << 20)
    try:
        ring.bind_offload(cache, 0, L, ct, sinks, drain_threads=args.fill_threads)
        times, drain, wait, st = [], [], [], {}
        kvx.kvx_offload_to_staging(ring, bt_src)  # warm-up
        for _ in range(args.offload_reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            kvx.kvx_offload_to_staging(ring, bt_src)  # returns once every byte is in the sinks
            times.append(time.perf_counter() - t0)
            st = ring.stats()
            drain.append(st["fill_ms"])
            wait.append(st["wait_fill_ms"])
        kvx.kvx_check()
        deferred = deferred_store(ring, bt_src, dev, statistics.median(times))
    finally:
        ring.close()
    t = statistics.median(times)
    gbps = image.nbytes / t / 1e9
    log("offload leg done")
    return {"offload_ms": round(t * 1e3, 3), "offload_GBps": round(gbps, 2),
            "offload_frac_of_d2h": round(gbps / probe["d2h_GBps"], 4),
            "reps": args.offload_reps,
            "d2h_copies": copies_desc(st),
            "breakdown_ms": {"drain_thread_sum": round(statistics.median(drain), 2),
                             "wait_for_drain": round(statistics.median(wait), 2)},
            "deferred_store": deferred}


def deferred_store(ring, bt_src, dev, offload_s):
    """The store deferred to the next iteration (kvx_offload_begin, gathers on a
    side stream) beside a compute-bound stand-in for that iteration's forward
    pass (bf16 8192^3 GEMMs on another stream, as many as take about as long as
    the offload alone). overlap = time hidden / the shorter of the two alone
    (1: the shorter one is fully hidden)."""
    import torch

    import paper_2609_11744_amd as kvx

    side, comp = torch.cuda.Stream(), torch.cuda.Stream()
    a = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    b = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    c = torch.empty(8192, 8192, device=dev, dtype=torch.bfloat16)

    def gemms(k):
        with torch.cuda.stream(comp):
            for _ in range(k):
                torch.matmul(a, b, out=c)

    gemms(5)
    comp.synchronize()
    t0 = time.perf_counter()
    gemms(20)
    comp.synchronize()
    per = (time.perf_counter() - t0) / 20
    k = max(1, int(offload_s / per))
    alone = []
    for _ in range(3):
        t0 = time.perf_counter()
        gemms(k)
        comp.synchronize()
        alone.append(time.perf_counter() - t0)
    both, during = [], []
    for _ in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        kvx.kvx_offload_begin(ring, bt_src, stream=side)
        t1 = time.perf_counter()
        gemms(k)
        comp.synchronize()
        during.append(time.perf_counter() - t1)
        kvx.kvx_offload_wait(ring)
        both.append(time.perf_counter() - t0)
    kvx.kvx_check(side)
    t_c, t_b = statistics.median(alone), statistics.median(both)
    flops = 2.0 * 8192 ** 3 * k
    return {"gemms": k, "compute_alone_ms": round(t_c * 1e3, 2),
            "offload_alone_ms": round(offload_s * 1e3, 2),
            "both_ms": round(t_b * 1e3, 2),
            "compute_during_store_ms": round(statistics.median(during) * 1e3, 2),
            "compute_TFLOPs_alone": round(flops / t_c / 1e12, 1),
            "overlap": round((t_c + offload_s - t_b) / min(t_c, offload_s), 3)}


def cpu_baseline(args, L, BS, H, D, E, perm):
    """Time the oracle (plain C slab memcpy) gathering and scattering a bounded
    sample of the same workload on this host: once on one thread, and once as
    independent calls on disjoint chunk ranges, one per core (the oracle
    itself is unchanged; its C calls release the GIL)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import kvsynth
    import oracle

    ct = args.chunk_tokens
    bpc = ct // BS
    m = args.cpu_sample_blocks
    shape = oracle.Shape(L, args.num_blocks, BS, H, D, E)
    ids = perm[:m]
    dst_ids = perm[args.prefix_blocks:args.prefix_blocks + m]
    k, v = oracle.new_mirror(shape)
    offs = ids.astype(np.uint64) * np.uint64(shape.slab_bytes)
    for l in range(L):
        kvsynth.fill_ranges(k[l], offs, shape.slab_bytes, args.seed,
                            kvsynth.cache_stream(kvsynth.ROLE_SRC, l, 0), threads=16)
        kvsynth.fill_ranges(v[l], offs, shape.slab_bytes, args.seed,
                            kvsynth.cache_stream(kvsynth.ROLE_SRC, l, 1), threads=16)
    out = np.empty(oracle.packed_bytes(shape, 0, L, m), dtype=np.uint8)
    per_block = oracle.packed_bytes(shape, 0, L, 1)

    def one(lo, hi):  # chunk-aligned block range [lo, hi): its image is out[lo*pb, hi*pb)
        part = out[lo * per_block:hi * per_block]
        oracle.gather(shape, k, v, 0, L, ids[lo:hi], ct, out=part)
        oracle.scatter(shape, k, v, 0, L, dst_ids[lo:hi], ct, part)

    one(0, m)  # touch every page once
    times1 = []
    for _ in range(3):
        t0 = time.perf_counter()
        one(0, m)
        times1.append(time.perf_counter() - t0)
    # every core of the process's affinity mask, unless OMP_NUM_THREADS says
    # the process's CPU share is smaller (on a machine shared by several GPUs it
    # is set to one GPU's share of the host, 16 threads)
    affinity = len(os.sched_getaffinity(0))
    share = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    cores = max(1, min(affinity, share) if share > 0 else affinity)
    nch = (m + bpc - 1) // bpc
    bounds = [min(m, (nch * i // cores) * bpc) for i in range(cores + 1)]
    timesn = []
    with ThreadPoolExecutor(cores) as ex:
        for _ in range(3):
            t0 = time.perf_counter()
            list(ex.map(lambda i: one(bounds[i], bounds[i + 1]), range(cores)))
            timesn.append(time.perf_counter() - t0)
    rw = 2 * 2 * out.nbytes
    one_core = rw / statistics.median(times1) / 1e9

    def rates(times):
        return {"median": round(rw / statistics.median(times) / 1e9, 2),
                "mean": round(rw / statistics.mean(times) / 1e9, 2),
                "min": round(rw / max(times) / 1e9, 2), "max": round(rw / min(times) / 1e9, 2)}

    cpu_model, numa_nodes = host_cpu()
    return {"value": round(rw / statistics.median(timesn) / 1e9, 2), "unit": "GB/s",
            "cores": cores, "kind": "oracle",
            "sample": f"gather + scatter of {m} of the {args.prefix_blocks} prefix blocks "
                      f"({out.nbytes / 1e9:.2f} GB payload each way, GB/s of bytes read + "
                      f"written), 3 repetitions; {cores} threads each running the C oracle on "
                      f"a disjoint chunk range; single thread: {one_core:.2f} GB/s",
            "rates_GBps": {"threads": rates(timesn), "single_thread": rates(times1)},
            "affinity_cores": affinity, "omp_num_threads": share or None,
            "cpu_model": cpu_model, "numa_nodes": numa_nodes}


def host_cpu():
    """The host's CPU model name and NUMA node count (None where unknown)."""
    import glob

    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    nodes = len(glob.glob("/sys/devices/system/node/node[0-9]*")) or None
    return model, nodes


# ---- 32k-token granularity sweep --------------------------------------------------------

def run_sweep(args):
    import numpy as np
    import torch

    import kvsynth
    import paper_2609_11744_amd as kvx

    dev = torch.device("cuda:0")
    L, BS, H, D, E = 32, 16, 8, 128, 2
    NB, n = args.num_blocks, 2048
    slab = BS * H * D * E
    payload = n * L * 2 * slab
    cache = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev)
    fill_cache(cache, args.seed, kvsynth.ROLE_SRC)
    perm = np.random.default_rng(args.seed).permutation(NB).astype(np.int32)
    bt_src = torch.from_numpy(perm[:n].copy()).to(dev)
    bt_dst = torch.from_numpy(perm[n:2 * n].copy()).to(dev)
    packed = torch.empty(payload, dtype=torch.uint8, device=dev)
    image = kvx.PinnedBuffer(payload)
    kvsynth.fill_host(image.array, args.seed, kvsynth.image_stream(2), threads=16)
    probe = probes(dev, args.probe_reps)
    reps = max(args.steps, 3)
    rows = []
    t_begin = time.perf_counter()
    for ct in (16, 64, 256, 1024):
        g = event_ms(lambda: kvx.kvx_gather_blocks(cache, 0, L, bt_src, n, ct, packed), reps)
        s = event_ms(lambda: kvx.kvx_scatter_blocks(cache, 0, L, bt_dst, n, ct, packed), reps)
        row = {"chunk_tokens": ct, "gather_GBps_rw": round(2 * payload / statistics.median(g) / 1e6, 1),
               "scatter_GBps_rw": round(2 * payload / statistics.median(s) / 1e6, 1), "restore": []}
        for slots in (2, 4, 8):
            ring = kvx.StagingRing(dev, slots, args.slot_mib << 20)
            ring.bind(cache, 0, L, n, ct, image, fill_threads=args.fill_threads)
            times = []
            for i in range(reps + 1):
                t0 = time.perf_counter()
                kvx.kvx_restore_from_staging(ring, bt_dst)
                torch.cuda.synchronize()
                if i:
                    times.append((time.perf_counter() - t0) * 1e3)
            ms = statistics.median(times)
            row["restore"].append({"slots": slots, "ms": round(ms, 3),
                                   "GBps": round(payload / ms / 1e6, 2),
                                   "frac_of_h2d": round(payload / ms / 1e6 / probe["h2d_GBps"], 4),
                                   "pieces": ring.stats()["pieces"]})
            ring.close()
        rows.append(row)
        log(f"chunk {ct}: {row}")
    extras = {}
    # Block-id locality: the same 256-token-chunk gather / scatter with the
    # source and destination ids each sorted ascending instead of random.
    bs_src = torch.sort(bt_src).values.contiguous()
    bs_dst = torch.sort(bt_dst).values.contiguous()
    g = event_ms(lambda: kvx.kvx_gather_blocks(cache, 0, L, bs_src, n, 256, packed), reps)
    s = event_ms(lambda: kvx.kvx_scatter_blocks(cache, 0, L, bs_dst, n, 256, packed), reps)
    extras["sorted_ids_chunk256"] = {
        "gather_GBps_rw": round(2 * payload / statistics.median(g) / 1e6, 1),
        "scatter_GBps_rw": round(2 * payload / statistics.median(s) / 1e6, 1)}
    # Transfer granularity: one 16-token chunk (2 MiB) per host-link copy
    # (4 slots of 2 MiB) against the same chunks packed into 64 MiB slots.
    for name, slot_bytes in (("one_chunk_per_copy", 2 << 20), ("packed_64MiB_slots", 64 << 20)):
        ring = kvx.StagingRing(dev, 4, slot_bytes)
        ring.bind(cache, 0, L, n, 16, image, fill_threads=args.fill_threads)
        times = []
        for i in range(reps + 1):
            t0 = time.perf_counter()
            kvx.kvx_restore_from_staging(ring, bt_dst)
            torch.cuda.synchronize()
            if i:
                times.append((time.perf_counter() - t0) * 1e3)
        ms = statistics.median(times)
        extras[name] = {"chunk_tokens": 16, "slots": 4, "slot_bytes": slot_bytes,
                        "pieces": ring.stats()["pieces"], "restore_ms": round(ms, 3),
                        "frac_of_h2d": round(payload / ms / 1e6 / probe["h2d_GBps"], 4)}
        ring.close()
    log(f"extras: {extras}")
    kvx.kvx_check()
    wall = (time.perf_counter() - t_begin) * 1e3
    best = max(min(r["gather_GBps_rw"], r["scatter_GBps_rw"]) for r in rows)
    out = base_record(args, "KV gather/scatter GB/s across transfer chunk sizes (32k-token prefix)",
                      "GB/s", best, round(wall, 1),
                      {"workload": "llama-3-8b-shaped paged KV, 32k-token prefix (2048 blocks) of "
                                   "a 20000-block pool; chunks 16/64/256/1024; rings 2/4/8 x 64 MiB",
                       "num_blocks": NB, "prefix_tokens": n * BS, "parallelism": "single GPU"})
    out["ms_per_step_note"] = "wall time of the whole sweep"
    out.update({"sweep": rows, "extras": extras,
                "probes": {k: round(v, 2) for k, v in probe.items()}})
    print(json.dumps(out), flush=True)
    image.free()


# ---- 70B-shaped batched step -------------------------------------------------------

def run_batch(args):
    import numpy as np
    import torch

    import kvsynth
    import kvsynth.prefix_tree as pt
    import paper_2609_11744_amd as kvx
    from paper_2609_11744_amd import step

    dev = torch.device("cuda:0")
    L, BS, H, D, E = 80, 16, 8, 128, 2
    reqs = pt.make_requests(5, n=64)
    plan = step.plan_step(reqs, BS, 256)
    NB = plan.restore_blocks + plan.offload_blocks + 64
    per_block = L * 2 * BS * H * D * E
    rb, ob = plan.restore_blocks * per_block, plan.offload_blocks * per_block
    log(f"70B batch: {len(plan.restore)} distinct missing chunks ({rb / 1e9:.1f} GB), "
        f"{plan.resident_hits} resident chunks, {plan.offload_blocks} new blocks "
        f"({ob / 1e9:.1f} GB); pool {NB} blocks")
    ids = np.random.default_rng(5).permutation(NB).astype(np.int32)
    rbt = torch.from_numpy(ids[:plan.restore_blocks].copy()).to(dev)
    obt = torch.from_numpy(ids[plan.restore_blocks:plan.restore_blocks + plan.offload_blocks]
                           .copy()).to(dev)
    cache = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev)
    fill_cache(cache, 5, kvsynth.ROLE_NEW)
    store = np.empty(rb, dtype=np.uint8)
    chunks = []
    for c in plan.restore:
        view = store[c.bt_offset * per_block:(c.bt_offset + c.n_blocks) * per_block]
        kvsynth.fill_host(view, 5, pt.chunk_stream(reqs[c.origin[0]].chunk_owner[c.origin[1]]),
                          threads=16)
        chunks.append((view, c.bt_offset, c.n_blocks))
    sink = np.ones(ob, dtype=np.uint8)  # touched up front: no page faults while draining
    sinks = [(sink[c.bt_offset * per_block:(c.bt_offset + c.n_blocks) * per_block],
              c.bt_offset, c.n_blocks) for c in plan.offload]
    probe = probes(dev, args.probe_reps)
    r_ring = kvx.StagingRing(dev, args.slots, args.slot_mib << 20)
    o_ring = kvx.StagingRing(dev, args.slots, args.slot_mib << 20)
    r_ring.bind_chunks(cache, 0, L, 256, chunks, fill_threads=args.fill_threads)
    o_ring.bind_offload(cache, 0, L, 256, sinks, drain_threads=args.fill_threads)
    s_r, s_o = torch.cuda.Stream(), torch.cuda.Stream()

    def one_step():
        """Both transfers run on the rings' own threads (kvx_restore_begin,
        kvx_offload_begin); this thread starts them and collects them. The
        restore is timed to its last scatter, the offload by its ring (from
        the start of its transfer until every destination holds its image)."""
        t = {}
        t0 = time.perf_counter()
        kvx.kvx_restore_begin(r_ring, rbt, stream=s_r)
        kvx.kvx_offload_begin(o_ring, obt, stream=s_o)
        kvx.kvx_restore_wait(r_ring, stream=s_r)
        s_r.synchronize()
        t["restore"] = time.perf_counter() - t0
        kvx.kvx_offload_wait(o_ring)
        t["step"] = time.perf_counter() - t0
        t["offload"] = o_ring.stats()["enqueue_ms"] / 1e3
        return t

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    recs = [one_step() for _ in range(args.steps)]
    kvx.kvx_check(s_r)
    kvx.kvx_check(s_o)
    med = {k: statistics.median(r[k] for r in recs) for k in recs[0]}
    # each leg alone, for comparison with the concurrent step
    alone = {"restore": [], "offload": []}
    for _ in range(2):
        t0 = time.perf_counter()
        kvx.kvx_restore_from_staging(r_ring, rbt, stream=s_r)
        s_r.synchronize()
        alone["restore"].append(time.perf_counter() - t0)
        t0 = time.perf_counter()
        kvx.kvx_offload_to_staging(o_ring, obt, stream=s_o)
        alone["offload"].append(time.perf_counter() - t0)
    kvx.kvx_check(s_r)
    kvx.kvx_check(s_o)
    alone = {k: min(v) for k, v in alone.items()}
    o_stats = o_ring.stats()
    r_stats = r_ring.stats()
    out = base_record(args, "KV staged restore GB/s (70B batched step, offload concurrent)", "GB/s",
                      round(rb / med["restore"] / 1e9, 2), round(med["step"] * 1e3, 2),
                      {"workload": "70b-shaped paged KV, 64 requests on a seeded prefix tree "
                                   "(log-uniform 1k-32k tokens, branching 1-4, 50% resident), "
                                   "256-token chunks, 2 rings of 4 x 64 MiB",
                       "distinct_missing_chunks": len(plan.restore),
                       "restore_blocks": plan.restore_blocks,
                       "offload_blocks": plan.offload_blocks,
                       "resident_chunks": plan.resident_hits, "parallelism": "single GPU"})
    out.update({"step_calls": "kvx_restore_begin / kvx_offload_begin from one thread, then "
                              "kvx_restore_wait / kvx_offload_wait",
                "restore_GBps": round(rb / med["restore"] / 1e9, 2),
                "restore_frac_of_h2d": round(rb / med["restore"] / 1e9 / (probe["h2d_GBps"]), 4),
                "offload_GBps": round(ob / med["offload"] / 1e9, 2),
                "offload_frac_of_d2h": round(ob / med["offload"] / 1e9 / probe["d2h_GBps"], 4),
                "restore_ms": round(med["restore"] * 1e3, 2),
                "offload_ms": round(med["offload"] * 1e3, 2),
                "link_GBps_both_ways": round((rb + ob) / med["step"] / 1e9, 2),
                "h2d_copies": copies_desc(r_stats), "d2h_copies": copies_desc(o_stats),
                "alone": {"restore_GBps": round(rb / alone["restore"] / 1e9, 2),
                          "offload_GBps": round(ob / alone["offload"] / 1e9, 2),
                          "offload_drain_thread_ms": round(o_stats["fill_ms"], 2),
                          "offload_wait_for_drain_ms": round(o_stats["wait_fill_ms"], 2)},
                "probes": {k: round(v, 2) for k, v in probe.items()}})
    print(json.dumps(out), flush=True)
    r_ring.close()
    o_ring.close()


# ---- storage tier: chunk files -----------------------------------------------------------

def run_files(args):
    """The 8B-shaped 32k-token prefix (2,048 blocks, 4 GiB) offloaded through a
    4 x 64 MiB ring into one file per 256-token chunk (128 files of 32 MiB,
    hash-addressed, flushed and published), then restored from the files into
    other blocks. Beside it, the device's own direct-I/O rates through the same
    engine from ordinary page-aligned memory (4 GiB as 32 MiB files)."""
    import shutil

    import numpy as np
    import torch

    import kvsynth
    import paper_2609_11744_amd as kvx

    dev = torch.device("cuda:0")
    L, BS, H, D, E = 32, 16, 8, 128, 2
    NB, n, ct = args.num_blocks, 2048, 256
    bpc = ct // BS
    per_block = 2 * L * BS * H * D * E
    payload = n * per_block
    root = os.path.abspath(args.tier_dir)
    shutil.rmtree(root, ignore_errors=True)
    cache = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev)
    fill_cache(cache, args.seed, kvsynth.ROLE_SRC)
    perm = np.random.default_rng(args.seed).permutation(NB).astype(np.int32)
    bt_src = torch.from_numpy(perm[:n].copy()).to(dev)
    bt_dst = torch.from_numpy(perm[n:2 * n].copy()).to(dev)
    chunks = [(kvx.kvx_chunk_path(root, "llama-3-8b-bf16", 0xA5A5A5A5A5A5A5A5 ^ (c * 0x9E3779B97F4A7C15)),
               c * bpc, bpc) for c in range(n // bpc)]
    reps = max(3, args.steps)
    try:
        # device probe: direct I/O from ordinary memory, same engine and depth
        buf = np.empty(payload, dtype=np.uint8)
        buf[:] = 7
        files = [(os.path.join(root, "probe", f"p{i:04d}.bin"), buf[i << 25:(i + 1) << 25], 0)
                 for i in range(payload >> 25)]
        t0 = time.perf_counter()
        kvx.kvx_write_files(files, io_depth=args.io_depth)
        w_dev = payload / (time.perf_counter() - t0) / 1e9
        t0 = time.perf_counter()
        kvx.kvx_read_files(files, io_depth=args.io_depth)
        r_dev = payload / (time.perf_counter() - t0) / 1e9
        shutil.rmtree(os.path.join(root, "probe"), ignore_errors=True)
        del buf
        ring = kvx.StagingRing(dev, args.slots, args.slot_mib << 20)
        t_off, t_res = [], []
        try:
            ring.bind_offload_files(cache, 0, L, ct, chunks, io_depth=args.io_depth)
            for i in range(reps):
                if i:  # later offloads write the same content and keep the published files
                    shutil.rmtree(os.path.join(root, "llama-3-8b-bf16"), ignore_errors=True)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                kvx.kvx_offload_to_staging(ring, bt_src)
                t_off.append(time.perf_counter() - t0)
            engine = ring.stats()["dma_engine"]
            ring.bind_files(cache, 0, L, ct, chunks, io_depth=args.io_depth)
            for _ in range(reps):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                kvx.kvx_restore_from_staging(ring, bt_dst)
                torch.cuda.synchronize()
                t_res.append(time.perf_counter() - t0)
            kvx.kvx_check()
        finally:
            ring.close()
        log("files done")
    finally:
        shutil.rmtree(root, ignore_errors=True)
    off = payload / statistics.median(t_off) / 1e9
    res = payload / statistics.median(t_res) / 1e9
    out = base_record(
        args, "KV restore from chunk files GB/s (32k-token prefix, storage tier)", "GB/s",
        round(res, 2), round(statistics.median(t_res) * 1e3, 2),
        {"workload": "llama-3-8b-shaped paged KV, 32k-token prefix (2048 blocks, 4 GiB) as 128 "
                     "chunk files of 256 tokens; 4 x 64 MiB ring",
         "num_blocks": NB, "prefix_tokens": n * BS, "chunk_tokens": ct, "slots": args.slots,
         "slot_mib": args.slot_mib, "io_depth": args.io_depth, "parallelism": "single GPU"})
    out.update({
        "restore_from_files_GBps": round(res, 2),
        "offload_to_files_GBps": round(off, 2),
        "restore_frac_of_device_read": round(res / r_dev, 4),
        "offload_frac_of_device_write": round(off / w_dev, 4),
        "probes": {"device_direct_read_GBps": round(r_dev, 2),
                   "device_direct_write_GBps": round(w_dev, 2)},
        "offload_d2h_engine_bit": engine, "reps": reps,
        "note": "ring files use buffered I/O (pinned slots cannot take direct transfers "
                "here), flushed before publication and dropped from the page cache after use"})
    print(json.dumps(out), flush=True)


def run_preload(args):
    """Preloading (Sec. 6.5) on the 8B-shaped 32k-token prefix stored as 128 chunk
    files of 32 MiB (4 GiB): the request path of a restore (from the call until
    the cache holds the prefix) when the files are read only on demand (the
    ring restoring straight from the files), when a preloader read them while
    the request waited (the path is then the host-to-device copy out of the
    preloader's pinned pool), and when the request starts halfway through the
    preload (waiting time half the demand restore)."""
    import shutil

    import numpy as np
    import torch

    import kvsynth
    import paper_2609_11744_amd as kvx

    dev = torch.device("cuda:0")
    L, BS, H, D, E = 32, 16, 8, 128, 2
    NB, n, ct = args.num_blocks, 2048, 256
    bpc = ct // BS
    per_block = 2 * L * BS * H * D * E
    payload = n * per_block
    chunk_bytes = bpc * per_block
    root = os.path.abspath(args.tier_dir)
    shutil.rmtree(root, ignore_errors=True)
    cache = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev)
    fill_cache(cache, args.seed, kvsynth.ROLE_SRC)
    perm = np.random.default_rng(args.seed).permutation(NB).astype(np.int32)
    bt_src = torch.from_numpy(perm[:n].copy()).to(dev)
    bt_dst = torch.from_numpy(perm[n:2 * n].copy()).to(dev)
    chunks = [(kvx.kvx_chunk_path(root, "llama-3-8b-bf16", 0x5A5A5A5A5A5A5A5A ^ (c * 0x9E3779B97F4A7C15)),
               c * bpc, bpc) for c in range(n // bpc)]
    paths = [c[0] for c in chunks]
    reps = max(3, args.steps)
    probe = probes(dev, 5)
    reserve = args.io_depth
    res = {"demand": [], "preloaded": [], "half": [], "half_overlapped": [], "pool_demand": []}
    read_s, mode_stats = [], {}
    try:
        ring = kvx.StagingRing(dev, args.slots, args.slot_mib << 20)
        try:
            ring.bind_offload_files(cache, 0, L, ct, chunks, io_depth=args.io_depth)
            kvx.kvx_offload_to_staging(ring, bt_src)
            # demand only: the ring reads the files as it restores
            ring.bind_files(cache, 0, L, ct, chunks, io_depth=args.io_depth)
            for _ in range(reps):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                kvx.kvx_restore_from_staging(ring, bt_dst)
                torch.cuda.synchronize()
                res["demand"].append(time.perf_counter() - t0)
            kvx.kvx_check()
            log("demand restores done")

            def request(pre):
                """The request path with a preloader: claim the images, restore
                them straight from the pool, drop the holds."""
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                imgs = pre.fetch(paths)
                ring.bind_chunks(cache, 0, L, ct, [(img, c[1], c[2]) for img, c in zip(imgs, chunks)],
                                 fill_threads=0)
                kvx.kvx_restore_from_staging(ring, bt_dst)
                torch.cuda.synchronize()
                dt = time.perf_counter() - t0
                pre.release(paths)
                return dt

            def request_overlapped(pre):
                """The request path through a ring bound to the preloader: the
                restore holds the files and copies each piece as soon as its
                files are staged, while the rest are still being read."""
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                ring.bind_preloaded(cache, 0, L, ct, pre, chunks)
                kvx.kvx_restore_from_staging(ring, bt_dst)
                torch.cuda.synchronize()
                return time.perf_counter() - t0

            half = statistics.median(res["demand"]) / 2
            for rep_i in range(reps):
                for mode in ("preloaded", "half", "half_overlapped", "pool_demand"):
                    pre = kvx.Preloader(len(paths) + reserve, chunk_bytes, io_depth=args.io_depth,
                                        reserve=reserve, pinned=True)
                    try:
                        t0 = time.perf_counter()
                        if mode != "pool_demand":
                            pre.hint(paths)  # the request is still waiting
                        if mode == "preloaded":
                            pre.wait_idle()
                            read_s.append(time.perf_counter() - t0)
                        elif mode != "pool_demand":
                            time.sleep(half)
                        if mode in ("preloaded", "half"):
                            res[mode].append(request(pre))
                        else:
                            res[mode].append(request_overlapped(pre))
                        mode_stats[mode] = pre.stats()
                    finally:
                        pre.close()
                log(f"preload repetition {rep_i + 1} of {reps} done")
            kvx.kvx_check()
        finally:
            ring.close()
        log("preload restores done")
    finally:
        shutil.rmtree(root, ignore_errors=True)
    med = {k: statistics.median(v) for k, v in res.items()}
    out = base_record(
        args, "KV restore request path ms with preloading (32k-token prefix, storage tier)", "ms",
        round(med["preloaded"] * 1e3, 2), round(med["preloaded"] * 1e3, 2),
        {"workload": "llama-3-8b-shaped paged KV, 32k-token prefix (2048 blocks, 4 GiB) as 128 "
                     "chunk files of 256 tokens; 4 x 64 MiB ring; preloader pool of 128 + "
                     "io_depth slots of 32 MiB",
         "num_blocks": NB, "prefix_tokens": n * BS, "chunk_tokens": ct, "io_depth": args.io_depth,
         "parallelism": "single GPU"}, higher=False)
    out.update({
        "request_path_ms": {k: round(v * 1e3, 2) for k, v in med.items()},
        "speedup_preloaded_vs_demand": round(med["demand"] / med["preloaded"], 2),
        "speedup_half_vs_demand": round(med["demand"] / med["half"], 2),
        "speedup_half_overlapped_vs_demand": round(med["demand"] / med["half_overlapped"], 2),
        "preloaded_restore_GBps": round(payload / med["preloaded"] / 1e9, 2),
        "preloaded_frac_of_h2d": round(payload / med["preloaded"] / 1e9 / probe["h2d_GBps"], 4),
        "demand_restore_GBps": round(payload / med["demand"] / 1e9, 2),
        "preload_read_GBps": round(payload / statistics.median(read_s) / 1e9, 2),
        "stats": mode_stats,
        "probes": {"h2d_GBps": round(probe["h2d_GBps"], 2)}, "reps": reps,
        "note": "each request path starts from files whose pages were dropped from the page "
                "cache; 'half' starts the request after half the demand restore time of "
                "preloading, so its fetch claims what is staged, joins what is being read and "
                "reads the rest on demand before the restore; 'half_overlapped' starts at the "
                "same time but restores through a ring bound to the preloader, copying each "
                "piece as soon as its files are staged; 'pool_demand' does the same with "
                "nothing hinted (every file read on demand, overlapped with the copies)"})
    print(json.dumps(out), flush=True)


# ---- allocation placement -------------------------------------------------------------

def run_placements(args):
    """The default workload's gather and scatter (80k-token prefix, 256-token
    chunks, the same seeded ids) on every (cache, packed buffer) pair of
    --caches caches and --packed packed buffers, all allocated up front and
    alive together: each pair sits at other physical addresses, and the spread
    of the rates over the pairs is the placement's share of a run-to-run
    spread (the code and the ids are the same for every pair)."""
    import numpy as np
    import torch

    import kvsynth
    import paper_2609_11744_amd as kvx

    dev = torch.device("cuda:0")
    L, BS, H, D, E = 32, 16, args.kv_heads, 128, 2
    NB, n, ct = args.num_blocks, args.prefix_blocks, args.chunk_tokens
    slab = BS * H * D * E
    payload = n * L * 2 * slab
    need = args.caches * NB * L * 2 * slab + args.packed * payload
    free, _ = torch.cuda.mem_get_info()
    if need > 0.9 * free:
        raise SystemExit(f"{need / 1e9:.0f} GB of caches and packed buffers do not fit")
    perm = np.random.default_rng(args.seed).permutation(NB).astype(np.int32)
    bt_src = torch.from_numpy(perm[:n].copy()).to(dev)
    bt_dst = torch.from_numpy(perm[n:2 * n].copy()).to(dev)
    caches, packs = [], []
    for i in range(max(args.caches, args.packed)):
        if i < args.caches:
            c = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev)
            fill_cache(c, args.seed, kvsynth.ROLE_SRC)
            caches.append(c)
        if i < args.packed:
            packs.append(torch.empty(payload, dtype=torch.uint8, device=dev))
    torch.cuda.synchronize()
    reps = max(args.steps, 3)
    pct = lambda ms: 100 * 2 * payload / ms / 1e6 / HBM_PEAK_GBPS
    rows = []
    for ci, c in enumerate(caches):
        for pi, p in enumerate(packs):
            g = event_ms(lambda: kvx.kvx_gather_blocks(c, 0, L, bt_src, n, ct, p), reps)
            sc = event_ms(lambda: kvx.kvx_scatter_blocks(c, 0, L, bt_dst, n, ct, p), reps)
            rows.append({"cache": ci, "packed": pi,
                         "gather_pct_hbm_peak": round(pct(statistics.median(g)), 2),
                         "scatter_pct_hbm_peak": round(pct(statistics.median(sc)), 2)})
    kvx.kvx_check()
    log(f"placements: {[(r['cache'], r['packed'], r['gather_pct_hbm_peak'], r['scatter_pct_hbm_peak']) for r in rows]}")

    def spread(key):
        v = [r[key] for r in rows]
        return {"mean": round(statistics.mean(v), 2), "min": min(v), "max": max(v)}

    gs = spread("gather_pct_hbm_peak")
    ss = spread("scatter_pct_hbm_peak")
    mean_rate = (gs["mean"] + ss["mean"]) / 2 * HBM_PEAK_GBPS / 100
    out = base_record(
        args, "KV gather/scatter GB/s & % HBM peak over allocation placements", "GB/s",
        round(mean_rate, 1), None,
        {"workload": "llama-3-8b-shaped paged KV, 80k-token prefix (5000 blocks), 256-token "
                     f"chunks, on each of {args.caches} caches x {args.packed} packed buffers",
         "num_blocks": NB, "prefix_tokens": n * BS, "chunk_tokens": ct, "kv_heads": H,
         "caches": args.caches, "packed": args.packed, "parallelism": "single GPU"})
    out.update({"gather_pct_hbm_peak": gs, "scatter_pct_hbm_peak": ss, "pairs": rows,
                "reps_per_pair": reps,
                "note": "value: mean of the gather and scatter rates over the pairs; each "
                        "call timed as in the default workload (median of reps_per_pair)"})
    print(json.dumps(out), flush=True)


def run_layouts(args):
    """The default workload's gather and scatter with each cache read as the
    default (NHD), HND and paged-attention layouts. A layout only decides
    where a cache tensor's bytes belong, so one allocation serves all three
    (views of the same tensors, holding random data): on every (cache, packed
    buffer) pair the three layouts move equal bytes at equal addresses, and
    their difference is the layout's own cost, with the placement share of a
    run-to-run spread held fixed."""
    import numpy as np
    import torch

    import kvsynth
    import paper_2609_11744_amd as kvx

    dev = torch.device("cuda:0")
    L, BS, H, D, E = 32, 16, args.kv_heads, 128, 2
    NB, n, ct = args.num_blocks, args.prefix_blocks, args.chunk_tokens
    slab = BS * H * D * E
    payload = n * L * 2 * slab
    caches_n, packed_n = min(args.caches, 2), min(args.packed, 2)
    need = caches_n * NB * L * 2 * slab + packed_n * payload
    free, _ = torch.cuda.mem_get_info()
    if need > 0.9 * free:
        raise SystemExit(f"{need / 1e9:.0f} GB of caches and packed buffers do not fit")
    perm = np.random.default_rng(args.seed).permutation(NB).astype(np.int32)
    bt_src = torch.from_numpy(perm[:n].copy()).to(dev)
    bt_dst = torch.from_numpy(perm[n:2 * n].copy()).to(dev)
    x = 16 // E
    views = []
    for _ in range(caches_n):
        c = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev)
        fill_cache(c, args.seed, kvsynth.ROLE_SRC)
        views.append({
            "nhd": c,
            "hnd": kvx.PagedKVCache([t.view(NB, H, BS, D) for t in c.k],
                                    [t.view(NB, H, BS, D) for t in c.v], kvx.KVX_LAYOUT_HND),
            "paged_attn": kvx.PagedKVCache([t.view(NB, H, D // x, BS, x) for t in c.k],
                                           [t.view(NB, H, D, BS) for t in c.v],
                                           kvx.KVX_LAYOUT_PAGED_ATTN)})
    packs = [torch.empty(payload, dtype=torch.uint8, device=dev) for _ in range(packed_n)]
    torch.cuda.synchronize()
    reps = max(args.steps, 3)
    pct = lambda ms: 100 * 2 * payload / ms / 1e6 / HBM_PEAK_GBPS
    layouts = ("nhd", "hnd", "paged_attn")
    rows = []
    for ci, cv in enumerate(views):
        for pi, p in enumerate(packs):
            row = {"cache": ci, "packed": pi}
            for lay in layouts:
                c = cv[lay]
                g = event_ms(lambda: kvx.kvx_gather_blocks(c, 0, L, bt_src, n, ct, p), reps)
                sc = event_ms(lambda: kvx.kvx_scatter_blocks(c, 0, L, bt_dst, n, ct, p), reps)
                row[f"{lay}_gather_pct"] = round(pct(statistics.median(g)), 2)
                row[f"{lay}_scatter_pct"] = round(pct(statistics.median(sc)), 2)
            rows.append(row)
    kvx.kvx_check()
    log(f"layouts: {rows}")
    summary = {}
    for lay in layouts:
        for d in ("gather", "scatter"):
            v = [r[f"{lay}_{d}_pct"] for r in rows]
            s = {"mean": round(statistics.mean(v), 2), "min": min(v), "max": max(v)}
            if lay != "nhd":
                diff = [r[f"{lay}_{d}_pct"] - r[f"nhd_{d}_pct"] for r in rows]
                s["minus_nhd"] = {"mean": round(statistics.mean(diff), 2),
                                  "min": round(min(diff), 2), "max": round(max(diff), 2)}
            summary[f"{lay}_{d}_pct_hbm_peak"] = s
    mean_rate = statistics.mean([summary[f"{lay}_{d}_pct_hbm_peak"]["mean"] for lay in layouts
                                 for d in ("gather", "scatter")]) * HBM_PEAK_GBPS / 100
    out = base_record(
        args, "KV gather/scatter GB/s & % HBM peak per cache layout, same allocations", "GB/s",
        round(mean_rate, 1), None,
        {"workload": "llama-3-8b-shaped paged KV, 80k-token prefix (5000 blocks), 256-token "
                     "chunks, the cache read as NHD, HND and paged attention on each of "
                     f"{caches_n} caches x {packed_n} packed buffers",
         "num_blocks": NB, "prefix_tokens": n * BS, "chunk_tokens": ct, "kv_heads": H,
         "caches": caches_n, "packed": packed_n, "parallelism": "single GPU"})
    out.update(summary)
    out.update({"pairs": rows, "reps_per_pair": reps,
                "note": "value: mean of the six rates (three layouts, two directions) over "
                        "the pairs; minus_nhd: each pair's rate less the NHD rate on the "
                        "same pair, in points of peak"})
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this path needs no collective, and the "
              "multi-GPU sharding is described, not built. Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch

    torch.cuda.set_device(torch.device("cuda:0"))
    {"8b-80k": run_80k, "8b-32k-sweep": run_sweep, "70b-batch": run_batch,
     "8b-files": run_files, "8b-preload": run_preload,
     "8b-placements": run_placements, "8b-layouts": run_layouts}[args.workload](args)


if __name__ == "__main__":
    main()
