#!/usr/bin/env python3
"""Benchmark: paged-KV gather / scatter / staged restore on one MI355X.

Workload (default): Llama-3-8B-shaped KV cache (32 layers, K and V each
[20000 blocks, 16 tokens, 8 KV heads, head dim 128] bf16, N(0,1) from a seed),
an 80,000-token prefix = 5,000 blocks at seeded random block ids, 256-token
transfer chunks (all layers per chunk, layer-major).

One step = the whole hot path once over that prefix:
  1. gather the 5,000 blocks into packed chunks (HBM -> HBM),
  2. scatter the packed chunks into 5,000 fresh blocks (HBM -> HBM),
  3. staged restore of an 80k-token packed image from pinned host memory
     through a 4 x 64 MiB pinned staging ring (fill -> H2D on a side stream ->
     scatter kernel, overlapped through HIP events) into another 5,000 blocks.
Inputs are resident (cache in HBM, image in pinned host memory) before the
timed region starts.

Prints ONE JSON line. `value` is the gather/scatter HBM throughput (bytes read
plus bytes written by the two kernels, per second of their event-timed
device time); the restore time is reported next to it.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, vendor figure


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--num-blocks", type=int, default=20000)
    ap.add_argument("--prefix-blocks", type=int, default=5000)
    ap.add_argument("--chunk-tokens", type=int, default=256)
    ap.add_argument("--slots", type=int, default=4)
    ap.add_argument("--slot-mib", type=int, default=64)
    ap.add_argument("--fill-threads", type=int, default=8)
    ap.add_argument("--seed", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-blocks", type=int, default=1250)
    ap.add_argument("--probe-reps", type=int, default=10)
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this path needs no collective, and the "
              "multi-GPU sharding is described, not built. Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import kvsynth
    import paper_2609_11744_amd as kvx

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    L, BS, H, D, E = 32, 16, 8, 128, 2
    NB, n, ct = args.num_blocks, args.prefix_blocks, args.chunk_tokens
    if 3 * n > NB:
        raise SystemExit("pool too small for three disjoint prefixes")
    slab = BS * H * D * E
    payload = n * L * 2 * slab
    log(f"workload: 8B-shaped cache {NB} blocks ({NB * L * 2 * slab / 1e9:.1f} GB), "
        f"prefix {n} blocks = {n * BS} tokens, payload {payload / 1e9:.3f} GB")

    # ---- inputs -----------------------------------------------------------
    cache = kvx.PagedKVCache.allocate(L, NB, BS, H, D, torch.bfloat16, dev)
    for l in range(L):
        kvsynth.fill_device(cache.k[l], args.seed, kvsynth.cache_stream(kvsynth.ROLE_SRC, l, 0))
        kvsynth.fill_device(cache.v[l], args.seed, kvsynth.cache_stream(kvsynth.ROLE_SRC, l, 1))
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

    # ---- same-run probes ----------------------------------------------------
    probe = {}
    h = torch.empty(1 << 30, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(1 << 30, dtype=torch.uint8, device=dev)

    def timed_copy(dst, src, reps):
        out = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            dst.copy_(src, non_blocking=True)
            b.record()
            b.synchronize()
            out.append(a.elapsed_time(b))
        return statistics.median(out)

    probe["h2d_GBps"] = (1 << 30) / timed_copy(d, h, args.probe_reps) / 1e6
    probe["d2h_GBps"] = (1 << 30) / timed_copy(h, d, args.probe_reps) / 1e6
    del h
    dd = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
    ds = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
    ms = timed_copy(dd, ds, 5)
    probe["d2d_copy_GBps_rw"] = 2 * (4 << 30) / ms / 1e6
    del dd, ds, d
    torch.cuda.empty_cache()
    log(f"probes: {probe}")

    # ---- steps --------------------------------------------------------------
    def step(record):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record()
        kvx.kvx_gather_blocks(cache, 0, L, bt_src, n, ct, packed)
        e[1].record()
        kvx.kvx_scatter_blocks(cache, 0, L, bt_dst, n, ct, packed)
        e[2].record()
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

    med = {k: statistics.median(v) for k, v in rec.items()}
    mean_g = statistics.mean(rec["gather_ms"])
    mean_s = statistics.mean(rec["scatter_ms"])
    rw = 2 * payload
    gs_GBps = 2 * rw / ((sum(rec["gather_ms"]) + sum(rec["scatter_ms"])) / args.steps) / 1e6
    gather_GBps = rw / mean_g / 1e6
    scatter_GBps = rw / mean_s / 1e6
    restore_GBps = payload / med["restore_ms"] / 1e6

    # ---- CPU baseline: the oracle on a bounded sample ------------------------
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, L, BS, H, D, E, perm)

    out = {
        "metric": "KV gather/scatter GB/s & % HBM peak; 80k-token prefix restore ms",
        "value": round(gs_GBps, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 KV, seeded random block ids)",
        "config": {"workload": "llama-3-8b-shaped paged KV, 80k-token prefix (5000 blocks), "
                               "256-token chunks, 4 x 64 MiB pinned staging ring",
                   "num_blocks": NB, "prefix_tokens": n * BS, "chunk_tokens": ct,
                   "slots": args.slots, "slot_mib": args.slot_mib,
                   "fill_threads": args.fill_threads, "parallelism": "single GPU"},
        "pct_hbm_peak": round(100 * gs_GBps / HBM_PEAK_GBPS, 2),
        "gather_GBps_rw": round(gather_GBps, 1),
        "scatter_GBps_rw": round(scatter_GBps, 1),
        "gather_ms": round(mean_g, 4),
        "scatter_ms": round(mean_s, 4),
        "restore_ms": round(med["restore_ms"], 3),
        "restore_GBps": round(restore_GBps, 2),
        "restore_frac_of_h2d": round(restore_GBps / probe["h2d_GBps"], 4),
        "restore_breakdown_ms": {"fill_thread_sum": round(med["fill_ms"], 2),
                                 "enqueue_wait_for_fill": round(med["wait_fill_ms"], 2),
                                 "device_span": round(med["restore_dev_ms"], 2)},
        "probes": {k: round(v, 2) for k, v in probe.items()},
        "roofline": {"bound": "hbm", "kernel": "gather (copy_units_kernel<true, 1024, 2>)",
                     "achieved": round(gather_GBps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(gather_GBps / HBM_PEAK_GBPS, 4),
                     "traffic": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    ring.close()
    image.free()


def cpu_baseline(args, L, BS, H, D, E, perm):
    """Time the oracle (plain C slab memcpy, one thread) gathering and
    scattering a bounded sample of the same workload on this host."""
    import numpy as np

    import kvsynth
    import oracle

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
    oracle.gather(shape, k, v, 0, L, ids, args.chunk_tokens, out=out)  # touch pages once
    oracle.scatter(shape, k, v, 0, L, dst_ids, args.chunk_tokens, out)
    times = []
    for _ in range(3):
        t0 = time.perf_counter()
        oracle.gather(shape, k, v, 0, L, ids, args.chunk_tokens, out=out)
        oracle.scatter(shape, k, v, 0, L, dst_ids, args.chunk_tokens, out)
        times.append(time.perf_counter() - t0)
    t = statistics.median(times)
    rw = 2 * 2 * out.nbytes
    return {"value": round(rw / t / 1e9, 2), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"gather + scatter of {m} of the {args.prefix_blocks} prefix blocks "
                      f"({out.nbytes / 1e9:.2f} GB payload each way), median of 3, "
                      f"single-threaded C slab memcpy"}


if __name__ == "__main__":
    main()
