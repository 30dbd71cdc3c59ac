"""Benchmark of the KV repack (fused pack + unpack) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME]

A step is one kvx_repack over the whole batch of the workload (default: the
Llama-3-8B-shaped KV of 16 requests, 32 layers x 8 KV heads x 128 dims, bf16,
into 16-token pages of a 65536-page pool), with the inputs already resident in
HBM.  Prints one JSON line on stdout: throughput in GB/s of algorithmic bytes
(read + written), the HBM roofline of the kernel (HIP-event kernel time on
the launch stream), pack and unpack alone, per-request latency, and the CPU
oracle timed on a bounded sample of the same workload.  Progress goes to
stderr.
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
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, AMD's published peak
METRIC = "KV repack GB/s (read+write) and % of MI355X HBM peak; per-request latency"
KERNEL_SRC = os.path.join(ROOT, "paper_2509_17542_amd", "csrc", "kvx_kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per repack launch from the committed rocprofv3 counter runs,
    or None if absent or taken on another version of the kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3_8b_bf16_bs16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="time the repack only (no pack/unpack/latency legs)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--calib-gib", type=float, default=4.0,
                    help="size of the plain device copy timed as a ceiling (and used to "
                         "calibrate rocprofv3 byte counters); 0 = skip")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the conversion runs on a single MI355X and this build "
              "has no multi-GPU path (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2509_17542_amd as K
    import workload as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    w = W.WORKLOADS[args.workload]
    if w.layers != w.total_layers:
        w = w.replace()   # layer-group workloads time their first group
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    log(f"{w.name}: {len(lens)} requests, {int(lens.sum())} tokens; generating inputs")
    t0 = time.time()
    shards = W.source_shards(w, lens)
    log(f"inputs generated in {time.time() - t0:.1f}s; uploading")
    dshards = [None if s is None else torch.from_numpy(s.view(np.int16)).cuda() for s in shards]
    bt_d = torch.from_numpy(bt).cuda()
    F = {"fp16": K.FP16, "bf16": K.BF16, "e4m3fn": K.E4M3FN}
    order = K.THD if w.src_order == "thd" else K.HTD

    def desc(seq):
        return K.make_desc(w.layers, w.heads, w.head_dim, w.src_tp, w.dst_tp, w.dst_rank,
                           F[w.src_dtype], F[w.dst_dtype], order, w.block_size, w.num_blocks, seq)

    plan = K.kvx_plan(desc(list(lens)))
    info = K.kvx_plan_info_get(plan)
    esz = 1 if w.dst_dtype == "e4m3fn" else 2
    n_rows = w.layers * 2 * w.num_blocks * w.block_size * w.hd
    cache = torch.empty(n_rows * w.head_dim * esz, dtype=torch.uint8, device="cuda")
    scales = torch.empty(n_rows, dtype=torch.float32, device="cuda") if esz == 1 else None
    log(f"pool {cache.numel() / 2**30:.1f} GiB allocated")
    stream = torch.cuda.current_stream()
    rep_bytes = info.read_bytes_repack + info.write_bytes_repack

    def timed(fn, steps, warmup):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        torch.cuda.synchronize()
        t = time.perf_counter()
        for a, b in ev:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t) / steps
        kern = [a.elapsed_time(b) for a, b in ev]
        return wall * 1e3, statistics.mean(kern), min(kern), statistics.median(kern)

    def repack():
        K.kvx_repack(plan, dshards, cache, scales, bt_d, stride, stream)

    log(f"repack: {args.warmup} warm-up + {args.steps} timed steps")
    ms_step, k_mean, k_min, k_med = timed(repack, args.steps, args.warmup)
    value = rep_bytes / (ms_step * 1e-3) / 1e9
    achieved = rep_bytes / (k_mean * 1e-3) / 1e9
    log(f"repack {ms_step:.3f} ms/step, kernel mean {k_mean:.3f} ms -> {achieved:.0f} GB/s")

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": w.layers, "kv_heads": w.heads,
                   "head_dim": w.head_dim, "requests": len(lens), "tokens": int(lens.sum()),
                   "src_tp": w.src_tp, "dst_tp": w.dst_tp, "dst_rank": w.dst_rank,
                   "src_dtype": w.src_dtype, "dst_dtype": w.dst_dtype,
                   "src_order": w.src_order, "block_size": w.block_size,
                   "pool_blocks": w.num_blocks, "bytes_per_step": rep_bytes},
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "repack_kernel_ms": {"mean": round(k_mean, 4), "min": round(k_min, 4),
                             "median": round(k_med, 4)},
    }
    if args.calib_gib > 0:
        # plain device copies of known size (read N + write N bytes): the HIP
        # runtime's copy kernel (hipMemcpyAsync device to device) and a torch
        # elementwise kernel; the references for the byte counters
        n = int(args.calib_gib * 2**30) // 4
        a = torch.empty(n, dtype=torch.int32, device="cuda")
        b = torch.empty_like(a)
        out["copy_ceiling"] = {}
        for kind, fn in (("hipMemcpy_d2d", lambda: b.copy_(a)),
                         ("torch_elementwise", lambda: torch.bitwise_not(a, out=b))):
            ms, km, _, _ = timed(fn, 10, 2)
            out["copy_ceiling"][kind] = {"bytes": 8 * n, "kernel_ms": round(km, 4),
                                         "GB/s": round(8 * n / (km * 1e-3) / 1e9, 1)}
            log(f"plain copy ({kind}): {8 * n / (km * 1e-3) / 1e9:.0f} GB/s")
        del a, b

    traffic = measured_traffic(w.name)
    out["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                       "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                       "traffic": traffic, "kernel": "kvx convert_rows<repack>",
                       "algorithmic_bytes_per_launch": rep_bytes}

    if not args.no_extras:
        wire = torch.empty(int(info.wire_bytes), dtype=torch.uint8, device="cuda")

        def pack():
            K.kvx_pack(plan, dshards, wire, stream)

        def unpack():
            K.kvx_unpack(plan, wire, cache, scales, bt_d, stride, stream)

        for name, fn, nbytes in (("pack", pack, info.read_bytes_pack + info.write_bytes_pack),
                                 ("unpack", unpack,
                                  info.read_bytes_unpack + info.write_bytes_unpack)):
            ms, km, _, _ = timed(fn, max(5, args.steps // 2), 2)
            out[name] = {"ms_per_step": round(ms, 4), "kernel_ms": round(km, 4),
                         "GB/s": round(nbytes / (km * 1e-3) / 1e9, 1)}
            log(f"{name}: kernel {km:.3f} ms")
        del wire

        # per-request latency: a single-request plan per request, host call to completion
        lat = []
        src_off = 0
        for r, T in enumerate(lens.tolist()):
            p1 = K.kvx_plan(desc([T]))
            sh = [None if s is None else s[src_off:] for s in dshards]
            src_off += w.layers * 2 * T * w.hs * w.head_dim
            row = bt_d[r:r + 1]
            ev = torch.cuda.Event()
            K.kvx_repack(p1, sh, cache, scales, row, stride, stream)   # warm
            torch.cuda.synchronize()
            reps = []
            for _ in range(5):
                t = time.perf_counter()
                K.kvx_repack(p1, sh, cache, scales, row, stride, stream)
                ev.record(stream)
                ev.synchronize()
                reps.append((time.perf_counter() - t) * 1e3)
            lat.append(statistics.median(reps))
        lat_sorted = sorted(lat)
        out["latency_ms_per_request"] = {
            "p50": round(statistics.median(lat), 4),
            "p90": round(lat_sorted[min(len(lat) - 1, int(0.9 * len(lat)))], 4),
            "max": round(max(lat), 4), "batch_over_requests": round(ms_step / len(lens), 4),
            "note": "single-request plan, host call to event completion, median of 5"}
        log(f"latency p50 {out['latency_ms_per_request']['p50']} ms")

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, lens, shards, args.cpu_seconds, value)
    print(json.dumps(out), flush=True)


def cpu_baseline(w, lens, shards, budget_s, gpu_value):
    """The oracle as it stands (single thread), on whole requests of the same
    workload until about budget_s seconds of CPU work; pages renumbered into a
    compact host pool (same rows, same bytes)."""
    import numpy as np

    import oracle as O

    f = {"fp16": O.FP16, "bf16": O.BF16, "e4m3fn": O.E4M3FN}
    order = O.TOKEN_MAJOR if w.src_order == "thd" else O.HEAD_MAJOR
    esz = 1 if w.dst_dtype == "e4m3fn" else 2
    done_bytes = 0
    spent = 0.0
    off = 0
    n = 0
    tokens = 0
    for r, T in enumerate(lens.tolist()):
        if spent >= budget_s:
            break
        nb = (T + w.block_size - 1) // w.block_size
        p = O.OracleProblem(w.layers, w.heads, w.head_dim, w.src_tp, w.dst_tp, w.dst_rank,
                            f[w.src_dtype], f[w.dst_dtype], order, w.block_size, max(nb, 1), [T])
        cnt = w.layers * 2 * T * w.hs * w.head_dim
        part = [None if s is None else np.ascontiguousarray(s[off:off + cnt]) for s in shards]
        off += cnt
        cache = np.empty(O.cache_bytes(p), dtype=np.uint8)
        sc = np.empty(O.scale_count(p), dtype=np.float32) if esz == 1 else None
        bt = np.arange(max(nb, 1), dtype=np.int32)[None, :]
        t = time.perf_counter()
        O.repack(p, part, cache, sc, bt, max(nb, 1))
        spent += time.perf_counter() - t
        rows = w.layers * 2 * T * w.hd
        done_bytes += rows * w.head_dim * (2 + esz) + (rows * 4 if esz == 1 else 0)
        n += 1
        tokens += T
    gbs = done_bytes / spent / 1e9 if spent > 0 else None
    log(f"cpu oracle: {n} requests, {done_bytes / 1e9:.2f} GB in {spent:.1f}s -> {gbs:.3f} GB/s")
    return {"value": round(gbs, 4) if gbs else None, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of {len(lens)} requests ({tokens} tokens, "
                      f"{done_bytes / 1e9:.2f} GB read+written) of {w.name}, single-threaded "
                      "plain-C oracle, pages renumbered into a compact host pool",
            "seconds": round(spent, 2),
            "gpu_over_cpu": round(gpu_value / gbs, 1) if gbs else None}


if __name__ == "__main__":
    main()
