"""Benchmark of the KV repack (fused pack + unpack) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME]

A step is one kvx_repack over the whole batch of the workload (default: the
Llama-3-8B-shaped KV of 16 requests, 32 layers x 8 KV heads x 128 dims, bf16,
into 16-token pages of a 65536-page pool), with the inputs already resident in
HBM.  Prints one JSON line on stdout: throughput in GB/s of algorithmic bytes
(read + written), the HBM roofline of the kernel (HIP-event kernel time on
the launch stream), pack, unpack and pack-then-unpack, per-request latency,
plain copies of known size beside it, the layer-streamed transfer through
pinned host memory, the P:D planner, every named workload in turn
(`configs`), and the CPU oracle timed on a bounded sample of the headline
workload.  Progress goes to stderr.
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


CONFIG_WORKLOADS = ("tiny_tp1to2_fp16_bf16", "llama3_8b_bf16_bs16", "llama3_70b_tp4to2_bf16_bs32",
                    "qwen7b_htd_fp16_bf16_bs64", "fp8_decode_61l_bf16_e4m3_bs16")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama3_8b_bf16_bs16")
    ap.add_argument("--configs", default=",".join(CONFIG_WORKLOADS),
                    help="comma-separated workloads measured one after another after the headline "
                         "one (repack, pack, unpack, request latency), each freed before the next; "
                         "'none' = skip")
    ap.add_argument("--pages", choices=("random", "consecutive"), default="random",
                    help="destination pages of the decode pool: the workload's seeded random "
                         "block table, or consecutive pages (a diagnostic of page scatter)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="time the repack only (no pack/unpack/latency legs)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--stream-chunk", type=int, default=4,
                    help="layers per chunk of the layer-streamed transfer leg (0 = skip it)")
    ap.add_argument("--stream-slots", type=int, default=3)
    ap.add_argument("--stream-extra-streams", type=int, default=0,
                    help="HIP streams the process creates (and keeps) before the layer-streamed "
                         "transfer's pipe: a diagnostic of the pipe's independence from how "
                         "earlier streams map onto hardware queues")
    ap.add_argument("--calib-gib", type=float, default=2.0,
                    help="bytes read (= bytes written) by the plain copies timed as ceilings "
                         "and as the reference of the rocprofv3 byte counters; 0 = skip")
    ap.add_argument("--derive-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter files (FETCH_SIZE, WRITE_SIZE) of "
                         "this benchmark into profiles/traffic.json and exit")
    args = ap.parse_args()
    if args.derive_traffic:
        derive_traffic(*args.derive_traffic, workload=args.workload, calib_gib=args.calib_gib)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the conversion runs on a single MI355X and the library "
              "has no multi-GPU path (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2509_17542_amd as K
    import workload as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

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

    w = W.WORKLOADS[args.workload]
    wb = Workbench(K, W, torch, w, stream, all_shards=True,
                   consecutive=args.pages == "consecutive")
    rep_bytes = wb.bytes("repack")

    log(f"repack: {args.warmup} warm-up + {args.steps} timed steps")
    ms_step, k_mean, k_min, k_med = timed(wb.repack, args.steps, args.warmup)
    value = rep_bytes / (ms_step * 1e-3) / 1e9
    achieved = rep_bytes / (k_mean * 1e-3) / 1e9
    log(f"repack {ms_step:.3f} ms/step, kernel mean {k_mean:.3f} ms -> {achieved:.0f} GB/s")

    stages, paged, lens = wb.stages, wb.paged, wb.lens
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.src_dtype if w.src_dtype == w.cdt == w.dst_dtype else
                 "->".join(dict.fromkeys([w.src_dtype, w.dst_dtype, w.cdt])),
        "data": "synthetic",
        "config": {"workload": w.name, "layers": w.layers, "kv_heads": w.heads,
                   "head_dim": w.head_dim, "requests": len(lens), "tokens": int(lens.sum()),
                   "src_tp": w.src_tp, "dst_tp": w.dst_tp, "dst_rank": w.dst_rank,
                   "src_dtype": w.src_dtype, "dst_dtype": w.dst_dtype,
                   **({"cache_dtype": w.cache_dtype} if w.cache_dtype else {}),
                   "src_order": w.src_order, "block_size": w.block_size,
                   "pool_blocks": w.num_blocks, "bytes_per_step": rep_bytes,
                   **({"dst_pages": "consecutive (diagnostic)"} if args.pages != "random"
                      else {})},
        **({"prefill_stages": [list(st) for st in stages], "launches_per_step": len(stages),
            "streams_per_step": len(stages)}
           if len(stages) > 1 else {}),
        **({"src_pages": {"block_size": w.src_block_size, "pool_blocks": w.src_num_blocks}}
           if paged else {}),
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "hbm_peak_from_device": device_hbm_peak(),
        "repack_kernel_ms": {"mean": round(k_mean, 4), "min": round(k_min, 4),
                             "median": round(k_med, 4)},
    }
    if args.calib_gib > 0:
        out["copy_ceiling"] = copy_legs(K, torch, args.calib_gib, timed, stream)

    traffic = measured_traffic(w.name)
    out["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                       "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                       "traffic": traffic, "kernel": "kvx_repack_kernel",
                       "algorithmic_bytes_per_launch": rep_bytes}

    headline = {"repack": {"kernel_ms": round(k_mean, 4), "GB/s": round(achieved, 1),
                           "frac": round(achieved / HBM_PEAK_GBS, 4)}}
    if not args.no_extras:
        for name in ("pack", "unpack", "pack_unpack"):
            ms, km, _, _ = timed(getattr(wb, name), max(5, args.steps // 2), 2)
            gbs = wb.bytes(name) / (km * 1e-3) / 1e9
            out[name] = {"ms_per_step": round(ms, 4), "kernel_ms": round(km, 4),
                         "GB/s": round(gbs, 1)}
            headline[name] = {"kernel_ms": round(km, 4), "GB/s": round(gbs, 1),
                              "frac": round(gbs / HBM_PEAK_GBS, 4)}
            log(f"{name}: kernel {km:.3f} ms")
        wb.free_wires()
        out["latency_ms_per_request"] = wb.latency()
        out["latency_ms_per_request"]["batch_over_requests"] = round(ms_step / len(lens), 4)
        headline["latency_ms_per_request"] = out["latency_ms_per_request"]
        log(f"latency p50 {out['latency_ms_per_request']['p50']} ms")

    if not args.no_extras and args.stream_chunk > 0 and len(stages) == 1:
        out["layer_stream"] = stream_leg(K, torch, wb.plans[0], wb.infos[0], wb.dshards[0],
                                         wb.sbt_d, wb.sstride, wb.cache, wb.scales, wb.bt_d,
                                         wb.stride, min(args.stream_chunk, w.layers),
                                         args.stream_slots, args.stream_extra_streams)

    if not args.no_extras:
        out["pd_planner"] = planner_leg(K, w)

    host_shards = wb.host_shards[0]
    sbt = wb.sbt
    wb.free()
    del wb
    torch.cuda.empty_cache()

    names = [] if args.configs == "none" else [n for n in args.configs.split(",") if n]
    if names:
        out["configs"] = configs_leg(K, W, torch, stream, timed, names, w.name, headline,
                                     args.steps, args.warmup)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, lens, host_shards, args.cpu_seconds, value, sbt,
                                           stages[0])
    print(json.dumps(out), flush=True)


class Workbench:
    """One workload resident on the device, ready to launch.  The decode
    side's paged pool is allocated first, as a serving engine reserves it at
    start-up; the source buffers of the requests come after it.  Prefill
    pipeline stages hold a layer range each in their own buffers and get a
    plan each; all of them fill the one decode cache.  Layer-group workloads
    hold their first group."""

    def __init__(self, K, W, torch, w, stream, all_shards=False, consecutive=False):
        import numpy as np
        self.K, self.torch, self.w, self.stream = K, torch, w, stream
        lens = self.lens = W.seq_lens(w)
        self.bt, self.stride = W.block_table(w, lens, consecutive)
        esz = 1 if w.cdt in ("e4m3fn", "e5m2") else 2   # the cache's element size
        n_rows = w.layers * 2 * w.num_blocks * w.block_size * w.hd
        self.cache = torch.empty(n_rows * w.head_dim * esz, dtype=torch.uint8, device="cuda")
        self.scales = (torch.empty(n_rows, dtype=torch.float32, device="cuda") if esz == 1
                       else None)
        log(f"{w.name}: pool {self.cache.numel() / 2**30:.1f} GiB allocated; {len(lens)} "
            f"requests, {int(lens.sum())} tokens; generating inputs")
        F = {"fp16": K.FP16, "bf16": K.BF16, "e4m3fn": K.E4M3FN, "e5m2": K.E5M2}
        order = {"thd": K.THD, "htd": K.HTD, "paged": K.PAGED}[w.src_order]
        self.paged = w.src_order == "paged"
        self.stages = W.src_stages(w)

        def desc(seq, stage):
            l0, n = stage
            return K.make_desc(n, w.heads, w.head_dim, w.src_tp, w.dst_tp, w.dst_rank,
                               F[w.src_dtype], F[w.dst_dtype], order, w.block_size, w.num_blocks,
                               seq, w.src_block_size, w.src_num_blocks, 0, n, l0, w.layers,
                               F[w.cache_dtype] if w.cache_dtype else 0)

        self.desc = desc
        self.plans = [K.kvx_plan(desc(list(lens), st)) for st in self.stages]
        self.infos = [K.kvx_plan_info_get(p) for p in self.plans]
        read = None if all_shards else \
            [j for j in range(w.src_tp) if K.kvx_plan_shard_bytes(self.plans[0], j) > 0]
        t0 = time.time()
        self.host_shards = [W.source_shards(w, lens, l0, n, read) for l0, n in self.stages]
        log(f"inputs generated in {time.time() - t0:.1f}s; uploading")
        self.dshards = [[None if s is None else torch.from_numpy(s.view(np.int16)).cuda()
                         for s in sh] for sh in self.host_shards]
        self.bt_d = torch.from_numpy(self.bt).cuda()
        self.sbt = self.sbt_d = None
        self.sstride = 0
        if self.paged:   # the prefill side's own paged cache and its block table
            self.sbt, self.sstride = W.src_block_table(w, lens)
            self.sbt_d = torch.from_numpy(self.sbt).cuda()
        self.wires = None
        # Prefill stages are independent transfers: each stage's launch goes
        # on a stream of its own (default priority), forked from the timed
        # stream and joined back into it, so that the stages write their
        # halves of the pool at the same time.
        self.side = [torch.cuda.Stream() for _ in self.stages[1:]]
        self.fork = torch.cuda.Event()

    def bytes(self, op):
        if op == "pack_unpack":
            return self.bytes("pack") + self.bytes("unpack")
        return sum(getattr(i, f"read_bytes_{op}") + getattr(i, f"write_bytes_{op}")
                   for i in self.infos)

    def _per_stage(self, launch):
        if self.side:
            self.fork.record(self.stream)
            for s in self.side:
                s.wait_event(self.fork)
        for k, st in enumerate([self.stream] + self.side):
            launch(k, st)
        for s in self.side:
            self.stream.wait_stream(s)

    def repack(self):
        K = self.K

        def launch(k, st):
            if self.paged:
                K.kvx_repack_paged(self.plans[k], self.dshards[k], self.sbt_d, self.sstride,
                                   self.cache, self.scales, self.bt_d, self.stride, st)
            else:
                K.kvx_repack(self.plans[k], self.dshards[k], self.cache, self.scales, self.bt_d,
                             self.stride, st)
        self._per_stage(launch)

    def _wires(self):
        if self.wires is None:
            self.wires = [self.torch.empty(int(i.wire_bytes), dtype=self.torch.uint8,
                                           device="cuda") for i in self.infos]
        return self.wires

    def pack(self):
        K, wires = self.K, self._wires()

        def launch(k, st):
            if self.paged:
                K.kvx_pack_paged(self.plans[k], self.dshards[k], self.sbt_d, self.sstride,
                                 wires[k], st)
            else:
                K.kvx_pack(self.plans[k], self.dshards[k], wires[k], st)
        self._per_stage(launch)

    def unpack(self):
        wires = self._wires()
        self._per_stage(lambda k, st: self.K.kvx_unpack(self.plans[k], wires[k], self.cache,
                                                        self.scales, self.bt_d, self.stride, st))

    def pack_unpack(self):
        """The two-step path: pack into the transfer tensor, then unpack it."""
        self.pack()
        self.unpack()

    def free_wires(self):
        self.wires = None

    def all_groups(self, timed, steps, warmup):
        """A layer-group workload's whole cache: one repack launch per group
        (groups of w.layers layers, the last one shorter), all into the one
        resident pool, events around the whole sequence.  Every group reads
        the first group's resident source buffer: a group's own values would
        need inputs generated for it, and the values do not change the work
        (no row of them holds a NaN, an infinity or only zeros, so every row
        takes the same path)."""
        K, w = self.K, self.w
        assert not self.paged and len(self.stages) == 1
        full, last = divmod(w.total_layers, w.layers)
        plans = [self.plans[0]] * full
        if last:
            plans.append(K.kvx_plan(self.desc(list(self.lens), (0, last))))
        nbytes = sum(i.read_bytes_repack + i.write_bytes_repack
                     for i in (K.kvx_plan_info_get(p) for p in plans))

        def step():
            for p in plans:
                K.kvx_repack(p, self.dshards[0], self.cache, self.scales, self.bt_d,
                             self.stride, self.stream)
        nw = settle(step, self.torch, warmup, CONFIG_SETTLE_MS)
        _, km, kmin, kmed = timed(step, steps, 0)
        gbs = nbytes / (km * 1e-3) / 1e9
        log(f"{w.name}: all {len(plans)} groups {km:.2f} ms -> {gbs:.0f} GB/s")
        return {"layers": w.total_layers, "launches": len(plans),
                "group_layers": [w.layers] * full + ([last] if last else []),
                "bytes": nbytes, "ms": round(km, 3), "ms_min": round(kmin, 3),
                "ms_median": round(kmed, 3), "GB/s": round(gbs, 1),
                "frac": round(gbs / HBM_PEAK_GBS, 4), "warmup_steps": nw,
                "sources": "every group reads the first group's resident source buffer"}

    def latency(self):
        """Per-request latency: single-request plans (one per prefill stage)
        per request, host call to completion; the stages of one request go on
        the timed stream one after the other (for launches this small a fork
        and join across streams costs more than it overlaps)."""
        K, w, torch, stream = self.K, self.w, self.torch, self.stream
        lat = []
        src_off = 0
        for r, T in enumerate(self.lens.tolist()):
            p1s = [K.kvx_plan(self.desc([T], st)) for st in self.stages]
            row = self.bt_d[r:r + 1]
            if self.paged:   # the same pools, this request's row of the source block table
                srow = self.sbt_d[r:r + 1]

                def one():
                    for p1, dsh in zip(p1s, self.dshards):
                        K.kvx_repack_paged(p1, dsh, srow, self.sstride, self.cache, self.scales,
                                           row, self.stride, stream)
            else:
                shs = [[None if s is None else s[src_off * n // w.layers:] for s in dsh]
                       for (_, n), dsh in zip(self.stages, self.dshards)]

                def one():
                    for p1, sh in zip(p1s, shs):
                        K.kvx_repack(p1, sh, self.cache, self.scales, row, self.stride, stream)
            src_off += w.layers * 2 * T * w.hs * w.head_dim
            ev = torch.cuda.Event()
            one()   # warm
            torch.cuda.synchronize()
            reps = []
            for _ in range(5):
                t = time.perf_counter()
                one()
                ev.record(stream)
                ev.synchronize()
                reps.append((time.perf_counter() - t) * 1e3)
            lat.append(statistics.median(reps))
        s = sorted(lat)
        return {"p50": round(statistics.median(lat), 4),
                "p90": round(s[min(len(s) - 1, int(0.9 * len(s)))], 4), "max": round(max(lat), 4),
                "requests": len(lat),
                "note": "single-request plan, host call to event completion, median of 5"}

    def free(self):
        self.cache = self.scales = self.dshards = self.bt_d = self.sbt_d = self.wires = None
        self.plans = self.side = None


CONFIG_SETTLE_MS = 50.0  # least wall time of warm-up launches per operation in the configs leg


def settle(fn, torch, launches, ms):
    """Warm-up: `launches` launches of fn, then more in groups of the same
    size until `ms` of wall time has passed.  Back-to-back launches after an
    idle spell run at first above and then below the clock the power limit
    settles at (kernel traces show the times falling for about 20 ms), so a
    short launch needs more than a fixed count to reach its steady rate.
    Returns the number of launches."""
    group = max(launches, 1)
    n = 0
    t0 = time.perf_counter()
    while n < launches or (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(group):
            fn()
        n += group
        torch.cuda.synchronize()
    return n


def configs_leg(K, W, torch, stream, timed, names, headline_name, headline, steps, warmup):
    """Each named workload measured after the headline one: repack, pack and
    unpack kernel time (HIP events, mean of the timed launches), GB/s over the
    algorithmic bytes, the fraction of the 8 TB/s HBM peak and per-request
    latency.  Each operation's timed launches follow at least `warmup`
    warm-up launches and CONFIG_SETTLE_MS of them (settle); the count is
    reported.  Each workload's buffers are freed before the next is
    allocated.  The headline workload's own figures are copied, not
    re-measured.  The 8-bit decode workload runs as 4-layer groups (its
    2^20-page pool over 61 layers does not fit in HBM); it reports its first
    group, and the repack of the whole 61-layer cache as its 16 group
    launches in a row (repack_all_groups)."""
    res = {}
    for name in names:
        w = W.WORKLOADS[name]
        entry = {"layers": w.layers, "requests": w.num_requests, "src_tp": w.src_tp,
                 "dst_tp": w.dst_tp, "dtype": f"{w.src_dtype}->{w.cdt}", "order": w.src_order,
                 "block_size": w.block_size, "pool_blocks": w.num_blocks}
        if w.layers != w.total_layers:
            entry["layer_group"] = (f"first {w.layers}-layer group of {w.total_layers} layers "
                                    f"({w.layer_groups} groups)")
        if name == headline_name:
            res[name] = {**entry, **headline, "measured": "headline run"}
            continue
        wb = Workbench(K, W, torch, w, stream)
        entry["tokens"] = int(wb.lens.sum())
        for op in ("repack", "pack", "unpack", "pack_unpack"):
            n = steps if op == "repack" else max(5, steps // 2)
            nw = settle(getattr(wb, op), torch, warmup, CONFIG_SETTLE_MS)
            _, km, kmin, kmed = timed(getattr(wb, op), n, 0)
            nbytes = wb.bytes(op)
            gbs = nbytes / (km * 1e-3) / 1e9
            entry[op] = {"bytes_per_launch": nbytes, "kernel_ms": round(km, 4),
                         "kernel_ms_min": round(kmin, 4), "kernel_ms_median": round(kmed, 4),
                         "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
                         "warmup_launches": nw}
            log(f"config {name}: {op} {km:.3f} ms -> {gbs:.0f} GB/s")
        wb.free_wires()
        if w.layers != w.total_layers:
            entry["repack_all_groups"] = wb.all_groups(timed, steps, warmup)
        entry["latency_ms_per_request"] = wb.latency()
        log(f"config {name}: latency p50 {entry['latency_ms_per_request']['p50']} ms")
        wb.free()
        del wb
        torch.cuda.empty_cache()
        res[name] = entry
    return res


def planner_leg(K, w):
    """The deployment planner of Eq. 1-6 (host code) for the workload's KV
    shape as a whole model on MI355X prefill and decode instances: the
    strategies and P:D ratio it picks for a 4096-token prompt / 512-token
    output service at 20 requests/s with TTFT <= 2 s and TPOT <= 50 ms, and
    the time one search takes.  MI355X: 2.5 PFLOP/s dense bf16, 8 TB/s, 288
    GB, 7 xGMI links of 153 GB/s; discounts 0.5 (compute), 0.8 (HBM, about
    what the repack reaches), 0.7 (links)."""
    # the model around the workload's KV shape: query heads, hidden size and
    # FFN of the Llama-3 models with this many layers and KV heads
    big = w.layers >= 80
    hq, ffn = (64, 28672) if big else (32, 14336)
    m = K.kvx_pd_model(w.layers, hq * w.head_dim, hq, w.heads, w.head_dim, ffn, 128256, 1, 1, 0,
                       2.0, 2.0, 2.0)
    g = K.kvx_pd_gpu(2.5e15, 8e12, 288e9, 7 * 153e9, 0.5, 0.8, 0.7, 8, 0)
    p = K.kvx_pd_problem(m, g, g, 4096, 512, 20.0, 2.0, 0.05, 256, 0)
    reps = 20
    t = time.perf_counter()
    for _ in range(reps):
        sol = K.kvx_pd_search(p)
    ms = (time.perf_counter() - t) / reps * 1e3

    def choice(c):
        return {"dp": c.dp, "tp": c.tp, "pp": c.pp, "batch": c.batch, "gpus": c.gpus,
                "latency_s": round(c.latency, 5), "vram_GB": round(c.vram / 1e9, 2),
                "throughput": round(c.throughput, 2)}

    res = {"model": f"{w.layers} layers, {hq} query / {w.heads} KV heads, hidden {hq * w.head_dim}",
           "prefill": choice(sol.prefill), "decode": choice(sol.decode),
           "instances": f"{sol.prefill_instances}:{sol.decode_instances}",
           "candidates": int(sol.candidates_prefill + sol.candidates_decode),
           "search_ms": round(ms, 3)}
    log(f"pd planner: P {res['prefill']['tp']}x{res['prefill']['pp']} b{res['prefill']['batch']}, "
        f"D {res['decode']['tp']}x{res['decode']['pp']} b{res['decode']['batch']}, "
        f"X:Y {res['instances']}, {ms:.2f} ms per search")
    return res


def stream_leg(K, torch, plan, info, dshards, sbt_d, sstride, cache, scales, bt_d, stride,
               chunk, slots, extra_streams=0):
    """The layer-streamed transfer through pinned host memory (kvx_pipe_run),
    against the same bytes moved serially (pack everything, copy it to pinned
    host memory, copy it back, unpack everything) and against plain copies of
    the transfer tensor in each direction.  Rates are transfer-tensor bytes
    per direction per second: this leg is bound by the host link, not HBM.
    The leg runs on a stream of its own, as a serving engine's transfers
    would (the legacy null stream synchronises with the pipe's CU-masked
    streams: work on it between runs costs the pipe about 2.5% per run, and
    the host sometimes waits in the enqueue).  `extra_streams` HIP streams
    are created before the pipe and destroyed after the leg; each pipe run is
    also timed on its own (HIP events)."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so") if extra_streams > 0 else None
    extra = []
    for _ in range(extra_streams):
        h = ctypes.c_void_p()
        if hip.hipStreamCreate(ctypes.byref(h)) != 0:
            raise RuntimeError("hipStreamCreate failed")
        extra.append(h)
    pipe = K.kvx_pipe_create(plan, chunk, slots)
    pinfo = K.kvx_pipe_info_get(pipe)
    nbytes = int(pinfo.bus_bytes)
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()   # the leg's own stream

    def timed_here(fn, steps, warmup):
        with torch.cuda.stream(stream):
            for _ in range(warmup):
                fn()
            torch.cuda.synchronize()
            t = time.perf_counter()
            for _ in range(steps):
                fn()
            torch.cuda.synchronize()
        return (time.perf_counter() - t) / steps * 1e3

    def piped():
        K.kvx_pipe_run(pipe, dshards, sbt_d, sstride, cache, scales, bt_d, stride, stream)

    wire = torch.empty(int(info.wire_bytes), dtype=torch.uint8, device="cuda")
    back = torch.empty_like(wire)
    host = torch.empty(int(info.wire_bytes), dtype=torch.uint8, pin_memory=True)

    def pack():
        if sbt_d is not None:
            K.kvx_pack_paged(plan, dshards, sbt_d, sstride, wire, stream)
        else:
            K.kvx_pack(plan, dshards, wire, stream)

    def serial():
        pack()
        host.copy_(wire, non_blocking=True)
        back.copy_(host, non_blocking=True)
        K.kvx_unpack(plan, back, cache, scales, bt_d, stride, stream)

    res = {"chunk_layers": chunk, "slots": slots, "chunks": int(pinfo.num_chunks),
           "bytes_each_way": nbytes, "pinned_host_bytes": int(pinfo.host_bytes),
           "stream": "created"}
    for name, fn, steps in (("pipe", piped, 5), ("serial", serial, 3),
                            ("d2h_copy", lambda: host.copy_(wire, non_blocking=True), 3),
                            ("h2d_copy", lambda: back.copy_(host, non_blocking=True), 3)):
        ms = timed_here(fn, steps, 1)
        res[name + "_ms"] = round(ms, 3)
        log(f"layer stream leg: {name} {ms:.2f} ms ({nbytes / (ms * 1e-3) / 1e9:.1f} GB/s each way)")
    each = []
    for _ in range(5):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a.record(stream)
            piped()
            b.record(stream)
        torch.cuda.synchronize()
        each.append(round(a.elapsed_time(b), 2))
    res["pipe_ms_each"] = each
    res["extra_streams_before_pipe"] = extra_streams
    res["pipe_GB/s_each_way"] = round(nbytes / (res["pipe_ms"] * 1e-3) / 1e9, 2)
    res["serial_over_pipe"] = round(res["serial_ms"] / res["pipe_ms"], 3)
    res["note"] = ("layer chunks packed straight into pinned host memory, copied back to the "
                   "device, unpacked; host-link bound, not an HBM figure")
    del pipe, wire, back, host
    for h in extra:
        hip.hipStreamDestroy(h)
    return res


def device_hbm_peak():
    """The HBM peak the HIP runtime's device attributes imply: 2 transfers per
    memory clock x bus width.  Context only; the roofline uses the published
    8 TB/s."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    bus, clk = ctypes.c_int(0), ctypes.c_int(0)
    # hipDeviceAttributeMemoryBusWidth (bits) = 59, hipDeviceAttributeMemoryClockRate (kHz) = 60
    if hip.hipDeviceGetAttribute(ctypes.byref(bus), 59, 0) or \
            hip.hipDeviceGetAttribute(ctypes.byref(clk), 60, 0):
        return None
    return {"bus_width_bits": bus.value, "memory_clock_khz": clk.value,
            "GB/s": round(2 * clk.value * 1e3 * bus.value / 8 / 1e9, 1),
            "formula": "2 x memory clock x bus width / 8"}


CALIB_TOKENS_PER_GIB = 1 << 18   # 1 layer, 8 heads, dim 128, bf16: 2 x 8 x 256 B per token


def copy_legs(K, torch, gib, timed, stream):
    """Plain copies of known size: the identity layout through kvx (one request,
    TP1 -> TP1, bf16, pages 0, 1, 2, ... in order: a memcpy of `gib` GiB done
    by the repack kernel, the reference for the counters), the HIP runtime's
    device copy and a torch elementwise kernel; and, for context, a pure write
    (torch fill) of the same bytes."""
    import numpy as np
    T = int(gib * CALIB_TOKENS_PER_GIB)
    nbytes = T * 2 * 8 * 128 * 2                     # read = written
    src = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    bt = torch.arange(T // 16, dtype=torch.int32, device="cuda")
    plan = K.kvx_plan(K.make_desc(1, 8, 128, 1, 1, 0, K.BF16, K.BF16, K.THD, 16, T // 16, [T]))
    legs = {}
    for kind, fn, rd, wr in (
            ("kvx_identity_memcpy", lambda: K.kvx_repack(plan, [src], dst, None, bt, T // 16,
                                                         stream), nbytes, nbytes),
            ("hipMemcpy_d2d", lambda: dst.view(torch.int16).copy_(src), nbytes, nbytes),
            ("torch_elementwise", lambda: torch.bitwise_not(src, out=dst.view(torch.int16)),
             nbytes, nbytes),
            # one direction only, for context: the HBM rate of pure writes
            ("torch_fill_write_only", lambda: dst.fill_(7), 0, nbytes)):
        ms, km, _, _ = timed(fn, 10, 2)
        gbs = (rd + wr) / (km * 1e-3) / 1e9
        legs[kind] = {"bytes_read": rd, "bytes_written": wr, "kernel_ms": round(km, 4),
                      "GB/s": round(gbs, 1)}
        log(f"plain {kind}: {gbs:.0f} GB/s")
    legs["kvx_identity_memcpy"]["grid_units"] = (T // 16) * 2
    del src, dst, bt, np
    return legs


def derive_traffic(fetch_csv, write_csv, workload, calib_gib):
    """HBM bytes per repack launch from rocprofv3 FETCH_SIZE / WRITE_SIZE
    (KiB per dispatch), each scaled by the ratio of known bytes to counted
    bytes of a plain copy kernel in the same run: torch's elementwise
    bitwise_not over calib_gib GiB (read once, written once, nothing else).
    The repack batch is the kvx_repack_kernel dispatch whose written bytes are
    not the identity-layout copy's; dispatches are told apart by grid size."""
    import csv
    calib_bytes = int(calib_gib * CALIB_TOKENS_PER_GIB) * 2 * 8 * 128 * 2

    def per_grid(path, counter, name):
        vals = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter and name in r["Kernel_Name"]:
                vals.setdefault(int(r["Grid_Size"]), []).append(float(r["Counter_Value"]) * 1024)
        return {g: statistics.median(v) for g, v in vals.items()}

    cf = per_grid(fetch_csv, "FETCH_SIZE", "bitwise_not")
    cw = per_grid(write_csv, "WRITE_SIZE", "bitwise_not")
    assert len(cf) == 1 and len(cw) == 1, (cf, cw)
    kf, kw = calib_bytes / next(iter(cf.values())), calib_bytes / next(iter(cw.values()))
    f = per_grid(fetch_csv, "FETCH_SIZE", "kvx_repack_kernel")
    wr = per_grid(write_csv, "WRITE_SIZE", "kvx_repack_kernel")
    # the identity-layout copy writes exactly calib_bytes; WRITE_SIZE counts
    # 64-byte write requests exactly
    batch = [g for g in wr if abs(wr[g] * kw - calib_bytes) > 0.01 * calib_bytes]
    assert len(batch) == 1 and batch[0] in f, (sorted(wr.items()), calib_bytes)
    g = batch[0]
    rec = {"workload": workload, "kernel_source_sha256": kernel_source_hash(),
           "calibration": f"torch bitwise_not copy, {calib_bytes} bytes read and written",
           "fetch_factor": round(kf, 4), "write_factor": round(kw, 4),
           "fetch_bytes_per_launch": round(f[g] * kf), "write_bytes_per_launch": round(wr[g] * kw),
           "bytes_per_launch": round(f[g] * kf + wr[g] * kw),
           "sources": [os.path.basename(fetch_csv), os.path.basename(write_csv)]}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec))


CPU_THREAD_CAP = 16   # the host CPU share of a one-GPU job on the MI355X boxes


def host_cpu():
    """nproc, the cores this process may run on, and the CPU model."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        allowed = os.cpu_count() or 1
    return {"nproc": os.cpu_count(), "cores_allowed": allowed, "model": model}


def cpu_baseline(w, lens, shards, budget_s, gpu_value, sbt=None, stage=None):
    """The oracle as it stands, on whole requests of the same workload, decode
    pages renumbered into a compact host pool (same rows, same bytes); a paged
    source is read in place through the request's row of the source block
    table; with prefill stages, the first stage's layers.  Two runs: one
    thread over the requests one by one (each a single-request problem, so
    its time is the oracle's per-request latency) until all are done or
    about budget_s seconds of CPU work; then the independent requests spread
    over the host's cores (at most CPU_THREAD_CAP threads; the C oracle
    releases the GIL) until all are done or about budget_s seconds of wall
    time.  `value` is the multi-threaded rate, `cores` the threads it used."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O

    f = {"fp16": O.FP16, "bf16": O.BF16, "e4m3fn": O.E4M3FN, "e5m2": O.E5M2}
    order = {"thd": O.TOKEN_MAJOR, "htd": O.HEAD_MAJOR, "paged": O.PAGED}[w.src_order]
    esz = 1 if w.cdt in ("e4m3fn", "e5m2") else 2   # the cache's element size
    L = stage[1] if stage else w.layers
    counts = [L * 2 * int(T) * w.hs * w.head_dim for T in lens]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)

    def one(r):
        """repack request r alone; returns (bytes read + written, tokens, seconds)"""
        T = int(lens[r])
        nb = (T + w.block_size - 1) // w.block_size
        extra = {}
        if sbt is not None:
            extra = dict(src_block_size=w.src_block_size, src_num_blocks=w.src_num_blocks,
                         src_block_table=sbt[r:r + 1], src_bt_stride=sbt.shape[1])
        if w.cache_dtype:
            extra["cache_fmt"] = f[w.cache_dtype]
        p = O.OracleProblem(L, w.heads, w.head_dim, w.src_tp, w.dst_tp, w.dst_rank,
                            f[w.src_dtype], f[w.dst_dtype], order, w.block_size, max(nb, 1), [T],
                            **extra)
        if sbt is not None:
            part = shards
        else:
            part = [None if s is None else
                    np.ascontiguousarray(s[offsets[r]:offsets[r] + counts[r]]) for s in shards]
        cache = np.empty(O.cache_bytes(p), dtype=np.uint8)
        sc = np.empty(O.scale_count(p), dtype=np.float32) if esz == 1 else None
        bt = np.arange(max(nb, 1), dtype=np.int32)[None, :]
        t = time.perf_counter()
        O.repack(p, part, cache, sc, bt, max(nb, 1))
        dt = time.perf_counter() - t
        rows = L * 2 * T * w.hd
        return rows * w.head_dim * (2 + esz) + (rows * 4 if esz == 1 else 0), T, dt

    host = host_cpu()
    # one thread: every request in turn, each timed alone
    done = spent = 0.0
    n1 = tok1 = 0
    per_req = []
    while n1 < len(lens) and spent < budget_s:
        b, T, dt = one(n1)
        done, spent, n1, tok1 = done + b, spent + dt, n1 + 1, tok1 + T
        per_req.append(dt * 1e3)
    gbs1 = done / spent / 1e9 if spent > 0 else None
    log(f"cpu oracle, 1 thread: {n1} requests, {done / 1e9:.2f} GB in {spent:.1f}s -> "
        f"{gbs1:.3f} GB/s")

    # independent requests on the host's cores
    threads = max(1, min(CPU_THREAD_CAP, host["cores_allowed"]))
    done = 0.0
    n = tok = 0
    t0 = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        while n < len(lens) and time.perf_counter() - t0 < budget_s:
            batch = list(range(n, min(len(lens), n + threads)))
            for b, T, _ in ex.map(one, batch):
                done, tok = done + b, tok + T
            n += len(batch)
    wall = time.perf_counter() - t0
    gbs = done / wall / 1e9 if wall > 0 else None
    log(f"cpu oracle, {threads} threads: {n} requests, {done / 1e9:.2f} GB in {wall:.1f}s -> "
        f"{gbs:.3f} GB/s")
    s = sorted(per_req)
    return {"value": round(gbs, 4) if gbs else None, "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"first {n} of {len(lens)} requests ({tok} tokens, {done / 1e9:.2f} GB read+"
                      f"written) of {w.name}, plain-C oracle, one request per thread on "
                      f"{threads} threads, pages renumbered into a compact host pool",
            "host": {**host, "threads_used": threads,
                     "thread_cap": f"{CPU_THREAD_CAP}: the host CPU share of a one-GPU job on "
                                   "this machine, whatever nproc reports"},
            "seconds": round(wall, 2),
            "single_thread": {"value": round(gbs1, 4) if gbs1 else None, "requests": n1,
                              "tokens": tok1, "seconds": round(spent, 2)},
            "latency_ms_per_request": {
                "p50": round(statistics.median(per_req), 3) if per_req else None,
                "p90": round(s[min(len(s) - 1, int(0.9 * len(s)))], 3) if s else None,
                "max": round(max(per_req), 3) if per_req else None, "requests": len(per_req),
                "note": "one thread, single-request problem, oracle call time"},
            "gpu_over_cpu": round(gpu_value / gbs, 1) if gbs else None}


if __name__ == "__main__":
    main()
