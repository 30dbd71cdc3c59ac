"""The benchmark's command line and its one JSON line.

The CPU test checks that a run asked for more than one GPU stops with a
message before touching any device.  The GPU test runs the benchmark on the
tiny workload (2 layers, 4 heads, dim 64, one 256-token request) in a child
process and checks the fields of the line it prints: the metric, whole-job
throughput, the roofline of the repack kernel and the CPU oracle baseline.
"""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True,
                       timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr or "single MI355X" in r.stderr
    assert r.stdout == ""


@pytest.mark.gpu
def test_bench_prints_one_json_line():
    r = subprocess.run([sys.executable, BENCH, "--workload", "tiny_tp1to2_fp16_bf16", "--steps", "3",
                        "--warmup", "1", "--stream-chunk", "0", "--calib-gib", "0.25",
                        "--cpu-seconds", "0.5", "--configs", "tiny_tp1to2_fp16_bf16"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1
    out = json.loads(lines[0])
    sys.path.insert(0, ROOT)
    import bench
    assert out["metric"] == bench.METRIC
    assert out["unit"] == "GB/s" and out["n_gpus"] == 1 and out["higher_is_better"] is True
    assert out["steps"] == 3 and out["warmup"] == 1 and out["data"] == "synthetic"
    assert out["value"] > 0 and out["ms_per_step"] > 0
    cfg = out["config"]
    assert cfg["workload"] == "tiny_tp1to2_fp16_bf16"
    # 2 layers x 2 planes x 256 tokens x 2 decode heads x 64 dims x (2 + 2) bytes
    assert cfg["bytes_per_step"] == 2 * 2 * 256 * 2 * 64 * 4
    assert out["dtype"] == "fp16->bf16"
    roof = out["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert roof["achieved"] > 0 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    assert roof["algorithmic_bytes_per_launch"] == cfg["bytes_per_step"]
    assert roof["traffic"] is None   # counters were taken on another workload
    cpu = out["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["unit"] == "GB/s"
    assert cpu["value"] > 0 and cpu["cores"] >= 1 and cpu["sample"]
    assert cpu["host"]["nproc"] >= 1 and cpu["host"]["threads_used"] == cpu["cores"]
    assert cpu["latency_ms_per_request"]["p50"] > 0
    cfg_leg = out["configs"]["tiny_tp1to2_fp16_bf16"]
    assert cfg_leg["repack"]["GB/s"] > 0 and cfg_leg["latency_ms_per_request"]["p50"] > 0
    assert out["latency_ms_per_request"]["p50"] > 0
    assert out["pack"]["GB/s"] > 0 and out["unpack"]["GB/s"] > 0
    assert out["pack_unpack"]["GB/s"] > 0
    fill = out["copy_ceiling"]["torch_fill_write_only"]
    assert fill["bytes_read"] == 0 and fill["GB/s"] > 0
    peak = out["hbm_peak_from_device"]
    assert peak is None or (peak["bus_width_bits"] > 0 and peak["GB/s"] > 0)


def test_settle_counts_launches_until_the_time_has_passed():
    """The configs leg's warm-up: at least the given launches, then whole
    groups of them until the wall time has passed (a fake launch of 1 ms)."""
    import time
    import types
    sys.path.insert(0, ROOT)
    import bench
    calls = []
    fake_torch = types.SimpleNamespace(cuda=types.SimpleNamespace(synchronize=lambda: None))

    def launch():
        calls.append(1)
        time.sleep(0.001)

    n = bench.settle(launch, fake_torch, 3, 0.0)
    assert n == 3 and len(calls) == 3
    calls.clear()
    n = bench.settle(launch, fake_torch, 3, 20.0)
    assert n == len(calls) and n % 3 == 0 and 18 <= n <= 60
    calls.clear()
    assert bench.settle(launch, fake_torch, 0, 5.0) == len(calls) >= 4
