"""GPU parity of the e5m2 transfer format (OCP e5m2 codes with per-row fp32
scales max|x| / 57344, a saturating round-to-nearest-even cast; and the
dequantising unpack of e5m2 codes into a 16-bit cache): the HIP path through
the C ABI against the oracle, byte for byte.

Small cases compare whole pools or transfer tensors.  Sweeps cover every
finite 16-bit source pattern under chosen row maxima (around 57344 and the
limits of the kernel's two-step divide), every code under special scales, and
quantise + dequantise in one repack.  The full Llama-3-8B workload runs in the
benchmark's launch configuration and is checked on sampled pages."""
import numpy as np
import pytest
import torch

from cases import (FULL, SMALL_E5M2, double_rounding_scales, e4m3_sweep_rows, inputs,
                   oracle_problem, pad_rows, sweep_case)
from gpu_util import (check_sampled, check_unused_pages, gpu_run, log, oracle_pool)

import oracle as O
import workload as W

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


@pytest.fixture(autouse=True)
def _release_device_memory():
    yield
    import gc
    gc.collect()
    torch.cuda.empty_cache()


def _eq(a, b):
    return np.array_equal(np.asarray(a).view(np.uint8), np.asarray(b).view(np.uint8))


def _diff(got, want):
    bad = np.nonzero(np.asarray(got).view(np.uint8) != np.asarray(want).view(np.uint8))[0]
    return f"{bad.size} bytes differ, first at {bad[:6]}"


@pytest.mark.parametrize("name", list(SMALL_E5M2))
def test_e5m2_repack_small(name):
    w = SMALL_E5M2[name]
    lens, bt, stride, shards = inputs(w)
    log(f"e5m2 repack {name} lens={list(lens)}")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
    got = cache.cpu().numpy()
    assert _eq(got, want_c), _diff(got, want_c)
    assert (scales is None) == (want_s is None)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


@pytest.mark.parametrize("name", list(SMALL_E5M2))
def test_e5m2_pack_small(name):
    w = SMALL_E5M2[name]
    lens, bt, stride, shards = inputs(w)
    log(f"e5m2 pack {name}")
    _, _, wire = gpu_run("pack", w, lens, bt, stride, shards)
    want = O.pack(oracle_problem(O, w, lens), shards)
    got = wire.cpu().numpy()[:want.size]
    assert _eq(got, want), _diff(got, want)


@pytest.mark.parametrize("name", list(SMALL_E5M2))
def test_e5m2_unpack_small(name):
    """Unpack alone, fed the oracle's transfer tensor."""
    w = SMALL_E5M2[name]
    lens, bt, stride, shards = inputs(w)
    wire = O.pack(oracle_problem(O, w, lens), shards)
    log(f"e5m2 unpack {name}")
    cache, scales, _ = gpu_run("unpack", w, lens, bt, stride, None, wire_in=wire)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards, op="unpack", wire=wire)
    assert _eq(cache.cpu().numpy(), want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


def _amaxes(fmt, rng):
    if fmt == "bf16":
        # subnormal and tiny maxima, around 57344 (0x4760), around the fast
        # path's limits 2^-80 * 57344 and 2^100 * 57344, the largest
        fixed = [0x0001, 0x0080, 0x00FF, 0x1F00, 0x1F80, 0x1FA0, 0x3F80, 0x475F, 0x4760,
                 0x4761, 0x7970, 0x7980, 0x7990, 0x7F7F]
        return sorted(set(fixed) | set(rng.integers(1, 0x7F80, 12).tolist()))
    # fp16: subnormal, smallest normal, 1, around 57344 (0x7B00), the largest
    fixed = [0x0001, 0x03FF, 0x0400, 0x3C00, 0x7AFF, 0x7B00, 0x7B01, 0x7BFF]
    return sorted(set(fixed) | set(rng.integers(1, 0x7C00, 8).tolist()))


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_e5m2_sweep(fmt):
    """Rows covering every finite source pattern under each row maximum, plus
    NaN / Inf / zero rows: codes and scales of the repack into an e5m2 cache."""
    rng = np.random.default_rng(515)
    rows = pad_rows(e4m3_sweep_rows(fmt, _amaxes(fmt, rng), rng))
    w, lens, bt, shards = sweep_case(fmt, "e5m2", rows)
    log(f"{fmt}->e5m2 sweep: {rows.shape[0]} rows")
    cache, scales, _ = gpu_run("repack", w, lens, bt, bt.shape[1], shards)
    want_c, want_s = oracle_pool(w, lens, bt, bt.shape[1], shards)
    got = cache.cpu().numpy()
    assert _eq(got, want_c), _diff(got, want_c)
    assert _eq(scales.cpu().numpy(), want_s)


@pytest.mark.parametrize("src,cache", [("bf16", "bf16"), ("bf16", "fp16"), ("fp16", "bf16"),
                                       ("fp16", "fp16")])
def test_e5m2_quantise_dequantise_sweep(src, cache):
    rng = np.random.default_rng(516)
    rows = pad_rows(e4m3_sweep_rows(src, _amaxes(src, rng)[::2], rng))
    w, lens, bt, shards = sweep_case(src, "e5m2", rows)
    w = w.replace(cache_dtype=cache)
    log(f"{src}->e5m2->{cache} sweep: {rows.shape[0]} rows")
    got, scales, _ = gpu_run("repack", w, lens, bt, bt.shape[1], shards)
    assert scales is None
    want, _ = oracle_pool(w, lens, bt, bt.shape[1], shards)
    got = got.cpu().numpy()
    assert _eq(got, want), _diff(got, want)


SPECIAL_SCALES = [0.0, -0.0, 2.0 ** -149, 1e-40, 2.0 ** -130, 2.0 ** -126, 2.0 ** -100,
                  1.0 / 57344, 1.0, 3.0, 57344.0, 2.0 ** 100, 3.4e38, np.inf, -np.inf, np.nan,
                  -1.5]


@pytest.mark.parametrize("cache_dtype", ["bf16", "fp16"])
def test_e5m2_dequant_every_code_under_special_scales(cache_dtype):
    """A transfer tensor written here: pairs of rows holding all 256 codes
    (infinities and NaNs included), each pair under one scale."""
    rng = np.random.default_rng(4)
    dr = double_rounding_scales(8) + double_rounding_scales(11)
    extra = 64 - len(SPECIAL_SCALES) - len(dr)
    scales = np.array(SPECIAL_SCALES + dr + list(rng.choice([-1.0, 1.0], extra) *
                                                 2.0 ** rng.uniform(-150, 128, extra)),
                      dtype=np.float32)
    rows = 2 * scales.size
    T = rows // 2
    w = W.Workload("codes5", 1, 1, 1, 128, 1, 1, 0, "bf16", "e5m2", "thd", 16, T // 16, 1, T, T,
                   seed=1, cache_dtype=cache_dtype)
    lens = np.array([T], dtype=np.int32)
    bt = np.arange(T // 16, dtype=np.int32)[None, :]
    doff, soff, total = O.wire_layout(oracle_problem(O, w, lens))
    wire = np.zeros(int(total), dtype=np.uint8)
    codes = (np.arange(rows * 128) % 256).astype(np.uint8)
    wire[int(doff[0]):int(doff[0]) + codes.size] = codes
    wire[int(soff[0]):int(soff[0]) + 4 * rows].view(np.float32)[:] = np.repeat(scales, 2)
    log(f"e5m2 codes -> {cache_dtype}: {scales.size} scales")
    cache, _, _ = gpu_run("unpack", w, lens, bt, bt.shape[1], None, wire_in=wire)
    want, _ = oracle_pool(w, lens, bt, bt.shape[1], None, op="unpack", wire=wire)
    got = cache.cpu().numpy()
    bad = np.nonzero(got.view(np.uint16) != want.view(np.uint16))[0]
    assert bad.size == 0, (f"{bad.size} elements differ, first {bad[:4]}: "
                           f"got {got.view(np.uint16)[bad[:4]]} want {want.view(np.uint16)[bad[:4]]}")


def test_full_llama3_8b_e5m2():
    w = FULL["llama3_8b_bf16_e5m2_bs16"]
    rng = np.random.default_rng(7)
    lens, bt, stride, shards = inputs(w)
    log(f"full {w.name}: repack on GPU ({int(lens.sum())} tokens)")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    edge = [(0, 0), (w.layers - 1, 1)]
    n = check_sampled(w, lens, bt, shards, cache, scales, w.layers, edge, range(len(lens)), rng)
    planes = [(int(rng.integers(w.layers)), int(rng.integers(2))) for _ in range(2)]
    n += check_sampled(w, lens, bt, shards, cache, scales, w.layers, planes,
                       rng.choice(len(lens), 4, replace=False), rng)
    check_unused_pages(w, lens, bt, cache, w.layers, rng)
    log(f"full {w.name}: {n} rows checked")
