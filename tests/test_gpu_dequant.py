"""GPU parity of the dequantising unpack (an e4m3fn transfer tensor with
per-row fp32 scales restored into a 16-bit decode cache, each element the fp32
product q * s rounded to nearest even): the HIP path through the C ABI against
the oracle, byte for byte.

Small cases compare whole pools (repack, unpack of the oracle's transfer
tensor, pack + unpack = repack).  A direct sweep unpacks every e4m3fn code
under special and random scales (zero, fp32 subnormals, the fp16 overflow
edge, infinities, NaN, negative).  The full Llama-3-8B workload runs in the
benchmark's launch configuration and is checked on sampled pages."""
import numpy as np
import pytest
import torch

from cases import (FULL, SMALL_DEQUANT, double_rounding_scales, e4m3_sweep_rows, inputs,
                   oracle_problem, pad_rows, sweep_case)
from gpu_util import (DEV, check_sampled, check_unused_pages, gpu_run, log, oracle_pool)

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


@pytest.mark.parametrize("name", list(SMALL_DEQUANT))
def test_dequant_repack_small(name):
    w = SMALL_DEQUANT[name]
    lens, bt, stride, shards = inputs(w)
    log(f"dequant repack {name} lens={list(lens)}")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    assert scales is None
    want, want_s = oracle_pool(w, lens, bt, stride, shards)
    assert want_s is None
    assert _eq(cache.cpu().numpy(), want)


@pytest.mark.parametrize("name", list(SMALL_DEQUANT))
def test_dequant_unpack_small(name):
    """Unpack alone, fed the oracle's transfer tensor."""
    w = SMALL_DEQUANT[name]
    lens, bt, stride, shards = inputs(w)
    wire = O.pack(oracle_problem(O, w, lens), shards)
    log(f"dequant unpack {name}")
    cache, _, _ = gpu_run("unpack", w, lens, bt, stride, None, wire_in=wire)
    want, _ = oracle_pool(w, lens, bt, stride, shards, op="unpack", wire=wire)
    assert _eq(cache.cpu().numpy(), want)


@pytest.mark.parametrize("name", list(SMALL_DEQUANT))
def test_dequant_pack_then_unpack_equals_repack(name):
    w = SMALL_DEQUANT[name]
    lens, bt, stride, shards = inputs(w)
    log(f"dequant pack+unpack {name}")
    c1, _, wire = gpu_run("pack_unpack", w, lens, bt, stride, shards)
    c2, _, _ = gpu_run("repack", w, lens, bt, stride, shards)
    assert torch.equal(c1, c2)
    # the transfer tensor is the plain e4m3fn plan's
    want = O.pack(oracle_problem(O, w.replace(cache_dtype=""), lens), shards)
    assert _eq(wire.cpu().numpy()[:want.size], want)


SPECIAL_SCALES = [0.0, -0.0, 2.0 ** -149, 1e-40, 2.0 ** -130, 2.0 ** -126, 2.0 ** -100,
                  2.0 ** -80, 1.0 / 448, 1.0, 3.0, 448.0, 65504.0 / 448, 146.3, 2.0 ** 100,
                  2.0 ** 120, 3.4e38, np.inf, -np.inf, np.nan, -1.5]


@pytest.mark.parametrize("cache_dtype", ["bf16", "fp16"])
def test_dequant_every_code_under_special_scales(cache_dtype):
    """A transfer tensor written here: pairs of rows that hold all 256 codes,
    each pair under one scale (the special ones above, scales whose products
    round differently through fp32 than at once, then 2^U(-150, 128) with
    random signs); one request, TP1, one head, 16-token pages in order."""
    rng = np.random.default_rng(3)
    dr = double_rounding_scales(8) + double_rounding_scales(11)
    extra = 64 - len(SPECIAL_SCALES) - len(dr)
    assert extra > 8
    scales = np.array(SPECIAL_SCALES + dr + list(rng.choice([-1.0, 1.0], extra) *
                                                 2.0 ** rng.uniform(-150, 128, extra)),
                      dtype=np.float32)
    rows = 2 * scales.size                     # 128 rows: 64 tokens, k and v
    T = rows // 2
    w = W.Workload("codes", 1, 1, 1, 128, 1, 1, 0, "bf16", "e4m3fn", "thd", 16, T // 16, 1, T, T,
                   seed=1, cache_dtype=cache_dtype)
    lens = np.array([T], dtype=np.int32)
    bt = np.arange(T // 16, dtype=np.int32)[None, :]
    p = oracle_problem(O, w, lens)
    doff, soff, total = O.wire_layout(p)
    wire = np.zeros(int(total), dtype=np.uint8)
    codes = (np.arange(rows * 128) % 256).astype(np.uint8)
    wire[int(doff[0]):int(doff[0]) + codes.size] = codes
    wire[int(soff[0]):int(soff[0]) + 4 * rows].view(np.float32)[:] = np.repeat(scales, 2)
    log(f"dequant codes -> {cache_dtype}: {scales.size} scales")
    cache, _, _ = gpu_run("unpack", w, lens, bt, bt.shape[1], None, wire_in=wire)
    want, _ = oracle_pool(w, lens, bt, bt.shape[1], None, op="unpack", wire=wire)
    got = cache.cpu().numpy()
    bad = np.nonzero(got.view(np.uint16) != want.view(np.uint16))[0]
    assert bad.size == 0, (f"{bad.size} elements differ, first {bad[:4]}: "
                           f"got {got.view(np.uint16)[bad[:4]]} want {want.view(np.uint16)[bad[:4]]}")


@pytest.mark.parametrize("src,cache", [("bf16", "bf16"), ("bf16", "fp16"), ("fp16", "bf16"),
                                       ("fp16", "fp16")])
def test_quantise_dequantise_sweep(src, cache):
    """The repack through e4m3fn into a 16-bit cache on rows that cover every
    finite source pattern under chosen row maxima (subnormal, around 448,
    around the two-step divide's limits, the largest) plus NaN / Inf / zero
    rows: quantisation and dequantisation in one kernel, against the oracle."""
    rng = np.random.default_rng(77)
    if src == "bf16":
        amaxes = sorted(set([0x0001, 0x0080, 0x0100, 0x1000, 0x3F80, 0x43E0, 0x43E1, 0x7F7F,
                             0x7200, 0x7201, 0x1F80, 0x4780, 0x477F])
                        | set(rng.integers(1, 0x7F80, 6).tolist()))
    else:
        amaxes = sorted(set([0x0001, 0x03FF, 0x0400, 0x3C00, 0x5F00, 0x7BFF])
                        | set(rng.integers(1, 0x7C00, 6).tolist()))
    rows = pad_rows(e4m3_sweep_rows(src, amaxes, rng))
    w, lens, bt, shards = sweep_case(src, "e4m3fn", rows)
    w = w.replace(cache_dtype=cache)
    log(f"{src}->e4m3fn->{cache} sweep: {rows.shape[0]} rows, {len(amaxes)} row maxima")
    got, scales, _ = gpu_run("repack", w, lens, bt, bt.shape[1], shards)
    assert scales is None
    want, _ = oracle_pool(w, lens, bt, bt.shape[1], shards)
    got = got.cpu().numpy()
    bad = np.nonzero(got.view(np.uint16) != want.view(np.uint16))[0]
    assert bad.size == 0, (f"{bad.size} elements differ, first {bad[:4]}: "
                           f"got {got.view(np.uint16)[bad[:4]]} want {want.view(np.uint16)[bad[:4]]}")


def test_full_llama3_8b_dequant():
    w = FULL["llama3_8b_bf16_e4m3_bf16_bs16"]
    rng = np.random.default_rng(7)
    lens, bt, stride, shards = inputs(w)
    log(f"full {w.name}: repack on GPU ({int(lens.sum())} tokens)")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    edge = [(0, 0), (w.layers - 1, 1)]
    n = check_sampled(w, lens, bt, shards, cache, scales, w.layers, edge, range(len(lens)), rng)
    planes = [(int(rng.integers(w.layers)), int(rng.integers(2))) for _ in range(2)]
    picks = rng.choice(len(lens), 4, replace=False)
    n += check_sampled(w, lens, bt, shards, cache, scales, w.layers, planes, picks, rng)
    check_unused_pages(w, lens, bt, cache, w.layers, rng)
    log(f"full {w.name}: {n} rows checked")
