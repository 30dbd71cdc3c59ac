"""GPU parity over seeded random descriptors: heads, TP degrees (merges,
splits, replicated heads), ranks, dtype pairs and dequantising caches, the
three source orders, head_dim 8..1024, page sizes that are not powers of two,
empty requests, and block tables with about 10% of their entries outside the
pool (rows of such pages are neither read nor written).  Whole pools and
transfer tensors through the C ABI against the oracle, byte for byte."""
import numpy as np
import pytest
import torch

from cases import RANDOM, inputs, oracle_problem, out_of_pool
from gpu_util import gpu_run, log, oracle_pool

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


def _case(name):
    """The workload, its inputs and its block tables with entries moved out of
    the pool (the same draw as the oracle's skip test)."""
    w = RANDOM[name]
    rng = np.random.default_rng(int(name[4:]))
    lens, bt, stride, shards = inputs(w)
    sbt = None
    if w.src_order == "paged":
        sbt, _ = W.src_block_table(w, lens)
        sbt = out_of_pool(sbt, w.src_num_blocks, rng)
    bt = out_of_pool(bt, w.num_blocks, rng)
    log(f"{name}: L={w.layers} H={w.heads} D={w.head_dim} TP {w.src_tp}->{w.dst_tp} "
        f"rank {w.dst_rank} {w.src_dtype}->{w.dst_dtype}{'->' + w.cache_dtype if w.cache_dtype else ''} "
        f"{w.src_order} bs={w.block_size} lens={list(lens)}")
    return w, lens, bt, stride, shards, sbt


@pytest.mark.parametrize("name", list(RANDOM))
def test_random_repack(name):
    w, lens, bt, stride, shards, sbt = _case(name)
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards, sbt=sbt)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards, sbt=sbt)
    got = cache.cpu().numpy()
    assert _eq(got, want_c), _diff(got, want_c)
    assert (scales is None) == (want_s is None)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


@pytest.mark.parametrize("name", list(RANDOM))
def test_random_pack_and_unpack(name):
    """Pack against the oracle's transfer tensor (padding and skipped rows
    untouched), then unpack of the oracle's transfer tensor."""
    w, lens, bt, stride, shards, sbt = _case(name)
    _, _, wire = gpu_run("pack", w, lens, bt, stride, shards, sbt=sbt)
    want = O.pack(oracle_problem(O, w, lens, sbt=sbt), shards)
    got = wire.cpu().numpy()[:want.size]
    assert _eq(got, want), _diff(got, want)
    cache, scales, _ = gpu_run("unpack", w, lens, bt, stride, None, wire_in=want, sbt=sbt)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards, op="unpack", wire=want, sbt=sbt)
    got = cache.cpu().numpy()
    assert _eq(got, want_c), _diff(got, want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)
