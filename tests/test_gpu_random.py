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
from gpu_util import DEV, check_shapes, desc_for, dev_u16, gpu_run, log, oracle_pool, pool

import oracle as O
import workload as W

import paper_2509_17542_amd as K

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


@pytest.mark.parametrize("name", list(RANDOM))
def test_random_pipe(name):
    """The layer-streamed pipe (one-layer chunks, two ring slots, so a third
    layer reuses the first slot) against the oracle's repack.  Decode tables
    keep their out-of-pool entries; source tables stay in the pool, since a
    row whose source page is outside it reaches the cache with whatever its
    ring slot held."""
    w = RANDOM[name]
    lens, bt, stride, shards = inputs(w)
    bt = out_of_pool(bt, w.num_blocks, np.random.default_rng(int(name[4:])))
    sbt = sbt_d = None
    if w.src_order == "paged":
        sbt, _ = W.src_block_table(w, lens)
        sbt_d = torch.from_numpy(np.ascontiguousarray(sbt, dtype=np.int32)).to(DEV)
    dsh = [dev_u16(x) for x in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    check_shapes(w, lens, bt, stride, dsh, w.layers, sbt)
    log(f"pipe {name}: L={w.layers} TP {w.src_tp}->{w.dst_tp} {w.src_dtype}->{w.dst_dtype}"
        f"{'->' + w.cache_dtype if w.cache_dtype else ''} {w.src_order} lens={list(lens)}")
    plan = K.kvx_plan(desc_for(w, lens))
    pipe = K.kvx_pipe_create(plan, 1, 2)
    cache, scales = pool(w, w.layers)
    K.kvx_pipe_run(pipe, dsh, sbt_d, 0 if sbt is None else sbt.shape[1], cache, scales, bt_d,
                   stride)
    K.kvx_pipe_destroy(pipe)  # waits for the pipe's streams
    torch.cuda.synchronize()
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards, sbt=sbt)
    got = cache.cpu().numpy()
    assert _eq(got, want_c), _diff(got, want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)
