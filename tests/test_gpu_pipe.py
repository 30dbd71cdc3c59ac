"""GPU parity of the layer-streamed transfer (kvx_pipe_*): chunks of layers
packed, copied through a pinned host ring and unpacked, against the oracle's
whole-plan conversion, byte for byte (whole pools for the small cases, sampled
pages for the full Llama-3-8B workload).  Chunk sizes that do and do not
divide the layer count, one to three slots, two runs in a row on one pipe."""
import numpy as np
import pytest
import torch

from cases import FULL, SMALL, SMALL_DEQUANT, SMALL_E5M2, SMALL_PAGED, dst_size, inputs
from gpu_util import (DEV, check_sampled, check_shapes, check_unused_pages, desc_for, dev_u16, log,
                      oracle_pool, pool)

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


def _pipe_run(w, lens, bt, stride, shards, chunk, slots, runs=1):
    plan = K.kvx_plan(desc_for(w, lens))
    pipe = K.kvx_pipe_create(plan, chunk, slots)
    info = K.kvx_pipe_info_get(pipe)
    assert info.num_chunks == -(-w.layers // chunk) and info.host_bytes == slots * info.slot_bytes
    dsh = [dev_u16(s) for s in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    sbt = sbt_d = None
    sstride = 0
    if w.src_order == "paged":
        sbt, sstride = W.src_block_table(w, lens)
        sbt_d = torch.from_numpy(sbt).to(DEV)
    check_shapes(w, lens, bt, stride, dsh, w.layers, sbt)
    out = []
    for _ in range(runs):
        cache, scales = pool(w, w.layers)
        K.kvx_pipe_run(pipe, dsh, sbt_d, sstride, cache, scales, bt_d, stride)
        torch.cuda.synchronize()
        out.append((cache, scales))
    del pipe
    return out


CASES = [("llama3_8b_small", 1, 1), ("fp8_small", 1, 2), ("qwen_htd_small", 2, 3),
         ("llama3_70b_small_r1", 1, 3), ("fp16_e4m3_htd_empty", 1, 1),
         ("paged16_tp4to2_bs32_small", 1, 2), ("paged16_e4m3_bs24", 2, 1),
         ("gqa_src_rep_tp8to2_r1", 2, 2), ("bf16_fp16_overflow", 1, 2),
         ("dequant_bf16_e4m3_bf16", 1, 2), ("dequant_paged_tp4to2_bf16", 2, 1),
         ("e5m2_bf16", 2, 2), ("e5m2_dequant_fp16_empty", 1, 1)]


@pytest.mark.parametrize("name,chunk,slots", CASES)
def test_pipe_small(name, chunk, slots):
    w = (SMALL | SMALL_PAGED | SMALL_DEQUANT | SMALL_E5M2)[name]
    lens, bt, stride, shards = inputs(w)
    log(f"pipe {name}: chunk {chunk} of {w.layers} layers, {slots} slots")
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
    for cache, scales in _pipe_run(w, lens, bt, stride, shards, chunk, slots, runs=2):
        assert np.array_equal(cache.cpu().numpy(), want_c)
        if want_s is not None:
            assert np.array_equal(scales.cpu().numpy().view(np.uint32), want_s.view(np.uint32))


@pytest.mark.parametrize("chunk,slots", [(1, 2), (2, 3), (3, 2), (5, 1)])
def test_pipe_chunkings_of_five_layers(chunk, slots):
    w = SMALL["llama3_70b_small_r0"].replace(layers=5, total_layers=5)
    lens, bt, stride, shards = inputs(w)
    log(f"pipe 5 layers: chunk {chunk}, {slots} slots")
    want_c, _ = oracle_pool(w, lens, bt, stride, shards)
    (cache, _), = _pipe_run(w, lens, bt, stride, shards, chunk, slots)
    assert np.array_equal(cache.cpu().numpy(), want_c)


def test_pipe_full_llama3_8b():
    w = FULL["llama3_8b_bf16_bs16"]
    rng = np.random.default_rng(5)
    lens, bt, stride, shards = inputs(w)
    log("pipe full 8B: chunks of 4 layers, 3 slots")
    (cache, _), = _pipe_run(w, lens, bt, stride, shards, 4, 3)
    planes = [(0, 0), (3, 1), (4, 0), (31, 1), (17, 0)]
    n = check_sampled(w, lens, bt, shards, cache, None, w.layers, planes, range(len(lens)), rng)
    check_unused_pages(w, lens, bt, cache, w.layers, rng)
    log(f"pipe full 8B: {n} rows checked")


def test_pipe_run_with_a_missing_shard_fails_then_runs():
    """A run whose first pack is refused (a NULL shard, passed straight to the
    C call) returns KVX_EINVAL with nothing but stream waits enqueued; the
    caller's stream still completes, and the next run of the same pipe gives
    the whole-plan result."""
    w = SMALL["llama3_8b_small"]
    lens, bt, stride, shards = inputs(w)
    plan = K.kvx_plan(desc_for(w, lens))
    pipe = K.kvx_pipe_create(plan, 1, 2)
    dsh = [dev_u16(s) for s in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    cache, scales = pool(w, w.layers)
    null = (K._vp * 1)()
    st = K._lib.kvx_pipe_run(pipe, null, None, 0, cache.data_ptr(), None, bt_d.data_ptr(), stride,
                             torch.cuda.current_stream().cuda_stream)
    assert st == K.EINVAL and "NULL" in K.kvx_last_error()
    torch.cuda.synchronize()
    assert bool((cache == W.SENTINEL).all())
    K.kvx_pipe_run(pipe, dsh, None, 0, cache, scales, bt_d, stride)
    torch.cuda.synchronize()
    want_c, _ = oracle_pool(w, lens, bt, stride, shards)
    assert np.array_equal(cache.cpu().numpy(), want_c)
    del pipe


def _stream(kind):
    return torch.cuda.Stream() if kind == "side" else torch.cuda.current_stream()


@pytest.mark.parametrize("kind", ["side", "default"])
@pytest.mark.parametrize("name", ["llama3_8b_small", "fp8_small"])
def test_pipe_orders_with_the_callers_stream(name, kind):
    """On a created stream (an event each way) and on the default (legacy
    null) stream (the pipe enqueues nothing there; its streams synchronise
    with it by themselves): the pipe's stages start after the stream's
    earlier work (the pool filled with sentinels on it just before the run,
    over junk written before that), and the stream's later work (a copy of
    the pool) sees the whole result, with no device synchronisation in
    between."""
    w = (SMALL | SMALL_DEQUANT)[name]
    lens, bt, stride, shards = inputs(w)
    log(f"pipe {name} on the {kind} stream")
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
    plan = K.kvx_plan(desc_for(w, lens))
    pipe = K.kvx_pipe_create(plan, 1, 2)
    dsh = [dev_u16(s) for s in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    check_shapes(w, lens, bt, stride, dsh, w.layers)
    cache, scales = pool(w, w.layers, fill=0x5A)
    torch.cuda.synchronize()
    st = _stream(kind)
    for _ in range(2):
        with torch.cuda.stream(st):
            cache.fill_(W.SENTINEL)
            if scales is not None:
                scales.view(torch.uint8).fill_(W.SENTINEL)
            K.kvx_pipe_run(pipe, dsh, None, 0, cache, scales, bt_d, stride, st)
            got_c = cache.clone()
            got_s = None if scales is None else scales.clone()
            cache.fill_(0x5A)  # later work on the stream must not overtake the copies
        st.synchronize()
        assert np.array_equal(got_c.cpu().numpy(), want_c)
        if want_s is not None:
            assert np.array_equal(got_s.cpu().numpy().view(np.uint32), want_s.view(np.uint32))
    del pipe


@pytest.mark.parametrize("kind", ["side", "default"])
def test_pipe_runs_back_to_back(kind):
    """Three runs of one pipe enqueued one after another with nothing between
    them, into three pools: the pipe orders its own runs (they share the
    slots), so each pool holds the whole result.  Three chunks over two
    slots, so every run reuses a slot of the one before."""
    w = SMALL["llama3_70b_small_r1"].replace(layers=3, total_layers=3)
    lens, bt, stride, shards = inputs(w)
    log(f"pipe back to back on the {kind} stream")
    want_c, _ = oracle_pool(w, lens, bt, stride, shards)
    plan = K.kvx_plan(desc_for(w, lens))
    pipe = K.kvx_pipe_create(plan, 1, 2)
    dsh = [dev_u16(s) for s in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    check_shapes(w, lens, bt, stride, dsh, w.layers)
    pools = [pool(w, w.layers)[0] for _ in range(3)]
    torch.cuda.synchronize()
    st = _stream(kind)
    for c in pools:
        K.kvx_pipe_run(pipe, dsh, None, 0, c, None, bt_d, stride, st)
    st.synchronize()
    torch.cuda.synchronize()
    for c in pools:
        assert np.array_equal(c.cpu().numpy(), want_c)
    del pipe


def test_two_pipes_run_at_once():
    """Two pipes of one plan, each with its own ring, run on two created
    streams at the same time (runs of different pipes may overlap), with
    their own sources and pools; each pool holds its own whole result.  Three
    chunks over two slots in each pipe."""
    w = SMALL["fp8_small"].replace(layers=3, total_layers=3)
    lens, bt, stride, shards = inputs(w)
    variants = [shards, [None if s is None else np.roll(s, 37) for s in shards]]
    plan = K.kvx_plan(desc_for(w, lens))
    pipes = [K.kvx_pipe_create(plan, 1, 2) for _ in variants]
    dsh = [[dev_u16(s) for s in v] for v in variants]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    for d in dsh:
        check_shapes(w, lens, bt, stride, d, w.layers)
    pools = [pool(w, w.layers) for _ in variants]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in variants]
    log("two pipes at once on two streams")
    for _ in range(2):
        for p, d, (c, s), st in zip(pipes, dsh, pools, streams):
            K.kvx_pipe_run(p, d, None, 0, c, s, bt_d, stride, st)
    torch.cuda.synchronize()
    for v, (c, s) in zip(variants, pools):
        want_c, want_s = oracle_pool(w, lens, bt, stride, v)
        assert np.array_equal(c.cpu().numpy(), want_c)
        assert np.array_equal(s.view(torch.uint8).cpu().numpy(), want_s.view(np.uint8))
    del pipes
