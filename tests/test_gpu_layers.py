"""GPU parity of pipeline-stage layer ranges: stage plans through the C ABI
(source buffers holding a prefill stage's layers, caches holding a decode
stage's layers) against the oracle, byte for byte.

Small cases compose every (source stage, decode stage) pair, through the
repack, through pack then unpack, or through the layer-streamed pipe (whose
chunks shift within the stage's layers), and compare whole decode-stage
pools with the oracle's whole-model pool; the full-size
case converts the Llama-3-8B workload from two prefill stages of 16 layers
into one decode cache and is checked on sampled requests and planes."""
import numpy as np
import pytest
import torch

from cases import (FP8_NAMES, FULL, SMALL, SMALL_DEQUANT, SMALL_PAGED, dst_size,
                   oracle_problem, read_shards)
from gpu_util import DEV, check_sampled, check_unused_pages, desc_for, dev_u16, log

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


def _stages(total, sizes):
    out, l0 = [], 0
    for n in sizes:
        out.append((l0, n))
        l0 += n
    assert l0 == total
    return out


def _stage_desc(w, lens, conv0, nconv, src_stage, dst_stage):
    d = desc_for(w, lens, nconv)
    d.src_layer_offset, d.src_layers = conv0 - src_stage[0], src_stage[1]
    d.dst_layer_offset, d.dst_layers = conv0 - dst_stage[0], dst_stage[1]
    return d


def _run_stage(w, lens, bt_d, stride, dshards, sbt_d, sstride, desc, cache, scales, how):
    """One stage plan: repack ("repack"), pack then unpack ("wire"), or the
    layer-streamed pipe in chunks of n layers over 2 slots ("pipeN").
    Host-side shape checks first: the shards hold the source stage's layers,
    the cache the decode stage's layers."""
    Hs, D = w.hs, w.head_dim
    if w.src_order == "paged":
        need = desc.src_layers * 2 * w.src_num_blocks * w.src_block_size * Hs * D
    else:
        need = sum(desc.src_layers * 2 * int(t) * Hs * D for t in lens)
    for j in read_shards(w):
        assert dshards[j].numel() >= need
    rows = desc.dst_layers * 2 * w.num_blocks * w.block_size * w.hd
    assert cache.numel() == rows * D * dst_size(w)
    assert scales is None or scales.numel() == rows
    plan = K.kvx_plan(desc)
    if how.startswith("pipe"):
        # chunks of the stage's converted layers (at most all of them); the
        # last may be shorter
        pipe = K.kvx_pipe_create(plan, min(int(how[4:]), desc.num_layers), 2)
        K.kvx_pipe_run(pipe, dshards, sbt_d, sstride, cache, scales, bt_d, stride)
        K.kvx_pipe_destroy(pipe)  # waits for the pipe's streams
    elif how == "wire":
        info = K.kvx_plan_info_get(plan)
        wire = torch.empty(max(int(info.wire_bytes), 16), dtype=torch.uint8, device=DEV)
        if sbt_d is not None:
            K.kvx_pack_paged(plan, dshards, sbt_d, sstride, wire)
        else:
            K.kvx_pack(plan, dshards, wire)
        K.kvx_unpack(plan, wire, cache, scales, bt_d, stride)
    elif sbt_d is not None:
        K.kvx_repack_paged(plan, dshards, sbt_d, sstride, cache, scales, bt_d, stride)
    else:
        K.kvx_repack(plan, dshards, cache, scales, bt_d, stride)


CASES = [("llama3_8b_small", 6, (3, 3), (2, 2, 2), "repack"),
         ("fp8_small", 5, (1, 4), (2, 3), "wire"),
         ("llama3_70b_small_r1", 4, (4,), (1, 1, 2), "repack"),
         ("qwen_htd_small", 5, (2, 1, 2), (5,), "wire"),
         ("paged16_tp4to2_bs32_small", 4, (2, 2), (3, 1), "repack"),
         ("paged16_e4m3_bs24", 3, (1, 2), (3,), "wire"),
         # the layer-streamed pipe over stage plans: chunks shifted within a
         # stage's layers, chunk sizes that do not divide them
         ("llama3_8b_small", 6, (3, 3), (2, 4), "pipe1"),
         ("fp8_small", 5, (1, 4), (2, 3), "pipe2"),
         ("llama3_70b_small_r1", 7, (4, 3), (7,), "pipe3"),
         ("paged16_tp4to2_bs32_small", 5, (2, 3), (4, 1), "pipe2"),
         ("dequant_bf16_e4m3_bf16", 6, (6,), (3, 3), "pipe2")]


@pytest.mark.parametrize("name,L,src_sizes,dst_sizes,how", CASES)
def test_stage_plans_small(name, L, src_sizes, dst_sizes, how):
    w = (SMALL | SMALL_PAGED | SMALL_DEQUANT)[name].replace(layers=L, total_layers=L)
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    log(f"stages {name}: prefill {src_sizes} -> decode {dst_sizes}, {how}")
    whole = oracle_problem(O, w, lens, L)
    want_c = np.full(O.cache_bytes(whole), W.SENTINEL, dtype=np.uint8)
    want_s = None
    if w.cdt in FP8_NAMES:
        want_s = np.full(4 * O.scale_count(whole), W.SENTINEL, dtype=np.uint8).view(np.float32)
    O.repack(whole, W.source_shards(w, lens, 0, L), want_c, want_s, bt, stride)

    bt_d = torch.from_numpy(bt).to(DEV)
    sbt_d, sstride = None, 0
    if w.src_order == "paged":
        sbt, sstride = W.src_block_table(w, lens)
        sbt_d = torch.from_numpy(sbt).to(DEV)
    src_st, dst_st = _stages(L, src_sizes), _stages(L, dst_sizes)
    src_bufs = [[dev_u16(s) for s in W.source_shards(w, lens, l0, n)] for l0, n in src_st]
    got_c, got_s = [], []
    for d0, dn in dst_st:
        rows = dn * 2 * w.num_blocks * w.block_size * w.hd
        cache = torch.full((rows * w.head_dim * dst_size(w),), W.SENTINEL, dtype=torch.uint8,
                           device=DEV)
        scales = None
        if w.cdt in FP8_NAMES:
            scales = torch.full((rows * 4,), W.SENTINEL, dtype=torch.uint8,
                                device=DEV).view(torch.float32)
        for (s0, sn), dsh in zip(src_st, src_bufs):
            lo, hi = max(s0, d0), min(s0 + sn, d0 + dn)
            if lo < hi:
                desc = _stage_desc(w, lens, lo, hi - lo, (s0, sn), (d0, dn))
                _run_stage(w, lens, bt_d, stride, dsh, sbt_d, sstride, desc, cache, scales,
                           how)
        torch.cuda.synchronize()
        got_c.append(cache.cpu().numpy())
        if scales is not None:
            got_s.append(scales.cpu().numpy())
    assert np.array_equal(np.concatenate(got_c), want_c)
    if want_s is not None:
        assert np.array_equal(np.concatenate(got_s).view(np.uint32), want_s.view(np.uint32))


def test_full_llama3_8b_two_prefill_stages():
    """The 8B workload from two prefill pipeline stages (layers 0-15 and
    16-31, each with its own source buffer) into one decode cache."""
    w = FULL["llama3_8b_bf16_bs16"]
    rng = np.random.default_rng(3)
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    bt_d = torch.from_numpy(bt).to(DEV)
    rows = w.layers * 2 * w.num_blocks * w.block_size * w.hd
    cache = torch.full((rows * w.head_dim * 2,), W.SENTINEL, dtype=torch.uint8, device=DEV)
    for s0 in (0, 16):
        log(f"full 8B: prefill stage layers {s0}..{s0 + 15}")
        dsh = [dev_u16(s) for s in W.source_shards(w, lens, s0, 16)]
        desc = _stage_desc(w, lens, s0, 16, (s0, 16), (0, 32))
        _run_stage(w, lens, bt_d, stride, dsh, None, 0, desc, cache, None, "repack")
        torch.cuda.synchronize()
        del dsh
    shards = W.source_shards(w, lens, 0, w.layers)
    planes = [(0, 0), (15, 1), (16, 0), (31, 1)]
    n = check_sampled(w, lens, bt, shards, cache, None, w.layers, planes, range(len(lens)), rng)
    check_unused_pages(w, lens, bt, cache, w.layers, rng)
    log(f"full 8B two stages: {n} rows checked")
