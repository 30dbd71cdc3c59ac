"""Pack, unpack and repack recorded into a HIP graph and replayed, against
the oracle and against eager launches, byte for byte, through the C ABI.

The launch path of these calls allocates nothing, copies nothing and does
not synchronise (the plan uploads its work-item table when it is built), so
a serving loop may record a transfer once and replay it with new contents
in the same buffers.  Each case records one call (torch.cuda.CUDAGraph on
its capture stream) over buffers allocated beforehand, then replays it three
times.  Before every replay the host writes new source values and a new
block table into the same device buffers and refills the outputs with the
sentinel (fill kernels and copies outside the graph, then a synchronisation),
so each replay must read what is there at replay time.  Every replay is
compared with the oracle on those inputs and with an eager launch of the
same call.

The allocation-free repack rebuilds its static work-item table inside the
graph; between its replays an eager call on a different problem overwrites
that table, and the next replay must still be exact.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workload as W
from cases import SMALL, SMALL_DEQUANT, SMALL_E5M2, SMALL_PAGED, inputs
from gpu_util import DEV, check_shapes, desc_for, dev_u16, log, oracle_pool, pool

import paper_2509_17542_amd as K

pytestmark = pytest.mark.gpu

REPLAYS = 3


def _variant(w, lens, bt, shards, k, rng):
    """Inputs of replay k: the source values rotated by a k-dependent offset
    and the in-pool page ids sent through a fixed permutation of the pool
    (out-of-pool ids stay, so the kernel still skips them)."""
    new_shards = [None if s is None else np.roll(s, 7919 * k) for s in shards]
    perm = rng.permutation(w.num_blocks).astype(np.int32)
    inside = (bt >= 0) & (bt < w.num_blocks)
    new_bt = np.where(inside, perm[np.clip(bt, 0, w.num_blocks - 1)], bt).astype(np.int32)
    return new_bt, new_shards


def _write(dshards, bt_d, new_bt, new_shards, outs):
    """Host-side update of the recorded buffers between replays."""
    for d, s in zip(dshards, new_shards):
        if d is not None:
            d.copy_(torch.from_numpy(s.view(np.int16)))
    bt_d.copy_(torch.from_numpy(new_bt))
    for o in outs:
        if o is not None:
            o.view(torch.uint8).fill_(W.SENTINEL)
    torch.cuda.synchronize()


def _record(call):
    """Warm the call up once eagerly on a side stream, then record it."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        call()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call()  # the binding passes the current stream: the capture stream
    torch.cuda.synchronize()
    return g


def _equal(name, k, cache, scales, ref_cache, ref_scales, what):
    assert np.array_equal(cache.cpu().numpy(), ref_cache), f"{name} replay {k}: cache != {what}"
    if scales is not None:
        got = scales.view(torch.uint8).cpu().numpy()
        want = ref_scales.view(np.uint8) if isinstance(ref_scales, np.ndarray) else \
            ref_scales.view(torch.uint8).cpu().numpy()
        assert np.array_equal(got, want), f"{name} replay {k}: scales != {what}"


def _setup(w):
    lens, bt, stride, shards = inputs(w)
    dshards = [dev_u16(s) for s in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    sbt = sbt_d = None
    if w.src_order == "paged":
        sbt, _ = W.src_block_table(w, lens)
        sbt = np.ascontiguousarray(sbt, dtype=np.int32)
        sbt_d = torch.from_numpy(sbt).to(DEV)
    check_shapes(w, lens, bt, stride, dshards, w.layers, sbt)
    return lens, bt, stride, shards, dshards, bt_d, sbt, sbt_d


def _repack_call(w, plan, dshards, sbt, sbt_d, cache, scales, bt_d, stride):
    if w.src_order == "paged":
        return lambda: K.kvx_repack_paged(plan, dshards, sbt_d, sbt.shape[1], cache, scales,
                                          bt_d, stride)
    return lambda: K.kvx_repack(plan, dshards, cache, scales, bt_d, stride)


REPACK = {
    "llama3_8b_small": SMALL["llama3_8b_small"],
    "qwen_htd_small": SMALL["qwen_htd_small"],
    "llama3_70b_small_r1": SMALL["llama3_70b_small_r1"],
    "fp8_small": SMALL["fp8_small"],
    "dequant_bf16_e4m3_bf16": SMALL_DEQUANT["dequant_bf16_e4m3_bf16"],
    "e5m2_bf16": SMALL_E5M2["e5m2_bf16"],
    "paged16_tp4to2_bs32_small": SMALL_PAGED["paged16_tp4to2_bs32_small"],
}


@pytest.mark.parametrize("name", list(REPACK))
def test_graph_replays_repack(name):
    w = REPACK[name]
    lens, bt, stride, shards, dshards, bt_d, sbt, sbt_d = _setup(w)
    plan = K.kvx_plan(desc_for(w, lens))
    cache, scales = pool(w, w.layers)
    eager_c, eager_s = pool(w, w.layers)
    log(f"graph repack {name}: record")
    g = _record(_repack_call(w, plan, dshards, sbt, sbt_d, cache, scales, bt_d, stride))
    eager = _repack_call(w, plan, dshards, sbt, sbt_d, eager_c, eager_s, bt_d, stride)
    rng = np.random.default_rng(1000 + len(name))
    for k in range(1, REPLAYS + 1):
        new_bt, new_shards = _variant(w, lens, bt, shards, k, rng)
        _write(dshards, bt_d, new_bt, new_shards, (cache, scales, eager_c, eager_s))
        log(f"graph repack {name}: replay {k}")
        g.replay()
        eager()
        torch.cuda.synchronize()
        ref_c, ref_s = oracle_pool(w, lens, new_bt, stride, new_shards, sbt=sbt)
        _equal(name, k, cache, scales, ref_c, ref_s, "oracle")
        _equal(name, k, cache, scales, eager_c.cpu().numpy(), eager_s, "eager launch")


PACK_UNPACK = {
    "llama3_70b_small_r1": SMALL["llama3_70b_small_r1"],
    "fp8_small": SMALL["fp8_small"],
    "paged16_bs64_small": SMALL_PAGED["paged16_bs64_small"],
    "dequant_fp16_e4m3_fp16_htd": SMALL_DEQUANT["dequant_fp16_e4m3_fp16_htd"],
    "e5m2_fp16_htd_tp2to4": SMALL_E5M2["e5m2_fp16_htd_tp2to4"],
}


@pytest.mark.parametrize("name", list(PACK_UNPACK))
def test_graph_replays_pack_then_unpack(name):
    """Both steps of the unfused path recorded into one graph."""
    w = PACK_UNPACK[name]
    lens, bt, stride, shards, dshards, bt_d, sbt, sbt_d = _setup(w)
    plan = K.kvx_plan(desc_for(w, lens))
    info = K.kvx_plan_info_get(plan)
    wire = torch.full((max(int(info.wire_bytes), 16),), W.SENTINEL, dtype=torch.uint8,
                      device=DEV)
    cache, scales = pool(w, w.layers)

    def both():
        if w.src_order == "paged":
            K.kvx_pack_paged(plan, dshards, sbt_d, sbt.shape[1], wire)
        else:
            K.kvx_pack(plan, dshards, wire)
        K.kvx_unpack(plan, wire, cache, scales, bt_d, stride)

    log(f"graph pack+unpack {name}: record")
    g = _record(both)
    rng = np.random.default_rng(2000 + len(name))
    for k in range(1, REPLAYS + 1):
        new_bt, new_shards = _variant(w, lens, bt, shards, k, rng)
        _write(dshards, bt_d, new_bt, new_shards, (cache, scales, wire))
        log(f"graph pack+unpack {name}: replay {k}")
        g.replay()
        torch.cuda.synchronize()
        ref_c, ref_s = oracle_pool(w, lens, new_bt, stride, new_shards, sbt=sbt)
        _equal(name, k, cache, scales, ref_c, ref_s, "oracle")


NOALLOC = {
    "llama3_8b_small": SMALL["llama3_8b_small"],
    "fp8_small": SMALL["fp8_small"],
    "qwen_htd_small": SMALL["qwen_htd_small"],
}


@pytest.mark.parametrize("name", list(NOALLOC))
def test_graph_replays_noalloc(name):
    w = NOALLOC[name]
    lens, bt, stride, shards, dshards, bt_d, _, _ = _setup(w)
    desc = desc_for(w, lens)
    cache, scales = pool(w, w.layers)
    log(f"graph noalloc {name}: record")
    g = _record(lambda: K.kvx_repack_noalloc(desc, dshards, cache, scales, bt_d, stride))
    # another problem (a TP merge with other lengths and pages), run eagerly
    # between replays: it rewrites the static work-item table with its own items
    o = SMALL["llama3_70b_small_r0"]
    olens, obt, ostride, oshards = inputs(o)
    od = [dev_u16(s) for s in oshards]
    obt_d = torch.from_numpy(np.ascontiguousarray(obt, dtype=np.int32)).to(DEV)
    check_shapes(o, olens, obt, ostride, od, o.layers)
    oc, osc = pool(o, o.layers)
    odesc = desc_for(o, olens)
    rng = np.random.default_rng(3000 + len(name))
    for k in range(1, REPLAYS + 1):
        K.kvx_repack_noalloc(odesc, od, oc, osc, obt_d, ostride)
        new_bt, new_shards = _variant(w, lens, bt, shards, k, rng)
        _write(dshards, bt_d, new_bt, new_shards, (cache, scales))
        log(f"graph noalloc {name}: replay {k}")
        g.replay()
        torch.cuda.synchronize()
        ref_c, ref_s = oracle_pool(w, lens, new_bt, stride, new_shards)
        _equal(name, k, cache, scales, ref_c, ref_s, "oracle")
    ref_c, _ = oracle_pool(o, olens, obt, ostride, oshards)
    assert np.array_equal(oc.cpu().numpy(), ref_c), "the interleaved eager call"
