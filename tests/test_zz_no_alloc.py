"""The allocation-free repack (kvx_repack_noalloc) against the plan-based
kvx_repack, byte for byte, through the C ABI.

Each case runs two calls in a row on the same device, the second with a
smaller problem (fewer requests and tokens), so the second reads a static
work-item table that still holds the first call's longer contents.  Cases
cover token- and head-major sources, a TP merge (two head segments), an fp8
cache with scales, a quantise-dequantise cache, and the Qwen-7B workload at
full size (32 requests, 486 pages).  Also: the call at its table's limit, a
pipeline-stage descriptor, and the random descriptors with token- or
head-major sources against the oracle.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workload as W
from cases import FULL, RANDOM, SMALL, SMALL_DEQUANT, inputs, out_of_pool
from gpu_util import DEV, desc_for, dev_u16, log, oracle_pool, pool

import paper_2509_17542_amd as K

pytestmark = pytest.mark.gpu


def _both(w, lens, bt, stride, shards):
    """kvx_repack (plan) and kvx_repack_noalloc of the same problem into two
    sentinel-filled pools; returns the two (cache, scales) pairs."""
    dsh = [dev_u16(s) for s in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    ref_c, ref_s = pool(w, w.layers)
    K.kvx_repack(K.kvx_plan(desc_for(w, lens)), dsh, ref_c, ref_s, bt_d, stride)
    got_c, got_s = pool(w, w.layers)
    K.kvx_repack_noalloc(desc_for(w, lens), dsh, got_c, got_s, bt_d, stride)
    torch.cuda.synchronize()
    return (ref_c, ref_s), (got_c, got_s)


def _check(w, lens, bt, stride, shards):
    (rc, rs), (gc, gs) = _both(w, lens, bt, stride, shards)
    assert torch.equal(rc, gc), f"{w.name}: cache differs from kvx_repack"
    if rs is not None:
        assert torch.equal(rs.view(torch.uint8), gs.view(torch.uint8)), f"{w.name}: scales differ"


CASES = {
    "llama3_8b_small": SMALL["llama3_8b_small"],
    "qwen_htd_small": SMALL["qwen_htd_small"],
    "llama3_70b_small_r1": SMALL["llama3_70b_small_r1"],
    "fp8_small": SMALL["fp8_small"],
}
CASES.update({k: v for k, v in SMALL_DEQUANT.items() if v.src_order != "paged"})


def _smaller(w):
    if w.lens_override:
        lens = tuple(t // 2 for t in w.lens_override[:-1]) or (1,)
        return w.replace(lens_override=lens, num_requests=len(lens))
    return w.replace(num_requests=max(1, w.num_requests - 1), len_hi=max(w.len_lo, w.len_hi // 2))


@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_matches_repack_twice(name):
    w = CASES[name]
    log(f"noalloc {name}: first call")
    lens, bt, stride, shards = inputs(w)
    _check(w, lens, bt, stride, shards)
    # second call: fewer requests, shorter ones
    small = _smaller(w)
    lens2, bt2, stride2, shards2 = inputs(small)
    assert lens2.sum() < lens.sum()
    log(f"noalloc {name}: second, smaller call ({int(lens2.sum())} tokens)")
    _check(small, lens2, bt2, stride2, shards2)


def test_noalloc_full_qwen_then_small():
    w = FULL["qwen7b_htd_fp16_bf16_bs64"]
    lens, bt, stride, shards = inputs(w)
    log(f"noalloc full {w.name}: {int(lens.sum())} tokens")
    _check(w, lens, bt, stride, shards)
    small = SMALL["qwen_htd_small"]
    lens2, bt2, stride2, shards2 = inputs(small)
    log(f"noalloc then {small.name}: {int(lens2.sum())} tokens")
    _check(small, lens2, bt2, stride2, shards2)


def test_noalloc_at_its_table_limit():
    """256 requests and 65536 pages, the most the static table holds (one-token
    pages of one 16-byte row), against the plan-based repack and the oracle;
    then a smaller call."""
    w = SMALL["llama3_8b_small"].replace(name="noalloc_limit", heads=1, head_dim=8,
                                         block_size=1, num_blocks=65536, num_requests=256,
                                         lens_override=(256,) * 256)
    lens, bt, stride, shards = inputs(w)
    assert int(lens.sum()) == 65536
    log(f"noalloc at its limit: {len(lens)} requests, {int(lens.sum())} pages")
    (rc, _), (gc, _) = _both(w, lens, bt, stride, shards)
    assert torch.equal(rc, gc), "cache differs from kvx_repack"
    want, _ = oracle_pool(w, lens, bt, stride, shards)
    assert np.array_equal(gc.cpu().numpy(), want), "cache differs from the oracle"
    small = SMALL["llama3_8b_small"]
    _check(small, *inputs(small))


def test_noalloc_stage_plan():
    """A pipeline-stage descriptor: the source buffers hold prefill layers
    1-3, the cache decode layers 2-4 of a 5-layer model, and the two common
    layers are converted (layer offsets on both sides)."""
    w = SMALL["llama3_8b_small"].replace(layers=5, total_layers=5)
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    shards = W.source_shards(w, lens, 1, 3)
    desc = desc_for(w, lens, 2)
    desc.src_layer_offset, desc.src_layers = 1, 3
    desc.dst_layer_offset, desc.dst_layers = 0, 3
    dsh = [dev_u16(x) for x in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    ref_c, _ = pool(w, 3)
    K.kvx_repack(K.kvx_plan(desc), dsh, ref_c, None, bt_d, stride)
    got_c, _ = pool(w, 3)
    log("noalloc stage plan: prefill layers 1-3 -> decode layers 2-4")
    K.kvx_repack_noalloc(desc, dsh, got_c, None, bt_d, stride)
    torch.cuda.synchronize()
    assert torch.equal(ref_c, got_c)
    assert not torch.equal(got_c, pool(w, 3)[0]), "nothing was written"


@pytest.mark.parametrize("name", [n for n, w in RANDOM.items() if w.src_order != "paged"])
def test_noalloc_random_descriptor(name):
    """The random descriptors with token- or head-major sources (replicated
    heads, page sizes that are not powers of two, empty requests, about 10% of
    the block-table entries outside the pool) against the oracle."""
    w = RANDOM[name]
    lens, bt, stride, shards = inputs(w)
    bt = out_of_pool(bt, w.num_blocks, np.random.default_rng(int(name[4:])))
    log(f"noalloc {name}: TP {w.src_tp}->{w.dst_tp} {w.src_dtype}->{w.dst_dtype} "
        f"{w.src_order} bs={w.block_size} lens={list(lens)}")
    dsh = [dev_u16(x) for x in shards]
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    cache, scales = pool(w, w.layers)
    K.kvx_repack_noalloc(desc_for(w, lens), dsh, cache, scales, bt_d, stride)
    torch.cuda.synchronize()
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
    assert np.array_equal(cache.cpu().numpy(), want_c)
    if want_s is not None:
        assert np.array_equal(scales.view(torch.uint8).cpu().numpy(), want_s.view(np.uint8))


def test_noalloc_rejects_beyond_its_table():
    """Past 256 requests or 65536 pages the call refuses, before any launch."""
    w = SMALL["llama3_8b_small"]
    with pytest.raises(K.KvxError, match="256 requests"):
        K.kvx_repack_noalloc(desc_for(w, [1] * 257), [None], None, None, None, 1)
    with pytest.raises(K.KvxError, match="65536 pages"):
        K.kvx_repack_noalloc(desc_for(w.replace(block_size=1, num_blocks=1 << 20), [65537]),
                             [None], None, None, None, 65537)
