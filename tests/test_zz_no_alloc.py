"""The allocation-free repack (kvx_repack_noalloc) against the plan-based
kvx_repack, byte for byte, through the C ABI.

Each case runs two calls in a row on the same device, the second with a
smaller problem (fewer requests and tokens), so the second reads a static
work-item table that still holds the first call's longer contents.  Cases
cover token- and head-major sources, a TP merge (two head segments), an fp8
cache with scales, a quantise-dequantise cache, and the Qwen-7B workload at
full size (32 requests, 486 pages).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workload as W
from cases import FULL, SMALL, SMALL_DEQUANT, inputs
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


def test_noalloc_rejects_beyond_its_table():
    """Past 256 requests or 65536 pages the call refuses, before any launch."""
    w = SMALL["llama3_8b_small"]
    with pytest.raises(K.KvxError, match="256 requests"):
        K.kvx_repack_noalloc(desc_for(w, [1] * 257), [None], None, None, None, 1)
    with pytest.raises(K.KvxError, match="65536 pages"):
        K.kvx_repack_noalloc(desc_for(w.replace(block_size=1, num_blocks=1 << 20), [65537]),
                             [None], None, None, None, 65537)
