"""Pins of the oracle's layer ranges (pipeline-parallel stages on either side:
the prefill side's pipeline stages each hold a range of layers, Sec. III-B-3
and the strategy search of Sec. III-C; here the decode side may be staged
differently).  A plan converts layers that lie in one source stage and one
decode stage; the pins reduce a set of stage plans to the whole-model
conversion, which the layout pins already fix."""
import numpy as np
import pytest

from cases import (L8B, L70B, SMALL, SMALL_PAGED, consumer_rows, dst_size, gather_pages,
                   oracle_problem)

import oracle as O
import workload as W


def _pool(p, sentinel=W.SENTINEL):
    cache = np.full(O.cache_bytes(p), sentinel, dtype=np.uint8)
    scales = None
    if p.cache_fmt_eff in O.FP8:
        scales = np.full(4 * O.scale_count(p), sentinel, dtype=np.uint8).view(np.float32)
    return cache, scales


def _stages(total, sizes):
    out, l0 = [], 0
    for n in sizes:
        out.append((l0, n))
        l0 += n
    assert l0 == total
    return out


def _stage_problem(w, lens, conv0, nconv, src_stage, dst_stage):
    p = oracle_problem(O, w, lens, nconv)
    p.c.src_layer_offset = conv0 - src_stage[0]
    p.c.src_layers = src_stage[1]
    p.c.dst_layer_offset = conv0 - dst_stage[0]
    p.c.dst_layers = dst_stage[1]
    return p


CASES = [("llama3_8b_small", 6, (3, 3), (2, 2, 2)), ("fp8_small", 5, (1, 4), (2, 3)),
         ("llama3_70b_small_r1", 4, (4,), (1, 1, 2)), ("qwen_htd_small", 5, (2, 1, 2), (5,)),
         ("paged16_tp4to2_bs32_small", 4, (2, 2), (3, 1)), ("paged16_e4m3_bs24", 3, (1, 2), (3,))]


@pytest.mark.parametrize("name,L,src_sizes,dst_sizes", CASES)
def test_stage_plans_compose_to_the_whole_model(name, L, src_sizes, dst_sizes):
    """Prefill stages (src_sizes layers each, one source buffer per stage as
    the prefill side holds them) -> decode stages (dst_sizes, one cache per
    stage): one plan per overlapping (source stage, decode stage) pair.  The
    decode stages' caches, laid end to end, equal the whole-model cache."""
    w = (SMALL | SMALL_PAGED)[name].replace(layers=L, total_layers=L)
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    whole_p = oracle_problem(O, w, lens, L)
    whole_c, whole_s = _pool(whole_p)
    O.repack(whole_p, W.source_shards(w, lens, 0, L), whole_c, whole_s, bt, stride)

    src_st = _stages(L, src_sizes)
    dst_st = _stages(L, dst_sizes)
    src_bufs = [W.source_shards(w, lens, l0, n) for l0, n in src_st]
    got_c, got_s = [], []
    plans = 0
    for d0, dn in dst_st:
        cache, scales = None, None
        for (s0, sn), shards in zip(src_st, src_bufs):
            lo, hi = max(s0, d0), min(s0 + sn, d0 + dn)
            if lo >= hi:
                continue
            p = _stage_problem(w, lens, lo, hi - lo, (s0, sn), (d0, dn))
            assert O.validate(p) == 0
            if cache is None:
                cache, scales = _pool(p)
            O.repack(p, shards, cache, scales, bt, stride)
            plans += 1
        got_c.append(cache)
        got_s.append(scales)
    assert plans >= max(len(src_sizes), len(dst_sizes))
    assert np.array_equal(np.concatenate(got_c), whole_c)
    if whole_s is not None:
        assert np.array_equal(np.concatenate(got_s).view(np.uint32), whole_s.view(np.uint32))


def test_stage_cache_matches_paged_reader():
    """Decode stage holding layers [2, 5) of a 6-layer model, fed from the
    prefill stage holding [1, 6): the stage's pages hold exactly the logical KV
    of layers 2..4 (independent of the whole-model path)."""
    w = L8B.replace(layers=6, total_layers=6, num_requests=2, len_lo=20, len_hi=60, num_blocks=16)
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    shards = W.source_shards(w, lens, 1, 5)
    p = _stage_problem(w, lens, 2, 3, (1, 5), (2, 3))
    cache, _ = _pool(p)
    O.repack(p, shards, cache, None, bt, stride)
    for r in range(len(lens)):
        want, _ = consumer_rows(w, lens, r, 2, 3)
        got, _ = gather_pages(cache, w, lens, bt, r, 3)
        assert np.array_equal(got, want), r


def test_stage_wire_is_a_slice_of_the_whole_wire():
    """The transfer tensor of a stage plan holds, per request, the planes of
    its layers: a contiguous slice of the whole-model request segment."""
    w = SMALL["fp8_small"].replace(layers=4, total_layers=4)
    lens = W.seq_lens(w)
    whole = oracle_problem(O, w, lens, 4)
    doff, soff, _ = O.wire_layout(whole)
    wire = O.pack(whole, W.source_shards(w, lens, 0, 4))
    p = _stage_problem(w, lens, 1, 2, (0, 4), (1, 3))
    sdoff, ssoff, _ = O.wire_layout(p)
    swire = O.pack(p, W.source_shards(w, lens, 0, 4))
    for r, T in enumerate(lens.tolist()):
        plane = T * w.hd * w.head_dim * dst_size(w)
        a = doff[r] + 2 * plane
        assert np.array_equal(swire[sdoff[r]:sdoff[r] + 4 * plane], wire[a:a + 4 * plane])
        splane = T * w.hd * 4
        a = soff[r] + 2 * splane
        assert np.array_equal(swire[ssoff[r]:ssoff[r] + 4 * splane], wire[a:a + 4 * splane])


@pytest.mark.parametrize("kw", [dict(src_layer_offset=3), dict(dst_layer_offset=2, dst_layers=3),
                                dict(src_layers=1), dict(src_layer_offset=-1, src_layers=4),
                                dict(dst_layers=-2)])
def test_validate_rejects_layer_ranges(kw):
    w = L70B
    p = O.OracleProblem(2, w.heads, w.head_dim, w.src_tp, w.dst_tp, 0, O.BF16, O.BF16,
                        O.TOKEN_MAJOR, 32, 16, [40], **{**dict(src_layers=4), **kw})
    assert O.validate(p) == -1


def test_validate_accepts_a_layer_range():
    p = O.OracleProblem(2, 8, 128, 4, 2, 0, O.BF16, O.BF16, O.TOKEN_MAJOR, 32, 16, [40],
                        src_layer_offset=2, src_layers=4, dst_layer_offset=5, dst_layers=7)
    assert O.validate(p) == 0
