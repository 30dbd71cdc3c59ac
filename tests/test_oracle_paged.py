"""Pins of the oracle's paged-source path (the prefill side's own paged cache,
with its own page size and block table, Sec. III-B-2: both sides of the
transfer use paged attention with their own block size) to things other than
its own index formula: a paged-attention reader built from torch indexing over
the generator's page placement, the reduction of a one-page pool to the
token-major source, a chain through an intermediate paged cache, and the
write set when source page ids fall outside the pool."""
import numpy as np
import pytest

from cases import (L8B, SMALL_PAGED, consumer_rows, dst_size, gather_pages, inputs,
                   oracle_problem, read_shards, written_mask)

import oracle as O
import workload as W


def _pool(p, sentinel=W.SENTINEL):
    cache = np.full(O.cache_bytes(p), sentinel, dtype=np.uint8)
    scales = None
    if p.cache_fmt_eff in O.FP8:
        scales = np.full(4 * O.scale_count(p), sentinel, dtype=np.uint8).view(np.float32)
    return cache, scales


@pytest.mark.parametrize("name", list(SMALL_PAGED))
def test_paged_source_generator_places_every_token_once(name):
    """The generator's paged pool holds each (request, token) in exactly the
    slot its source block table names; every other slot keeps the sentinel."""
    w = SMALL_PAGED[name]
    lens = W.seq_lens(w)
    sbt, _ = W.src_block_table(w, lens)
    shards = W.source_shards(w, lens)
    used = np.zeros((w.src_num_blocks, w.src_block_size), dtype=bool)
    for r, T in enumerate(lens.tolist()):
        for t in range(T):
            b = sbt[r, t // w.src_block_size]
            assert not used[b, t % w.src_block_size]
            used[b, t % w.src_block_size] = True
    for j in read_shards(w):
        pool = shards[j].reshape(w.layers, 2, w.src_num_blocks, w.src_block_size, -1)
        sentinel = (pool == W.SENTINEL * 0x0101).all(-1)
        assert np.array_equal(sentinel, np.broadcast_to(~used, sentinel.shape)), j


@pytest.mark.parametrize("name", list(SMALL_PAGED))
def test_paged_repack_matches_paged_reader(name):
    """Decode pages gathered per request equal the logical KV of the decode
    rank's heads, cast by torch (independent of the oracle's formulas)."""
    w = SMALL_PAGED[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    assert O.validate(p) == 0
    cache, scales = _pool(p)
    O.repack(p, shards, cache, scales, bt, stride)
    for r in range(len(lens)):
        want, want_s = consumer_rows(w, lens, r, 0, w.layers)
        got, got_s = gather_pages(cache, w, lens, bt, r, w.layers, scales)
        assert np.array_equal(got, want), (name, r)
        if want_s is not None:
            assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32)), (name, r)
    # and nothing else is written
    m = written_mask(w, lens, bt, w.layers)
    row = w.hd * w.head_dim * dst_size(w)
    untouched = (cache.reshape(w.layers, 2, w.num_blocks, w.block_size, row) == W.SENTINEL)
    assert np.array_equal(untouched.all(-1), ~m)


@pytest.mark.parametrize("name", list(SMALL_PAGED))
def test_paged_pack_then_unpack_equals_repack(name):
    w = SMALL_PAGED[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    c1, s1 = _pool(p)
    O.repack(p, shards, c1, s1, bt, stride)
    c2, s2 = _pool(p)
    O.unpack(p, O.pack(p, shards), c2, s2, bt, stride)
    assert np.array_equal(c1, c2)
    if s1 is not None:
        assert np.array_equal(s1.view(np.uint32), s2.view(np.uint32))


@pytest.mark.parametrize("dtypes", [("bf16", "bf16"), ("fp16", "bf16"), ("bf16", "e4m3fn")])
def test_one_page_pool_is_the_token_major_source(dtypes):
    """One request whose prefill pool is a single page of exactly T tokens: the
    pool [L][2][1][T][Hs][D] is byte-for-byte the token-major source
    [L][2][T][Hs][D], so both source orders give the same decode cache."""
    T = 45
    base = L8B.replace(num_requests=1, lens_override=(T,), layers=2, total_layers=2,
                       num_blocks=8, src_dtype=dtypes[0], dst_dtype=dtypes[1], src_tp=2,
                       dst_tp=1)
    paged = base.replace(src_order="paged", src_block_size=T, src_num_blocks=1)
    lens, bt, stride, thd = inputs(base)
    _, _, _, pg = inputs(paged)
    for j in range(2):
        assert np.array_equal(pg[j], thd[j])
    sbt = np.zeros((1, 1), dtype=np.int32)
    out = []
    for w, shards, extra in ((base, thd, {}), (paged, pg, {"sbt": sbt})):
        p = oracle_problem(O, w, lens, **extra)
        cache, scales = _pool(p)
        O.repack(p, shards, cache, scales, bt, stride)
        out.append((cache, scales))
    assert np.array_equal(out[0][0], out[1][0])
    if out[0][1] is not None:
        assert np.array_equal(out[0][1].view(np.uint32), out[1][1].view(np.uint32))


@pytest.mark.parametrize("td,rho,dst", [(1, 0, "bf16"), (2, 1, "bf16"), (4, 2, "e4m3fn")])
def test_chain_through_an_intermediate_paged_cache(td, rho, dst):
    """Token-major source -> decode cache A (TP1, 16-token pages, table A);
    A read back as a paged source -> cache B (TP td, 24-token pages, table
    B) equals the token-major source -> cache B in one step."""
    base = L8B.replace(layers=2, total_layers=2, num_requests=3, len_lo=5, len_hi=70,
                       num_blocks=24, block_size=16)
    lens, bt_a, stride_a, shards = inputs(base)
    pa = oracle_problem(O, base, lens)
    cache_a, _ = _pool(pa)
    O.repack(pa, shards, cache_a, None, bt_a, stride_a)
    wb = base.replace(dst_tp=td, dst_rank=rho, dst_dtype=dst, block_size=24, num_blocks=16,
                      seed=base.seed + 1)
    bt_b, stride_b = W.block_table(wb, lens)
    pb = oracle_problem(O, wb, lens)
    want_c, want_s = _pool(pb)
    O.repack(pb, shards, want_c, want_s, bt_b, stride_b)
    wp = wb.replace(src_order="paged", src_block_size=16, src_num_blocks=24)
    pp = oracle_problem(O, wp, lens, sbt=bt_a)
    got_c, got_s = _pool(pp)
    O.repack(pp, [cache_a.view(np.uint16)], got_c, got_s, bt_b, stride_b)
    assert np.array_equal(got_c, want_c)
    if want_s is not None:
        assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32))


def test_source_pages_outside_the_pool_are_skipped():
    """A source page id outside [0, src_num_blocks) gives no row: the decode
    slots of its tokens keep the sentinel; every other slot is as usual.  A
    decode page id outside the pool is skipped likewise."""
    w = SMALL_PAGED["paged24_bs16_r1"]
    lens, bt, stride, shards = inputs(w)
    sbt, _ = W.src_block_table(w, lens)
    p = oracle_problem(O, w, lens, sbt=sbt)
    want, _ = _pool(p)
    O.repack(p, shards, want, None, bt, stride)
    bad = sbt.copy()
    bad[0, 1] = -1
    bad[2, 0] = w.src_num_blocks
    pbad = oracle_problem(O, w, lens, sbt=bad)
    got, _ = _pool(pbad)
    bad_dst = bt.copy()
    bad_dst[1, 2] = w.num_blocks + 3
    O.repack(pbad, shards, got, None, bad_dst, stride)
    row = w.hd * w.head_dim * 2
    want = want.reshape(w.layers, 2, w.num_blocks, w.block_size, row)
    sbs, bs = w.src_block_size, w.block_size
    for r, k in ((0, 1), (2, 0)):
        for t in range(k * sbs, min((k + 1) * sbs, int(lens[r]))):
            want[:, :, bt[r, t // bs], t % bs] = W.SENTINEL
    want[:, :, bt[1, 2]] = W.SENTINEL
    assert np.array_equal(got, want.reshape(-1))


def test_paged_wire_rows_without_source_keep_the_sentinel():
    w = SMALL_PAGED["paged16_e4m3_bs24"]
    lens, _, _, shards = inputs(w)
    sbt, _ = W.src_block_table(w, lens)
    bad = sbt.copy()
    bad[0, 2] = -5
    p = oracle_problem(O, w, lens, sbt=bad)
    doff, soff, _ = O.wire_layout(p)
    wire = O.pack(p, shards)
    T = int(lens[0])
    rows = wire[doff[0]:doff[0] + w.layers * 2 * T * w.hd * w.head_dim]
    rows = rows.reshape(w.layers, 2, T, w.hd * w.head_dim)
    sc = wire[soff[0]:soff[0] + w.layers * 2 * T * w.hd * 4].reshape(w.layers, 2, T, w.hd * 4)
    dead = np.zeros(T, dtype=bool)
    dead[2 * w.src_block_size:3 * w.src_block_size] = True
    assert np.all(rows[:, :, dead] == W.SENTINEL) and np.all(sc[:, :, dead] == W.SENTINEL)
    assert not np.any((rows[:, :, ~dead] == W.SENTINEL).all(-1))


@pytest.mark.parametrize("kw", [dict(src_block_size=0), dict(src_num_blocks=0),
                                dict(src_bt_stride=1), dict(src_block_table=None)])
def test_validate_rejects_paged(kw):
    w = SMALL_PAGED["paged16_bs64_small"]
    lens = W.seq_lens(w)
    sbt, stride = W.src_block_table(w, lens)
    args = dict(src_block_size=w.src_block_size, src_num_blocks=w.src_num_blocks,
                src_block_table=sbt, src_bt_stride=stride)
    args.update(kw)
    p = O.OracleProblem(w.layers, w.heads, w.head_dim, 1, 1, 0, O.BF16, O.BF16, O.PAGED,
                        w.block_size, w.num_blocks, lens, **args)
    assert O.validate(p) == -1
