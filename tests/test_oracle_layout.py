"""Pins of the oracle's index maps (parallel-strategy and VRAM-management
alignment) to things other than its own formulas: the paper's TP4->TP2
example, a paged-attention reader built from torch indexing, memcpy special
cases, round-trip identities and write-set enumeration."""
import numpy as np
import pytest

from cases import (RANDOM, SMALL, SMALL_SHAPES, TINY, L8B, consumer_rows, dst_size, gather_pages,
                   inputs, oracle_problem, out_of_pool, wire_size, written_mask)
from conftest import golden_lines

import oracle as O
import workload as W


def _pool(p, sentinel=W.SENTINEL):
    cache = np.full(O.cache_bytes(p), sentinel, dtype=np.uint8)
    scales = None
    if p.cache_fmt_eff in O.FP8:
        scales = np.full(4 * O.scale_count(p), sentinel, dtype=np.uint8).view(np.float32)
    return cache, scales


# ---- Sec. III-B-3: the paper's worked example --------------------------------

def test_tp_alignment_paper_example():
    rows = golden_lines("tp_alignment.txt")
    assert len(rows) == 6
    for ln in rows:
        dims, ranks, heads = [s.strip() for s in ln.split("|")]
        H, ts, td, rho = map(int, dims.split())
        p = O.OracleProblem(1, H, 16, ts, td, rho, O.BF16, O.BF16, O.TOKEN_MAJOR, 16, 4, [1])
        got = [O.head_source(p, i) for i in range(H // td)]
        assert sorted({j for j, _ in got}) == [int(x) for x in ranks.split(",")], ln
        want = [tuple(int(v) for v in hs.split(":")) for hs in heads.split()]
        assert got == want, ln


@pytest.mark.parametrize("H,ts,td", [(8, 1, 8), (8, 8, 1), (8, 4, 2), (8, 2, 4), (6, 2, 3),
                                     (6, 3, 2), (12, 4, 6), (4, 4, 4), (32, 8, 2)])
def test_head_map_partitions_heads(H, ts, td):
    """Across the decode ranks every global head appears exactly once, each rank
    holds a contiguous ascending run, and (shard, head) pairs are valid."""
    seen = []
    for rho in range(td):
        p = O.OracleProblem(1, H, 16, ts, td, rho, O.BF16, O.BF16, O.TOKEN_MAJOR, 16, 4, [1])
        for i in range(H // td):
            j, h = O.head_source(p, i)
            assert 0 <= j < ts and 0 <= h < H // ts
            seen.append(j * (H // ts) + h)
    assert seen == list(range(H))


@pytest.mark.parametrize("H,ts,td", [(4, 1, 8), (4, 8, 2), (2, 4, 8), (8, 16, 16), (4, 4, 8),
                                     (4, 8, 1), (1, 2, 4)])
def test_head_map_with_replicated_heads(H, ts, td):
    """More ranks than KV heads: decode rank rho holds head rho // (td / H)
    (td / H consecutive ranks per head), and the source chosen for every head
    is a prefill shard that stores it (per the generator's prefill storage),
    at that head's position in the shard."""
    w = L8B.replace(heads=H, src_tp=ts, dst_tp=td)
    seen = []
    for rho in range(td):
        p = O.OracleProblem(1, H, 16, ts, td, rho, O.BF16, O.BF16, O.TOKEN_MAJOR, 16, 4, [1])
        assert O.validate(p) == 0
        hd = p.hd
        for i in range(hd):
            g = rho * hd + i if td <= H else rho // (td // H)
            j, h = O.head_source(p, i)
            g0, g1 = w.replace(dst_rank=rho).shard_heads(j)
            assert g0 <= g < g1 and h == g - g0, (rho, i, j, h)
            seen.append(g)
    assert sorted(set(seen)) == list(range(H))
    assert all(seen.count(g) == max(1, td // H) for g in range(H))


# ---- the decode side reads what the prefill side wrote ------------------------

@pytest.mark.parametrize("name", list(SMALL) + list(SMALL_SHAPES) + list(RANDOM))
def test_repack_matches_paged_reader(name):
    w = (SMALL | SMALL_SHAPES | RANDOM)[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    cache, scales = _pool(p)
    O.repack(p, shards, cache, scales, bt, stride)
    for r in range(len(lens)):
        want, want_s = consumer_rows(w, lens, r, 0, w.layers)
        got, got_s = gather_pages(cache, w, lens, bt, r, w.layers, scales)
        assert np.array_equal(got, want), (name, r)
        if want_s is not None:
            assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32)), (name, r)


@pytest.mark.parametrize("name", list(SMALL) + list(RANDOM))
def test_pack_matches_flat_logical_layout(name):
    """The transfer tensor of request r is [L][2][T][Hd][D] (+ [L][2][T][Hd]
    scales), 256-byte aligned segments, padding untouched."""
    w = (SMALL | RANDOM)[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    doff, soff, total = O.wire_layout(p)
    wire = O.pack(p, shards)
    touched = np.zeros(total, dtype=bool)
    end = 0
    wt = w.replace(cache_dtype="")   # the transfer tensor's rows (8-bit codes before dequantising)
    for r in range(len(lens)):
        T = int(lens[r])
        n = w.layers * 2 * T * w.hd * w.head_dim * wire_size(w)
        assert doff[r] % 256 == 0 and doff[r] >= end
        want, want_s = consumer_rows(wt, lens, r, 0, w.layers)
        got = wire[doff[r]:doff[r] + n].reshape(want.shape)
        assert np.array_equal(got, want), (name, r)
        touched[doff[r]:doff[r] + n] = True
        end = doff[r] + n
        if want_s is not None:
            m = w.layers * 2 * T * w.hd
            assert soff[r] % 256 == 0 and soff[r] >= end
            got_s = wire[soff[r]:soff[r] + 4 * m].view(np.float32).reshape(want_s.shape)
            assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32))
            touched[soff[r]:soff[r] + 4 * m] = True
            end = soff[r] + 4 * m
    assert total >= end and total % 256 == 0
    assert np.all(wire[~touched] == W.SENTINEL)


@pytest.mark.parametrize("name", list(SMALL) + list(RANDOM))
def test_write_set_is_exactly_the_used_slots(name):
    """Two runs with different pool fills: the bytes that differ were never
    written.  They must be exactly the slots outside every request's pages
    (unused pages, and slots past T in a last page)."""
    w = (SMALL | RANDOM)[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    runs = []
    for fill in (0xA5, 0x5A):
        cache, scales = _pool(p, fill)
        O.repack(p, shards, cache, scales, bt, stride)
        runs.append((cache, scales))
    m = written_mask(w, lens, bt, w.layers)
    row = w.hd * w.head_dim * dst_size(w)
    same = (runs[0][0] == runs[1][0]).reshape(w.layers, 2, w.num_blocks, w.block_size, row)
    assert np.array_equal(same.all(-1), m)
    assert not np.any(same.any(-1) & ~m)
    if runs[0][1] is not None:
        s0 = runs[0][1].view(np.uint32).reshape(w.layers, 2, w.num_blocks, w.block_size, w.hd)
        s1 = runs[1][1].view(np.uint32).reshape(s0.shape)
        assert np.array_equal((s0 == s1).all(-1), m)


@pytest.mark.parametrize("name", list(SMALL) + list(RANDOM))
def test_unpack_of_pack_equals_repack(name):
    w = (SMALL | RANDOM)[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    c1, s1 = _pool(p)
    O.repack(p, shards, c1, s1, bt, stride)
    c2, s2 = _pool(p)
    O.unpack(p, O.pack(p, shards), c2, s2, bt, stride)
    assert np.array_equal(c1, c2)
    if s1 is not None:
        assert np.array_equal(s1.view(np.uint32), s2.view(np.uint32))


@pytest.mark.parametrize("name", list(RANDOM))
def test_out_of_pool_pages_are_skipped(name):
    """Block-table entries outside the pool (decode pages, and for paged
    sources the prefill pages) are skipped, not errors: the repack with about
    10% of the entries moved out of range equals the repack with the valid
    tables, except that the slots of a skipped decode page, and the token
    slots whose source page was skipped, keep the pool's fill."""
    w = RANDOM[name]
    rng = np.random.default_rng(int(name[4:]))
    lens, bt, stride, shards = inputs(w)
    sbt = sbt2 = None
    if w.src_order == "paged":
        sbt, _ = W.src_block_table(w, lens)
        sbt2 = out_of_pool(sbt, w.src_num_blocks, rng)
    bt2 = out_of_pool(bt, w.num_blocks, rng)
    p = oracle_problem(O, w, lens, sbt=sbt)
    full, full_s = _pool(p)
    O.repack(p, shards, full, full_s, bt, stride)
    got, got_s = _pool(p)
    O.repack(oracle_problem(O, w, lens, sbt=sbt2), shards, got, got_s, bt2, stride)
    row = w.hd * w.head_dim * dst_size(w)
    want = full.reshape(w.layers, 2, w.num_blocks, w.block_size, row).copy()
    want_s = None if full_s is None else \
        full_s.view(np.uint32).reshape(w.layers, 2, w.num_blocks, w.block_size, w.hd).copy()
    fill = np.full(4, W.SENTINEL, np.uint8).view(np.uint32)[0]
    for r, T in enumerate(lens):
        for t in range(int(T)):
            k = t // w.block_size
            skipped = bt2[r, k] != bt[r, k]
            if sbt is not None:
                skipped |= sbt2[r, t // w.src_block_size] != sbt[r, t // w.src_block_size]
            if skipped:
                want[:, :, bt[r, k], t % w.block_size] = W.SENTINEL
                if want_s is not None:
                    want_s[:, :, bt[r, k], t % w.block_size] = fill
    assert np.array_equal(got.reshape(want.shape), want)
    if want_s is not None:
        assert np.array_equal(got_s.view(np.uint32).reshape(want_s.shape), want_s)


# ---- special cases and identities ----------------------------------------------

def _single(w, T, **kw):
    return w.replace(num_requests=1, lens_override=(T,), **kw)


@pytest.mark.parametrize("dtype,order", [("bf16", "thd"), ("fp16", "thd")])
def test_identity_layout_is_memcpy(dtype, order):
    """Same type, token-major, TP1->TP1, one request whose length is a multiple
    of the page size and whose pages are 0, 1, 2, ... in order: the paged pool
    is byte-for-byte the source buffer."""
    w = _single(L8B, 64, layers=2, total_layers=2, num_blocks=4, src_dtype=dtype,
                dst_dtype=dtype, src_order=order)
    lens, _, _, shards = inputs(w)
    bt = np.arange(4, dtype=np.int32)[None, :]
    p = oracle_problem(O, w, lens)
    cache, _ = _pool(p)
    O.repack(p, shards, cache, None, bt, 4)
    assert np.array_equal(cache.view(np.uint16), shards[0])


def _as_identity_pool_shards(w, T):
    """Identity paging: decode pools of one request read back as token-major
    source shards (same bytes, see test_identity_layout_is_memcpy)."""
    return np.arange(T // w.block_size, dtype=np.int32)[None, :]


@pytest.mark.parametrize("ts,td", [(4, 2), (2, 4), (8, 1), (1, 8), (2, 8)])
def test_tp_reshard_then_inverse_is_identity(ts, td):
    """Prefill TP=ts -> decode TP=td (all ranks), then the decode pools taken
    as a TP=td source -> TP=ts (all ranks): the original shards come back."""
    T = 48
    base = _single(L8B, T, layers=2, total_layers=2, num_blocks=T // 16, block_size=16,
                   src_tp=ts, dst_tp=td)
    lens = W.seq_lens(base)
    shards = W.source_shards(base, lens, shards=list(range(ts)))
    bt = _as_identity_pool_shards(base, T)
    mid = []
    for rho in range(td):
        w = base.replace(dst_rank=rho)
        p = oracle_problem(O, w, lens)
        cache, _ = _pool(p)
        O.repack(p, shards, cache, None, bt, bt.shape[1])
        mid.append(cache.view(np.uint16))
    back = base.replace(src_tp=td, dst_tp=ts)
    for rho in range(ts):
        p = oracle_problem(O, back.replace(dst_rank=rho), lens)
        cache, _ = _pool(p)
        O.repack(p, mid, cache, None, bt, bt.shape[1])
        assert np.array_equal(cache.view(np.uint16), shards[rho]), rho


@pytest.mark.parametrize("name", ["llama3_8b_small", "qwen_htd_small", "fp8_small",
                                  "llama3_70b_small_r1"])
def test_batch_equals_requests_one_by_one(name):
    w = SMALL[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    c_batch, s_batch = _pool(p)
    O.repack(p, shards, c_batch, s_batch, bt, stride)
    c_one, s_one = _pool(p)
    off = 0
    for r in range(len(lens)):
        n = w.layers * 2 * int(lens[r]) * w.hs * w.head_dim
        part = [None if s is None else np.ascontiguousarray(s[off:off + n]) for s in shards]
        off += n
        p1 = oracle_problem(O, w, lens[r:r + 1])
        O.repack(p1, part, c_one, s_one, bt[r:r + 1], stride)
    assert np.array_equal(c_batch, c_one)
    if s_batch is not None:
        assert np.array_equal(s_batch.view(np.uint32), s_one.view(np.uint32))


def test_expected_rows_match_full_repack():
    """The sampled-output entry point agrees with the whole-pool result."""
    w = SMALL["fp8_small"]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    cache, scales = _pool(p)
    O.repack(p, shards, cache, scales, bt, stride)
    for r in range(len(lens)):
        got, got_s = gather_pages(cache, w, lens, bt, r, w.layers, scales)
        for l in range(w.layers):
            for kv in range(2):
                rows, sc = O.expected_rows(p, shards, r, l, kv, 3, int(lens[r]) - 3)
                assert np.array_equal(rows.reshape(-1), got[l, kv, 3:].reshape(-1))
                assert np.array_equal(sc.view(np.uint32), got_s[l, kv, 3:].reshape(-1).view(np.uint32))


# ---- rejected problems ------------------------------------------------------------

@pytest.mark.parametrize("kw,code", [
    (dict(heads=6, src_tp=4), -1), (dict(dst_tp=3), -1), (dict(dst_rank=2), -1),
    (dict(dst_rank=-1), -1), (dict(layers=0), -1), (dict(block_size=0), -1),
    (dict(src_fmt=O.E4M3FN, dst_fmt=O.E4M3FN), -2), (dict(src_fmt=O.BF16, dst_fmt=99), -2),
    (dict(heads=4, dst_tp=6), -1), (dict(heads=4, src_tp=6), -1), (dict(heads=6, dst_tp=4), -1),
])
def test_validate_rejects(kw, code):
    base = dict(layers=2, heads=8, head_dim=64, src_tp=1, dst_tp=2, dst_rank=0, src_fmt=O.FP16,
                dst_fmt=O.BF16, src_order=O.TOKEN_MAJOR, block_size=16, num_blocks=8,
                seq_lens=[10])
    base.update(kw)
    assert O.validate(O.OracleProblem(**base)) == code


def test_bf16_to_fp16_case_overflows_and_keeps_the_rest():
    """The bf16 -> fp16 overflow case holds infinities where |x| rounds above
    65504 and finite values elsewhere (the casts are pinned exhaustively in
    test_oracle_casts; this checks the case exercises both)."""
    w = SMALL["bf16_fp16_overflow"]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    cache, _ = _pool(p)
    O.repack(p, shards, cache, None, bt, stride)
    got = np.concatenate([gather_pages(cache, w, lens, bt, r, w.layers)[0].reshape(-1)
                          for r in range(len(lens))]).view(np.uint16)
    inf = (got & 0x7FFF) == 0x7C00
    assert 0.05 < inf.mean() < 0.5


def test_validate_rejects_negative_length():
    p = O.OracleProblem(1, 4, 64, 1, 1, 0, O.BF16, O.BF16, O.TOKEN_MAJOR, 16, 8, [3, -1])
    assert O.validate(p) == -1


def test_wire_layout_hand_worked():
    """Segment offsets of the transfer tensor against hand-worked values
    (tests/golden/wire_layout.txt)."""
    f = {"bf16": O.BF16, "fp16": O.FP16, "e4m3fn": O.E4M3FN, "e5m2": O.E5M2}
    rows = golden_lines("wire_layout.txt")
    assert len(rows) == 3
    for ln in rows:
        head, toks, doffs, soffs, total = (part.split() for part in ln.split("|"))
        fmt = f[head[0]]
        L, H, ts, td, rank, D = map(int, head[1:])
        lens = [int(t) for t in toks]
        p = O.OracleProblem(L, H, D, ts, td, rank, O.BF16, fmt, O.TOKEN_MAJOR, 16, 64, lens)
        d, s, n = O.wire_layout(p)
        assert list(d) == [int(x) for x in doffs], ln
        assert list(s) == [int(x) for x in soffs], ln
        assert n == int(total[0]), ln
