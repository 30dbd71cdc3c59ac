"""Host side of the C ABI (runs without a GPU): the library loads and exports
every entry point declared in include/kvx.h; plans validate their problem,
report the algorithmic byte counts and transfer-tensor segments; argument
errors come back as status codes."""
import ctypes
import os
import re

import numpy as np
import pytest

from cases import (FP8_NAMES, FULL, RANDOM, SMALL, SMALL_DEQUANT, SMALL_E5M2, SMALL_PAGED,
                   oracle_problem, rank_heads, read_shards)
from conftest import ROOT

import oracle as O
import workload as W

K = pytest.importorskip("paper_2509_17542_amd")


def declared_entry_points():
    with open(os.path.join(ROOT, "include", "kvx.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:kvx_status|const char \*|int32_t)\s*\*?\s*(kvx_\w+)\s*\(",
                                 text, re.M)))


def test_every_declared_symbol_is_exported():
    names = declared_entry_points()
    assert len(names) == 22, names
    for n in names:
        assert hasattr(K._lib, n), n
    assert sorted(K.EXPORTS) == names
    assert K.kvx_abi_version() == 9


def desc_for(w, lens, **over):
    f = {"fp16": K.FP16, "bf16": K.BF16, "e4m3fn": K.E4M3FN, "e5m2": K.E5M2}
    kw = dict(num_layers=w.layers, num_kv_heads=w.heads, head_dim=w.head_dim, src_tp=w.src_tp,
              dst_tp=w.dst_tp, dst_rank=w.dst_rank, src_dtype=f[w.src_dtype],
              dst_dtype=f[w.dst_dtype],
              src_order={"thd": K.THD, "htd": K.HTD, "paged": K.PAGED}[w.src_order],
              block_size=w.block_size, num_blocks=w.num_blocks, seq_lens=list(lens),
              src_block_size=w.src_block_size, src_num_blocks=w.src_num_blocks,
              cache_dtype=f[w.cache_dtype] if w.cache_dtype else 0)
    kw.update(over)
    return K.make_desc(**kw)


@pytest.mark.parametrize("name", list(SMALL) + list(SMALL_PAGED) + list(SMALL_DEQUANT) +
                         list(SMALL_E5M2) + list(FULL) + list(RANDOM))
def test_plan_bytes_and_segments(name):
    w = (SMALL | SMALL_PAGED | SMALL_DEQUANT | SMALL_E5M2 | FULL | RANDOM)[name]
    lens = W.seq_lens(w)
    plan = K.kvx_plan(desc_for(w, lens))
    info = K.kvx_plan_info_get(plan)
    rows = w.layers * 2 * int(lens.sum()) * w.hd

    def row_bytes(dt):  # a row of head_dim elements, plus its scale for e4m3fn
        return w.head_dim + 4 if dt in FP8_NAMES else 2 * w.head_dim

    rd, wr, cw = rows * 2 * w.head_dim, rows * row_bytes(w.dst_dtype), rows * row_bytes(w.cdt)
    assert (info.read_bytes_repack, info.write_bytes_repack) == (rd, cw)
    assert (info.read_bytes_pack, info.write_bytes_pack) == (rd, wr)
    assert (info.read_bytes_unpack, info.write_bytes_unpack) == (wr, cw)
    nb = [(int(t) + w.block_size - 1) // w.block_size for t in lens]
    assert info.max_blocks_per_request == max(nb + [0])
    assert info.num_items == sum(nb)
    assert info.total_tokens == int(lens.sum())
    if w.src_order == "paged":
        snb = [(int(t) + w.src_block_size - 1) // w.src_block_size for t in lens]
        assert info.max_src_blocks_per_request == max(snb + [0])
    else:
        assert info.max_src_blocks_per_request == 0
    # transfer-tensor segments agree with the oracle's layout
    doff, soff, total = O.wire_layout(oracle_problem(O, w, lens))
    assert info.wire_bytes == total
    for r in range(len(lens)):
        assert K.kvx_plan_segment(plan, r) == (int(doff[r]), int(soff[r]))
    # buffer sizes: the pool the tests allocate, the generator's source shards
    sz = K.kvx_plan_buffer_sizes(plan)
    slots = w.layers * 2 * w.num_blocks * w.block_size * w.hd
    assert sz.wire_bytes == total
    assert sz.cache_bytes == slots * w.head_dim * (1 if w.cdt in FP8_NAMES else 2)
    assert sz.scale_bytes == (4 * slots if w.cdt in FP8_NAMES else 0)
    assert (sz.num_requests, sz.src_tp) == (len(lens), w.src_tp)
    if w.src_order == "paged":
        elems = w.layers * 2 * w.src_num_blocks * w.src_block_size * w.hs * w.head_dim
    else:
        elems = sum(w.layers * 2 * int(t) * w.hs * w.head_dim for t in lens)
    # the shard read for each head of the rank: the one holding it, or with
    # replicated prefill heads its first replica (reading R2)
    lo, hi = rank_heads(w)
    read = {g // w.hs if w.src_tp <= w.heads else g * (w.src_tp // w.heads) for g in range(lo, hi)}
    read = read if info.num_items else set()
    assert read <= set(read_shards(w))
    for j in range(w.src_tp):
        assert K.kvx_plan_shard_bytes(plan, j) == (2 * elems if j in read else 0), j
    assert plan.shard_bytes == [K.kvx_plan_shard_bytes(plan, j) for j in range(w.src_tp)]


BASE = dict(num_layers=2, num_kv_heads=8, head_dim=64, src_tp=1, dst_tp=2, dst_rank=0,
            src_dtype=1, dst_dtype=2, src_order=0, block_size=16, num_blocks=64, seq_lens=[40, 7])


@pytest.mark.parametrize("over,status", [
    (dict(num_layers=0), K.EINVAL), (dict(num_kv_heads=0), K.EINVAL), (dict(head_dim=-64), K.EINVAL),
    (dict(src_tp=3), K.EINVAL), (dict(dst_tp=3), K.EINVAL), (dict(dst_rank=2), K.EINVAL),
    (dict(src_tp=16, dst_tp=16, dst_rank=16), K.EINVAL),
    (dict(dst_rank=-1), K.EINVAL), (dict(block_size=0), K.EINVAL), (dict(num_blocks=0), K.EINVAL),
    (dict(seq_lens=[4, -1]), K.EINVAL), (dict(src_order=3), K.EINVAL),
    (dict(src_order=2), K.EINVAL),                      # paged without a page size
    (dict(src_order=2, src_block_size=16), K.EINVAL),   # paged without a pool
    (dict(src_order=2, src_block_size=0, src_num_blocks=8), K.EINVAL),
    (dict(head_dim=4), K.EINVAL),                       # 8-byte rows
    (dict(head_dim=8, dst_dtype=3), K.EINVAL),          # 8-byte e4m3 rows
    (dict(src_dtype=3), K.EUNSUPPORTED), (dict(src_dtype=3, dst_dtype=1), K.EUNSUPPORTED),
    (dict(num_kv_heads=4, dst_tp=6), K.EINVAL), (dict(num_kv_heads=4, src_tp=6), K.EINVAL),
    (dict(dst_dtype=9), K.EINVAL), (dict(head_dim=1024), K.EUNSUPPORTED),
    (dict(num_kv_heads=4096, dst_tp=2), K.EUNSUPPORTED), (dict(num_layers=40000), K.EUNSUPPORTED),
    (dict(cache_dtype=1), K.EUNSUPPORTED),               # a 16-bit transfer tensor is not dequantised
    (dict(dst_dtype=3, cache_dtype=9), K.EINVAL),
    (dict(dst_dtype=3, cache_dtype=2, head_dim=2048), K.EUNSUPPORTED),  # 2048-byte e4m3fn rows
    (dict(dst_dtype=4, cache_dtype=3), K.EUNSUPPORTED),  # e5m2 on the wire, e4m3fn in the cache
    (dict(dst_dtype=3, cache_dtype=4), K.EUNSUPPORTED),
    (dict(src_dtype=4, dst_dtype=4), K.EUNSUPPORTED),    # an 8-bit source
    (dict(dst_dtype=5), K.EINVAL),
    # 128 one-head prefill shards merged into one decode rank: 128 head
    # segments, above the 64 a launch carries (64 are accepted)
    (dict(num_kv_heads=128, head_dim=16, src_tp=128, dst_tp=1), K.EUNSUPPORTED),
])
def test_plan_rejects(over, status):
    kw = dict(BASE)
    kw.update(over)
    with pytest.raises(K.KvxError) as e:
        K.kvx_plan(K.make_desc(**kw))
    assert e.value.status == status
    assert K.kvx_last_error()


# The largest launch a plan accepts is 2^24 - 8 work units (units of one
# (layer, k/v) plane, one page, one head segment and one workgroup pass).  With
# one 16-byte row per one-token page, each page gives one unit per plane.
UNIT_LIMIT_PAGES = (1 << 23) - 4


def test_plan_work_unit_limit():
    """Exactly 2^24 - 8 units plan; one page more is refused before anything
    is allocated on a device."""
    kw = dict(BASE, num_layers=1, num_kv_heads=1, head_dim=8, dst_tp=1, src_dtype=K.BF16,
              dst_dtype=K.BF16, block_size=1, num_blocks=UNIT_LIMIT_PAGES + 1)
    plan = K.kvx_plan(K.make_desc(**dict(kw, seq_lens=[UNIT_LIMIT_PAGES])))
    assert K.kvx_plan_info_get(plan).num_items == UNIT_LIMIT_PAGES
    del plan
    with pytest.raises(K.KvxError) as e:
        K.kvx_plan(K.make_desc(**dict(kw, seq_lens=[UNIT_LIMIT_PAGES + 1])))
    assert e.value.status == K.EUNSUPPORTED and "work units" in str(e.value)


def test_plan_accepts_64_head_segments():
    plan = K.kvx_plan(K.make_desc(**dict(BASE, num_kv_heads=64, head_dim=16, src_tp=64,
                                         dst_tp=1)))
    assert K.kvx_plan_segment(plan, 0)[0] == 0


def test_plan_accepts_empty_batches():
    """No tokens: nothing to move, the launch calls succeed without looking at
    any pointer (and launch nothing, so this is safe on any host)."""
    for lens in ([], [0, 0]):
        kw = dict(BASE, seq_lens=lens)
        plan = K.kvx_plan(K.make_desc(**kw))
        info = K.kvx_plan_info_get(plan)
        assert info.num_items == 0 and info.read_bytes_repack == 0
        K.kvx_repack(plan, [None], None, None, None, 0)
        K.kvx_pack(plan, [None], None)
        K.kvx_unpack(plan, None, None, None, None, 0)
        paged = K.kvx_plan(K.make_desc(**dict(kw, src_order=K.PAGED, src_block_size=16,
                                              src_num_blocks=4)))
        K.kvx_repack_paged(paged, [None], None, 0, None, None, None, 0)
        K.kvx_pack_paged(paged, [None], None, 0, None)
        K.kvx_unpack(paged, None, None, None, None, 0)


def test_plan_copies_seq_lens():
    """The plan keeps its own copy of the lengths: overwriting the caller's
    array afterwards changes neither its sizes nor its transfer-tensor
    segments."""
    d = K.make_desc(**BASE)
    plan = K.kvx_plan(d)
    before = K.kvx_plan_info_get(plan)
    segs = [K.kvx_plan_segment(plan, r) for r in range(2)]
    d._lens[0], d._lens[1] = 4000, 1
    after = K.kvx_plan_info_get(plan)
    assert (after.total_tokens, after.wire_bytes, after.num_items) == \
        (before.total_tokens, before.wire_bytes, before.num_items) == (47, before.wire_bytes, 4)
    assert [K.kvx_plan_segment(plan, r) for r in range(2)] == segs


def test_plans_and_errors_from_several_threads():
    """Plans built and refused from 8 host threads at once: each thread gets
    its own plan sizes and its own last-error message (kept per thread)."""
    import threading
    results, errors = {}, []
    start = threading.Barrier(8)

    def work(k):
        try:
            start.wait()
            for _ in range(50):
                plan = K.kvx_plan(K.make_desc(**dict(BASE, seq_lens=[40 + k, 7])))
                assert K.kvx_plan_info_get(plan).total_tokens == 47 + k
                st = K._lib.kvx_plan(ctypes.byref(K.make_desc(**dict(BASE, dst_rank=2 + k))),
                                     ctypes.byref(K._vp()))
                assert st == K.EINVAL and f"dst_rank {2 + k} outside" in K.kvx_last_error()
            results[k] = True
        except Exception as e:  # reported by the main thread
            errors.append((k, repr(e)))

    threads = [threading.Thread(target=work, args=(k,)) for k in range(8)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    assert len(results) == 8


def test_segment_out_of_range():
    plan = K.kvx_plan(K.make_desc(**BASE))
    with pytest.raises(K.KvxError) as e:
        K.kvx_plan_segment(plan, 2)
    assert e.value.status == K.EINVAL


def test_launch_argument_errors_before_device():
    """Pointer and shape errors are reported on the host, before any device
    work (on a host without a GPU the plan is host-only: EDEVICE last)."""
    plan = K.kvx_plan(K.make_desc(**BASE))        # fp16 -> bf16, TP1 -> TP2
    good = 0x10000
    cases = [
        (lambda: K.kvx_repack(plan, [None], good, None, good, 3), K.EINVAL),   # NULL shard
        (lambda: K.kvx_repack(plan, [good + 8], good, None, good, 3), K.EINVAL),  # misaligned
        (lambda: K.kvx_repack(plan, [good], good + 4, None, good, 3), K.EINVAL),
        (lambda: K.kvx_repack(plan, [good], good, good, good, 3), K.EINVAL),    # scales w/o fp8
        (lambda: K.kvx_repack(plan, [good], good, None, None, 3), K.EINVAL),    # NULL table
        (lambda: K.kvx_repack(plan, [good], good, None, good, 2), K.EINVAL),    # short stride
        (lambda: K.kvx_unpack(plan, None, good, None, good, 3), K.EINVAL),
        (lambda: K.kvx_pack(plan, [good], None), K.EINVAL),
    ]
    for call, status in cases:
        with pytest.raises(K.KvxError) as e:
            call()
        assert e.value.status == status, K.kvx_last_error()
    fp8 = K.kvx_plan(K.make_desc(**dict(BASE, dst_dtype=3)))
    with pytest.raises(K.KvxError) as e:
        K.kvx_repack(fp8, [good], good, None, good, 3)                      # fp8 needs scales
    assert e.value.status == K.EINVAL
    # a dequantising plan's cache holds no scales, whatever the transfer tensor carries
    dq = K.kvx_plan(K.make_desc(**dict(BASE, dst_dtype=3, cache_dtype=2)))
    for call in (lambda: K.kvx_repack(dq, [good], good, good, good, 3),
                 lambda: K.kvx_unpack(dq, good, good, good, good, 3)):
        with pytest.raises(K.KvxError) as e:
            call()
        assert e.value.status == K.EINVAL and "scales" in K.kvx_last_error()
    # the same cache dtype named explicitly is the plain plan
    same = K.kvx_plan(K.make_desc(**dict(BASE, dst_dtype=3, cache_dtype=3)))
    assert K.kvx_plan_info_get(same).write_bytes_unpack == K.kvx_plan_info_get(fp8).write_bytes_unpack


def test_merge_needs_every_overlapping_shard():
    """Decode rank 1 of TP2 over prefill TP4 reads shards 2 and 3 only; a
    missing or misaligned one of those is rejected, the others may be NULL.
    (No call here passes validation, so nothing is ever launched.)"""
    plan = K.kvx_plan(K.make_desc(**dict(BASE, src_tp=4, dst_tp=2, dst_rank=1)))
    g = 0x10000
    for shards in ([None, None, g, None], [None, None, None, g], [g, g, g + 2, g]):
        with pytest.raises(K.KvxError) as e:
            K.kvx_repack(plan, shards, g, None, g, 0)
        assert e.value.status == K.EINVAL
        assert "src_shards[" in K.kvx_last_error()


def test_check_block_table():
    plan = K.kvx_plan(K.make_desc(**BASE))        # 40 and 7 tokens: 3 + 1 pages
    ok = np.array([[5, 9, 63], [0, -1, -1]], dtype=np.int32)
    K.kvx_check_block_table(plan, ok, 3)
    for bad in ([[5, 9, 64], [0, -1, -1]], [[5, 9, 5], [0, -1, -1]], [[5, 9, 1], [-2, 0, 0]],
                [[5, 9, 1], [9, 0, 0]]):
        with pytest.raises(K.KvxError) as e:
            K.kvx_check_block_table(plan, np.array(bad, dtype=np.int32), 3)
        assert e.value.status == K.EINVAL
    with pytest.raises(K.KvxError):
        K.kvx_check_block_table(plan, ok, 2)


def test_workload_block_tables_are_valid():
    for w in list(SMALL.values()) + [FULL["llama3_8b_bf16_bs16"]]:
        lens = W.seq_lens(w)
        bt, stride = W.block_table(w, lens)
        K.kvx_check_block_table(K.kvx_plan(desc_for(w, lens)), bt, stride)


PAGED = dict(BASE, src_order=2, src_block_size=24, src_num_blocks=32)   # 40 and 7 tokens: 2 + 1 source pages


def test_paged_entry_points_match_the_plan():
    """A paged plan is served by the _paged calls only, a contiguous-source
    plan by the others; the source block table and its stride are checked."""
    g = 0x10000
    plain = K.kvx_plan(K.make_desc(**BASE))
    paged = K.kvx_plan(K.make_desc(**PAGED))
    assert K.kvx_plan_info_get(paged).max_src_blocks_per_request == 2
    cases = [
        (lambda: K.kvx_repack(paged, [g], g, None, g, 3), "kvx_repack_paged"),
        (lambda: K.kvx_pack(paged, [g], g), "kvx_pack_paged"),
        (lambda: K.kvx_repack_paged(plain, [g], g, 2, g, None, g, 3), "not paged"),
        (lambda: K.kvx_pack_paged(plain, [g], g, 2, g), "not paged"),
        (lambda: K.kvx_repack_paged(paged, [g], None, 2, g, None, g, 3), "NULL source block table"),
        (lambda: K.kvx_repack_paged(paged, [g], g, 1, g, None, g, 3), "src_bt_stride"),
        (lambda: K.kvx_pack_paged(paged, [g], g, 1, g), "src_bt_stride"),
        (lambda: K.kvx_repack_paged(paged, [None], g, 2, g, None, g, 3), "src_shards["),
        (lambda: K.kvx_repack_paged(paged, [g], g, 2, g, None, g, 2), "bt_stride"),
    ]
    for call, msg in cases:
        with pytest.raises(K.KvxError) as e:
            call()
        assert e.value.status == K.EINVAL and msg in K.kvx_last_error(), K.kvx_last_error()


def test_check_src_block_table():
    paged = K.kvx_plan(K.make_desc(**PAGED))
    ok = np.array([[5, 31], [5, -1]], dtype=np.int32)        # a shared page is allowed
    K.kvx_check_src_block_table(paged, ok, 2)
    for bad in ([[5, 32], [0, -1]], [[-1, 3], [0, 0]], [[1, 2], [40, 0]]):
        with pytest.raises(K.KvxError) as e:
            K.kvx_check_src_block_table(paged, np.array(bad, dtype=np.int32), 2)
        assert e.value.status == K.EINVAL
    with pytest.raises(K.KvxError):
        K.kvx_check_src_block_table(paged, ok, 1)
    with pytest.raises(K.KvxError):
        K.kvx_check_src_block_table(K.kvx_plan(K.make_desc(**BASE)), ok, 2)


def test_workload_source_block_tables_are_valid():
    for w in list(SMALL_PAGED.values()) + [FULL["llama3_8b_paged16_bf16_bs64"],
                                           FULL["llama3_70b_paged16_tp4to2_bf16_bs32"]]:
        lens = W.seq_lens(w)
        sbt, sstride = W.src_block_table(w, lens)
        bt, stride = W.block_table(w, lens)
        plan = K.kvx_plan(desc_for(w, lens))
        K.kvx_check_src_block_table(plan, sbt, sstride)
        K.kvx_check_block_table(plan, bt, stride)


@pytest.mark.parametrize("over", [dict(src_layer_offset=1), dict(src_layers=1),
                                  dict(dst_layer_offset=3, dst_layers=4),
                                  dict(src_layer_offset=-1, src_layers=4), dict(dst_layers=-1)])
def test_plan_rejects_layer_ranges(over):
    with pytest.raises(K.KvxError) as e:
        K.kvx_plan(K.make_desc(**dict(BASE, **over)))
    assert e.value.status == K.EINVAL and "layer" in K.kvx_last_error()


def test_plan_accepts_a_layer_range():
    """Layers 3..4 of a prefill stage holding 5 layers, into a decode stage
    holding 8 layers at 6..7: the byte counts and the transfer tensor cover
    the 2 converted layers only."""
    stage = K.kvx_plan(K.make_desc(**dict(BASE, src_layer_offset=3, src_layers=5,
                                          dst_layer_offset=6, dst_layers=8)))
    whole = K.kvx_plan(K.make_desc(**BASE))
    a, b = K.kvx_plan_info_get(stage), K.kvx_plan_info_get(whole)
    assert (a.read_bytes_repack, a.write_bytes_repack, a.wire_bytes) == \
        (b.read_bytes_repack, b.write_bytes_repack, b.wire_bytes)


def test_pipe_create_errors_on_the_host():
    """A host-only plan (no device here) cannot get a pipe; bad chunk sizes
    and slot counts are rejected first."""
    plan = K.kvx_plan(K.make_desc(**BASE))
    for chunk, slots, status in ((0, 2, K.EINVAL), (3, 2, K.EINVAL), (1, 0, K.EINVAL)):
        with pytest.raises(K.KvxError) as e:
            K.kvx_pipe_create(plan, chunk, slots)
        assert e.value.status == status, K.kvx_last_error()
    if K.kvx_plan_info_get(plan).device < 0:
        with pytest.raises(K.KvxError) as e:
            K.kvx_pipe_create(plan, 1, 2)
        assert e.value.status == K.EDEVICE


def test_pipe_of_a_plan_without_tokens():
    """No tokens: the pipe allocates nothing and its run returns at once, on
    any host (a device is not needed), like the plan's own launches."""
    for lens in ([], [0, 0]):
        plan = K.kvx_plan(K.make_desc(**dict(BASE, seq_lens=lens)))
        pipe = K.kvx_pipe_create(plan, 1, 3)
        info = K.kvx_pipe_info_get(pipe)
        assert (info.num_chunks, info.slots, info.host_bytes, info.bus_bytes) == (2, 3, 0, 0)
        assert K._lib.kvx_pipe_run(pipe, None, None, 0, None, None, None, 0, None) == K.OK
        K.kvx_pipe_destroy(pipe)


def test_buffer_size_queries_reject_bad_arguments():
    plan = K.kvx_plan(desc_for(SMALL["tiny"], W.seq_lens(SMALL["tiny"])))
    for j in (-1, SMALL["tiny"].src_tp):
        with pytest.raises(K.KvxError) as e:
            K.kvx_plan_shard_bytes(plan, j)
        assert e.value.status == K.EINVAL
    assert K._lib.kvx_plan_buffer_sizes(plan, None) == K.EINVAL
    assert K._lib.kvx_plan_buffer_sizes(None, ctypes.byref(K.kvx_buffer_sizes())) == K.EINVAL


@pytest.mark.parametrize("over", [dict(num_blocks=1 << 62), dict(num_blocks=1 << 46),
                                  dict(seq_lens=[(1 << 31) - 1] * 64, num_layers=32767)])
def test_plan_rejects_buffers_of_2_62_bytes(over):
    w = SMALL["llama3_8b_small"]
    d = desc_for(w, W.seq_lens(w), **over)
    with pytest.raises(K.KvxError) as e:
        K.kvx_plan(d)
    assert e.value.status == K.EUNSUPPORTED and "2^62" in str(e.value)


def test_binding_checks_tensor_arguments_before_any_launch():
    """Host tensors, short shard lists and wrong table types are refused by
    the binding before the C call (on a machine without a GPU the plan is
    host-only, and nothing reaches a device either way)."""
    import torch
    w = SMALL["llama3_8b_small"]
    lens = W.seq_lens(w)
    plan = K.kvx_plan(desc_for(w, lens))
    cpu = torch.empty(16, dtype=torch.uint8)
    with pytest.raises(ValueError, match="device tensor"):
        K.kvx_repack(plan, [cpu], None, None, None, 1)
    with pytest.raises(ValueError, match="source shards"):
        K.kvx_repack(plan, [], None, None, None, 1)
    with pytest.raises(ValueError, match="device tensor"):
        K.kvx_pack(plan, [None], cpu)
    with pytest.raises(ValueError, match="device tensor"):
        K.kvx_unpack(plan, None, cpu, None, None, 1)


def test_noalloc_repack_host_checks():
    """kvx_repack_noalloc validates its descriptor and arguments before any
    device work, with the status codes of kvx_plan and kvx_repack; its own
    limits are 256 requests and 65536 pages (its static work-item table).  An
    empty problem is a no-op; on a host without a device a valid call ends in
    KVX_EDEVICE (the static table's address cannot be found)."""
    w = SMALL["llama3_8b_small"]
    lens = W.seq_lens(w)
    lib = K._lib
    sh = (ctypes.c_void_p * 1)(0x10000)
    fake = ctypes.c_void_p(0x20000)

    def call(d, shards=sh, cache=fake, scales=None, bt=fake, stride=64):
        return lib.kvx_repack_noalloc(ctypes.byref(d) if d is not None else None, shards, cache,
                                      scales, bt, stride, None)

    assert call(None) == K.EINVAL
    assert call(desc_for(w, lens, head_dim=0)) == K.EINVAL
    assert call(desc_for(w, lens, src_order=K.PAGED, src_block_size=16, src_num_blocks=64)) == \
        K.EINVAL
    assert call(desc_for(w, [1] * 257)) == K.EUNSUPPORTED
    assert "256 requests" in K.kvx_last_error()
    # 65537 one-token pages: page size 1, 257 requests would trip the other limit
    assert call(desc_for(w, [65537], block_size=1, num_blocks=1 << 20)) == K.EUNSUPPORTED
    assert "65536 pages" in K.kvx_last_error()
    assert call(desc_for(w, [0, 0]), shards=None, cache=None, bt=None) == K.OK   # nothing to move
    assert call(desc_for(w, lens), shards=None) == K.EINVAL
    assert call(desc_for(w, lens), shards=(ctypes.c_void_p * 1)(0)) == K.EINVAL
    assert call(desc_for(w, lens), shards=(ctypes.c_void_p * 1)(0x10008)) == K.EINVAL
    assert call(desc_for(w, lens), cache=None) == K.EINVAL
    assert call(desc_for(w, lens), cache=ctypes.c_void_p(0x20004)) == K.EINVAL
    assert call(desc_for(w, lens), scales=fake) == K.EINVAL          # 16-bit cache
    assert call(desc_for(w, lens, dst_dtype=K.E4M3FN)) == K.EINVAL   # 8-bit cache, no scales
    assert call(desc_for(w, lens), bt=None) == K.EINVAL
    assert call(desc_for(w, lens), stride=1) == K.EINVAL
    if os.environ.get("HIP_VISIBLE_DEVICES", None) == "" or not _has_device():
        assert call(desc_for(w, lens)) == K.EDEVICE


def _has_device() -> bool:
    n = ctypes.c_int(0)
    try:
        rt = ctypes.CDLL("libamdhip64.so")
    except OSError:
        return False
    return rt.hipGetDeviceCount(ctypes.byref(n)) == 0 and n.value > 0
