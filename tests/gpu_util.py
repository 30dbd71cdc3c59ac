"""Helpers of the GPU tests: C-ABI calls on device buffers and sampled checks
against the oracle.  Device memory comes from torch; every conversion step
runs in libkvx.so."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
import workload as W
from cases import FP8_NAMES, dst_size, oracle_problem, read_shards

import paper_2509_17542_amd as K

DEV = "cuda"
_F = {"fp16": K.FP16, "bf16": K.BF16, "e4m3fn": K.E4M3FN, "e5m2": K.E5M2}


def log(msg: str) -> None:
    print(msg, flush=True)


_ORDER = {"thd": K.THD, "htd": K.HTD, "paged": K.PAGED}


def desc_for(w, lens, layers=None):
    return K.make_desc(layers or w.layers, w.heads, w.head_dim, w.src_tp, w.dst_tp, w.dst_rank,
                       _F[w.src_dtype], _F[w.dst_dtype], _ORDER[w.src_order], w.block_size,
                       w.num_blocks, list(lens), w.src_block_size, w.src_num_blocks,
                       cache_dtype=_F[w.cache_dtype] if w.cache_dtype else 0)


def dev_u16(a):
    return None if a is None else torch.from_numpy(a.view(np.int16)).to(DEV)


def pool(w, layers, fill=W.SENTINEL):
    row = w.head_dim * dst_size(w)
    n = layers * 2 * w.num_blocks * w.block_size * w.hd
    cache = torch.full((n * row,), fill, dtype=torch.uint8, device=DEV)
    scales = None
    if w.cdt in FP8_NAMES:
        scales = torch.full((n * 4,), fill, dtype=torch.uint8, device=DEV).view(torch.float32)
    return cache, scales


def check_shapes(w, lens, bt, stride, dshards, layers, sbt=None):
    """Host-side check that every buffer the kernels will touch has the size
    the plan assumes (run before each launch)."""
    Hs, D = w.hs, w.head_dim
    if w.src_order == "paged":
        need = layers * 2 * w.src_num_blocks * w.src_block_size * Hs * D
        snb = max([(int(t) + w.src_block_size - 1) // w.src_block_size for t in lens] + [0])
        assert len(lens) == 0 or (sbt.shape[0] == len(lens) and sbt.shape[1] >= snb)
    else:
        need = sum(layers * 2 * int(t) * Hs * D for t in lens)
    for j in read_shards(w):
        assert dshards[j] is not None and dshards[j].numel() >= need, (j, need)
    assert len(lens) == 0 or (bt.shape[0] == len(lens) and bt.shape[1] >= stride)
    # page ids outside [0, num_blocks) or [0, src_num_blocks) are allowed:
    # the kernel skips them


def gpu_run(op, w, lens, bt, stride, shards, layers=None, wire_in=None, sbt=None):
    """Run 'repack', 'pack', 'pack_unpack' or 'unpack' (of wire_in) on the GPU.
    A paged source uses the generator's source block table unless `sbt` is
    given.  Returns (cache, scales, wire) device tensors (None where not
    produced)."""
    layers = layers or w.layers
    plan = K.kvx_plan(desc_for(w, lens, layers))
    info = K.kvx_plan_info_get(plan)
    dshards = [dev_u16(s) for s in shards] if shards is not None else None
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    paged = w.src_order == "paged"
    sbt_d = None
    if paged:
        if sbt is None:
            sbt, _ = W.src_block_table(w, lens)
        sbt = np.ascontiguousarray(sbt, dtype=np.int32)
        sbt_d = torch.from_numpy(sbt).to(DEV)
    if dshards is not None:
        check_shapes(w, lens, bt, stride, dshards, layers, sbt)
    cache = scales = wire = None
    if op in ("pack", "pack_unpack"):
        wire = torch.full((max(int(info.wire_bytes), 16),), W.SENTINEL, dtype=torch.uint8,
                          device=DEV)
        if paged:
            K.kvx_pack_paged(plan, dshards, sbt_d, sbt.shape[1], wire)
        else:
            K.kvx_pack(plan, dshards, wire)
    if op == "unpack":
        wire = torch.from_numpy(wire_in).to(DEV)
        assert wire.numel() >= info.wire_bytes
    if op in ("repack", "pack_unpack", "unpack"):
        cache, scales = pool(w, layers)
        if op == "repack" and paged:
            K.kvx_repack_paged(plan, dshards, sbt_d, sbt.shape[1], cache, scales, bt_d, stride)
        elif op == "repack":
            K.kvx_repack(plan, dshards, cache, scales, bt_d, stride)
        else:
            K.kvx_unpack(plan, wire, cache, scales, bt_d, stride)
    torch.cuda.synchronize()
    return cache, scales, wire


def oracle_pool(w, lens, bt, stride, shards, layers=None, op="repack", wire=None, sbt=None):
    layers = layers or w.layers
    p = oracle_problem(O, w, lens, layers, sbt=sbt)
    cache = np.full(O.cache_bytes(p), W.SENTINEL, dtype=np.uint8)
    scales = None
    if w.cdt in FP8_NAMES:
        scales = np.full(4 * O.scale_count(p), W.SENTINEL, dtype=np.uint8).view(np.float32)
    if op == "repack":
        O.repack(p, shards, cache, scales, bt, stride)
    else:
        O.unpack(p, wire, cache, scales, bt, stride)
    return cache, scales


def check_sampled(w, lens, bt, shards, cache, scales, layers, planes, requests, rng):
    """Compare the pages of the given requests in the given (layer, k/v)
    planes with the oracle's expected rows, byte for byte; the slots past
    the end of each request's last page must keep the sentinel.  Returns the
    number of rows compared."""
    p = oracle_problem(O, w, lens, layers)
    row = w.head_dim * dst_size(w)
    page = w.block_size * w.hd * row
    pages = cache.view(layers, 2, w.num_blocks, page)
    spages = None
    if scales is not None:
        spages = scales.view(layers, 2, w.num_blocks, w.block_size * w.hd)
    rows = 0
    for r in requests:
        T = int(lens[r])
        if T == 0:
            continue
        nb = (T + w.block_size - 1) // w.block_size
        ids = torch.from_numpy(bt[r, :nb].astype(np.int64)).to(DEV)
        for (l, kv) in planes:
            got = pages[l, kv].index_select(0, ids).cpu().numpy().reshape(nb * w.block_size, -1)
            want, want_s = O.expected_rows(p, shards, int(r), l, kv, 0, T)
            assert np.array_equal(got[:T].reshape(-1), want.reshape(-1)), (w.name, r, l, kv)
            assert np.all(got[T:] == W.SENTINEL), (w.name, r, l, kv, "tail")
            if spages is not None:
                gs = spages[l, kv].index_select(0, ids).cpu().numpy().reshape(-1)
                assert np.array_equal(gs[:T * w.hd].view(np.uint32), want_s.view(np.uint32)), \
                    (w.name, r, l, kv, "scales")
                assert np.all(gs[T * w.hd:].view(np.uint8) == W.SENTINEL)
            rows += T * w.hd
    return rows


def check_unused_pages(w, lens, bt, cache, layers, rng, count=64):
    """A sample of pages outside every block-table row keeps the sentinel."""
    used = set()
    for r, t in enumerate(lens):
        used.update(bt[r, :(int(t) + w.block_size - 1) // w.block_size].tolist())
    free = np.setdiff1d(np.arange(w.num_blocks), np.fromiter(used, dtype=np.int64))
    if free.size == 0:
        return
    pick = torch.from_numpy(rng.choice(free, min(count, free.size), replace=False)).to(DEV)
    page = w.block_size * w.hd * w.head_dim * dst_size(w)
    pages = cache.view(layers, 2, w.num_blocks, page)
    for l in {0, layers - 1}:
        for kv in (0, 1):
            assert bool((pages[l, kv].index_select(0, pick) == W.SENTINEL).all())
