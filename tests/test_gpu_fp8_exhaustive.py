"""Exhaustive GPU parity of the 8-bit conversions (precision alignment,
Sec. I contribution 1; readings R9, R10, R25, R26) against the oracle.

The code an 8-bit conversion writes for an element depends only on that
element and on its row's scale, and the scale depends only on the row
maximum.  So rows that hold, for every finite 16-bit row maximum m, every
finite pattern x with |x| <= m in both signs cover every (scale, element)
pair a finite row can produce: 1.07e9 elements for bf16 sources (maxima
0x0001..0x7F7F), 1.01e9 for fp16 (0x0001..0x7BFF).  This pins the kernels'
scale sequence, their one-correction quotient and the hardware fp8 / bf8
conversions against the definition (an fp32 amax / fmax, then each x / s
rounded once to fp32 and once, saturating, to the 8-bit grid).  The rows
also hold:

* for every 16th row maximum, the same pairs in rows that also contain a NaN
  (their scale is finite, so every element goes through the general path's
  correctly rounded quotient);
* zero rows up to the padding (s = 0).

Per (source format, 8-bit format) the GPU runs, on one one-layer,
one-head, 128-dim problem of all those rows:

* kvx_pack: the transfer tensor's codes and scales are compared with the
  oracle's pack, byte for byte;
* kvx_repack into an 8-bit cache under the identity page table: compared
  on the device with the transfer tensor (same rows in the same order);
* for a bf16 and an fp16 cache: kvx_repack quantising and dequantising in
  one pass, and kvx_unpack dequantising the transfer tensor; the two are
  compared on the device, then with the oracle's unpack of its own transfer
  tensor (the oracle's repack equals its unpack of its pack, an invariant its
  own tests pin).

The oracle runs on host threads, one sub-problem of CHUNK_T tokens each.
"""
from __future__ import annotations

import os
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as O
from cases import FINITE_MAX, pair_rows
from gpu_util import DEV, log

import paper_2509_17542_amd as K

pytestmark = pytest.mark.gpu

CHUNK_T = 8192   # tokens of one oracle sub-problem (2 * CHUNK_T rows)
_K = {"bf16": K.BF16, "fp16": K.FP16, "e4m3fn": K.E4M3FN, "e5m2": K.E5M2}
_O = {"bf16": O.BF16, "fp16": O.FP16, "e4m3fn": O.E4M3FN, "e5m2": O.E5M2}


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def sweep_rows(src):
    """All (row maximum, element) pairs, the NaN rows, then zero rows up to a
    multiple of 2 * CHUNK_T rows."""
    top = FINITE_MAX[src]
    full = pair_rows(src, np.arange(1, top + 1))
    nan = pair_rows(src, np.unique(np.r_[np.arange(1, top + 1, 16), top]), nan=True)
    n = full.shape[0] + nan.shape[0]
    n_pad = -(-n // (2 * CHUNK_T)) * (2 * CHUNK_T)
    rows = np.zeros((n_pad, 128), dtype=np.uint16)
    rows[:full.shape[0]] = full
    rows[full.shape[0]:n] = nan
    return rows, full.shape[0], nan.shape[0]


def _plan(src, fmt, T, cache=None):
    return K.kvx_plan(K.make_desc(1, 1, 128, 1, 1, 0, _K[src], _K[fmt], K.THD, 16, T // 16, [T],
                                  cache_dtype=_K[cache] if cache else 0))


def _oracle_chunk(src, fmt, rows, c, codes, scales, caches):
    """Oracle for rows [2*CHUNK_T*c, 2*CHUNK_T*(c+1)): its pack, then its
    unpack of that transfer tensor into each 16-bit cache; each compared with
    the GPU's rows.  Returns a list of mismatch descriptions."""
    T = CHUNK_T
    r0, r1 = 2 * T * c, 2 * T * (c + 1)
    shard = np.ascontiguousarray(rows[r0:r1]).reshape(-1)
    p = O.OracleProblem(1, 1, 128, 1, 1, 0, _O[src], _O[fmt], O.TOKEN_MAJOR, 16, T // 16, [T])
    doff, soff, _ = O.wire_layout(p)
    wire = O.pack(p, [shard])
    bad = []
    want_c = wire[int(doff[0]):int(doff[0]) + 2 * T * 128]
    if not np.array_equal(want_c, codes[r0 * 128:r1 * 128]):
        i = int(np.nonzero(want_c != codes[r0 * 128:r1 * 128])[0][0])
        row = r0 + i // 128
        bad.append(f"code: row {row} col {i % 128} x=0x{int(rows[row, i % 128]):04x} "
                   f"gpu 0x{int(codes[r0 * 128 + i]):02x} oracle 0x{int(want_c[i]):02x}")
    want_s = wire[int(soff[0]):int(soff[0]) + 8 * T].view(np.uint32)
    got_s = scales[r0:r1]
    if not np.array_equal(want_s, got_s):
        i = int(np.nonzero(want_s != got_s)[0][0])
        bad.append(f"scale: row {r0 + i} gpu 0x{int(got_s[i]):08x} oracle 0x{int(want_s[i]):08x}")
    bt = np.arange(T // 16, dtype=np.int32)[None, :]
    for cache, got in caches.items():
        pc = O.OracleProblem(1, 1, 128, 1, 1, 0, _O[src], _O[fmt], O.TOKEN_MAJOR, 16, T // 16,
                             [T], cache_fmt=_O[cache])
        want = np.zeros(2 * T * 128, dtype=np.uint16)
        O.unpack(pc, wire, want.view(np.uint8), None, bt, T // 16)
        g = got[r0 * 128:r1 * 128]
        if not np.array_equal(want, g):
            i = int(np.nonzero(want != g)[0][0])
            row = r0 + i // 128
            bad.append(f"{cache} cache: row {row} col {i % 128} x=0x{int(rows[row, i % 128]):04x} "
                       f"gpu 0x{int(g[i]):04x} oracle 0x{int(want[i]):04x}")
    return bad


@pytest.mark.parametrize("src,fmt", [("bf16", "e4m3fn"), ("fp16", "e4m3fn"), ("bf16", "e5m2"),
                                     ("fp16", "e5m2")])
def test_every_row_maximum_and_element(src, fmt):
    t_start = time.time()
    rows, n_full, n_nan = sweep_rows(src)
    n = rows.shape[0]
    T = n // 2
    log(f"{src}->{fmt} exhaustive: {n_full} rows of all pairs, {n_nan} NaN rows, "
        f"{n - n_full - n_nan} zero rows ({n * 128} elements), generated in "
        f"{time.time() - t_start:.1f}s")
    assert T % CHUNK_T == 0

    src_d = torch.from_numpy(rows.reshape(-1).view(np.int16)).to(DEV)
    bt = torch.arange(T // 16, dtype=torch.int32, device=DEV)[None, :].contiguous()
    p8 = _plan(src, fmt, T)
    info = K.kvx_plan_info_get(p8)
    doff, soff = K.kvx_plan_segment(p8, 0)
    wire = torch.zeros(int(info.wire_bytes), dtype=torch.uint8, device=DEV)
    K.kvx_pack(p8, [src_d], wire)
    cache8 = torch.zeros(n * 128, dtype=torch.uint8, device=DEV)
    scales8 = torch.zeros(n, dtype=torch.float32, device=DEV)
    K.kvx_repack(p8, [src_d], cache8, scales8, bt, T // 16)
    torch.cuda.synchronize()
    codes_d = wire[doff:doff + n * 128]
    scales_d = wire[soff:soff + 4 * n]
    assert torch.equal(cache8, codes_d), "8-bit repack differs from the pack's codes"
    assert torch.equal(scales8.view(torch.uint8), scales_d), "repack scales differ from the pack's"
    del cache8, scales8
    caches = {}
    for cache in ("bf16", "fp16"):
        pc = _plan(src, fmt, T, cache)
        assert K.kvx_plan_info_get(pc).wire_bytes == info.wire_bytes
        qd = torch.zeros(n * 128, dtype=torch.int16, device=DEV)
        K.kvx_repack(pc, [src_d], qd, None, bt, T // 16)
        dq = torch.zeros(n * 128, dtype=torch.int16, device=DEV)
        K.kvx_unpack(pc, wire, dq, None, bt, T // 16)
        torch.cuda.synchronize()
        assert torch.equal(qd, dq), f"quantise-dequantise repack differs from the unpack ({cache})"
        del dq
        caches[cache] = qd.cpu().numpy().view(np.uint16)
        del qd
    codes = codes_d.cpu().numpy()
    scales = scales_d.cpu().numpy().view(np.uint32)
    del src_d, wire, codes_d, scales_d
    torch.cuda.empty_cache()
    log(f"{src}->{fmt} exhaustive: GPU done at {time.time() - t_start:.1f}s; oracle on "
        f"{_threads()} threads")

    chunks = n // (2 * CHUNK_T)
    with ThreadPoolExecutor(_threads()) as ex:
        results = list(ex.map(lambda c: _oracle_chunk(src, fmt, rows, c, codes, scales, caches),
                              range(chunks)))
    bad = [b for r in results for b in r]
    log(f"{src}->{fmt} exhaustive: {chunks} oracle chunks compared in "
        f"{time.time() - t_start:.1f}s, {len(bad)} mismatching")
    assert not bad, f"{len(bad)} chunks differ; first: {bad[:6]}"
