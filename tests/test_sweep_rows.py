"""Host checks of the exhaustive 8-bit sweep's inputs and bookkeeping (the
GPU half is tests/test_gpu_fp8_exhaustive.py).

* pair_rows: for each row maximum m, the rows have maximum exactly m and
  together hold every finite pattern of magnitude <= m in both signs; NaN
  rows hold exactly one NaN each.
* The chunked comparison: with the whole problem's expected outputs computed
  by the oracle in one call (its repack into 8-bit and 16-bit caches), the
  per-chunk oracle sub-problems find no difference, and a single flipped
  code, scale or cache element is found in the right row.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
import test_gpu_fp8_exhaustive as X
from cases import FINITE_MAX, pair_rows


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
@pytest.mark.parametrize("nan", [False, True])
def test_pair_rows_cover_every_pair(fmt, nan):
    inf = 0x7F80 if fmt == "bf16" else 0x7C00
    mags = [1, 2, 3, 125, 126, 127, 128, 300, 0x0400, FINITE_MAX[fmt]]
    rows = pair_rows(fmt, mags, nan=nan, block=3)
    r = 0
    for m in mags:
        k = -(-(2 * (m + 1)) // (127 - int(nan)))
        blk = rows[r:r + k]
        r += k
        mag = blk & 0x7FFF
        fin = mag < inf
        assert np.all((~fin).sum(1) == int(nan))
        if nan:
            assert np.all(mag[~fin] > inf)          # NaNs, not infinities
        assert np.all(np.where(fin, mag, 0).max(1) == m)
        got = set(blk[fin].tolist())
        want = set(range(m + 1)) | {0x8000 | x for x in range(m + 1)}
        assert want <= got and got <= want
    assert r == rows.shape[0]


def test_pair_rows_place_the_maximum_in_every_column():
    rows = pair_rows("bf16", np.arange(1, 0x0800))
    cols = np.argmax(rows & 0x7FFF, axis=1)
    assert set(cols.tolist()) == set(range(128))
    assert ((rows >> 15).astype(np.int64) * (rows & 0x7FFF) > 0).any()   # negative maxima too


def _whole_problem(src, fmt, rows, cache_fmt=0):
    T = rows.shape[0] // 2
    p = O.OracleProblem(1, 1, 128, 1, 1, 0, X._O[src], X._O[fmt], O.TOKEN_MAJOR, 16, T // 16,
                        [T], cache_fmt=cache_fmt)
    return p, T


@pytest.mark.parametrize("src,fmt", [("bf16", "e4m3fn"), ("fp16", "e5m2")])
def test_chunked_comparison(monkeypatch, src, fmt):
    monkeypatch.setattr(X, "CHUNK_T", 64)
    rows = np.concatenate([pair_rows(src, [1, 200, 0x3C00, FINITE_MAX[src]]),
                           pair_rows(src, [77, 0x3800], nan=True)])
    rows = np.concatenate([rows, np.zeros((-rows.shape[0] % 128, 128), np.uint16)])
    n = rows.shape[0]
    p, T = _whole_problem(src, fmt, rows)
    bt = np.arange(T // 16, dtype=np.int32)[None, :]
    shard = [rows.reshape(-1)]
    codes = np.zeros(n * 128, np.uint8)
    scales = np.zeros(n, np.float32)
    O.repack(p, shard, codes, scales, bt, T // 16)
    caches = {}
    for c in ("bf16", "fp16"):
        pc, _ = _whole_problem(src, fmt, rows, X._O[c])
        out = np.zeros(n * 128, np.uint16)
        O.repack(pc, shard, out.view(np.uint8), None, bt, T // 16)
        caches[c] = out
    scales = scales.view(np.uint32)
    chunks = n // (2 * X.CHUNK_T)
    assert chunks >= 3
    run = lambda: [b for c in range(chunks)  # noqa: E731
                   for b in X._oracle_chunk(src, fmt, rows, c, codes, scales, caches)]
    assert run() == []
    # a wrong code, scale or cache element is reported in its row
    row = n - 2 * X.CHUNK_T + 5
    codes[row * 128 + 3] ^= 1
    scales[row] ^= 1
    caches["fp16"][row * 128 + 9] ^= 1
    bad = run()
    assert len(bad) == 3 and all(f"row {row}" in b for b in bad), bad
