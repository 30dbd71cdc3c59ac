"""Pins of the oracle's dequantising unpack (reading R25: the transfer tensor
carries e4m3fn codes and per-row fp32 scales, the decode cache keeps 16-bit
values q * s; precision alignment, Sec. I, applied on the receiving side): the
dequantisation against torch's fp8 -> fp32 widening, fp32 product and 16-bit
cast for every code, the whole path against a paged-attention reader built
from torch, unpack of pack = repack, and the error bound of the round trip."""
import numpy as np
import pytest
import torch

from cases import (SMALL_DEQUANT, consumer_rows, double_rounding_scales, dst_size, gather_pages,
                   inputs, oracle_problem)

import oracle as O
import workload as W

_TDT = {O.BF16: torch.bfloat16, O.FP16: torch.float16}


@pytest.mark.parametrize("fmt", [O.BF16, O.FP16])
def test_dequant_every_code_vs_torch(fmt):
    """All 256 codes under 200 scales (2^-40 .. 2^30, random mantissas, plus
    exact powers of two) and the scales whose products round differently
    through fp32 than at once: bits equal torch's q.float() * s then .to()
    (an fp32 product, then the 16-bit cast); NaN codes give the quiet NaN
    with the code's sign."""
    rng = np.random.default_rng(7)
    dr = double_rounding_scales(11 if fmt == O.FP16 else 8)
    assert len(dr) >= 8
    scales = np.concatenate([2.0 ** rng.uniform(-40, 30, 190), 2.0 ** np.arange(-10, 0), dr])
    codes = np.arange(256, dtype=np.uint8)
    nan = (codes & 0x7F) == 0x7F
    canon = 0x7FC0 if fmt == O.BF16 else 0x7E00
    for s in scales.astype(np.float32):
        got = O.dequant_row(fmt, codes, s)
        q = torch.from_numpy(codes).view(torch.float8_e4m3fn).float()
        want = (q * torch.tensor(s, dtype=torch.float32)).to(_TDT[fmt]).view(torch.int16).numpy()
        want = want.view(np.uint16)
        assert np.array_equal(got[~nan], want[~nan]), s
        assert np.array_equal(got[nan], ((codes[nan].astype(np.uint16) >> 7) << 15) | canon)


def test_dequant_fp16_overflow_and_subnormals():
    """Products above 65504 round to infinity in an fp16 cache; tiny ones
    become fp16 subnormals or zero, all by round to nearest even."""
    codes = np.array([0x7E, 0xFE, 0x01, 0x08, 0x38], dtype=np.uint8)   # 448, -448, 2^-9, 2^-6, 1
    got = O.dequant_row(O.FP16, codes, np.float32(2.0 ** 8))
    assert list(got[:2]) == [0x7C00, 0xFC00]             # 448 * 256 > 65504
    got = O.dequant_row(O.FP16, codes, np.float32(2.0 ** -16))
    assert got[2] == 0x0000                               # 2^-25: tie to even, 0
    assert got[3] == 0x0004                               # 2^-22 = 4 units of 2^-24
    assert got[4] == 0x0100                               # 2^-16 = 256 units
    # the edge of the fp16 range: the fp32 product 448 * 146.2 (about 65497.6)
    # lies between the fp16 points 65472 and 65504 (spacing 32 in [2^15,
    # 2^16)), nearer 65504 = 0x7BFF, so it stays finite; 448 * 146.25 = 65520
    # is the midpoint of 65504 (odd significand) and 65536 (even, past the
    # largest finite value), so it rounds to infinity
    got = O.dequant_row(O.FP16, codes[:2], np.float32(146.2))
    assert list(got) == [0x7BFF, 0xFBFF]
    got = O.dequant_row(O.FP16, codes[:2], np.float32(146.25))
    assert list(got) == [0x7C00, 0xFC00]


@pytest.mark.parametrize("name", list(SMALL_DEQUANT))
def test_dequant_repack_matches_paged_reader(name):
    w = SMALL_DEQUANT[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    assert O.validate(p) == 0
    cache = np.full(O.cache_bytes(p), W.SENTINEL, dtype=np.uint8)
    O.repack(p, shards, cache, None, bt, stride)
    for r in range(len(lens)):
        want, _ = consumer_rows(w, lens, r, 0, w.layers)
        got, _ = gather_pages(cache, w, lens, bt, r, w.layers)
        assert np.array_equal(got, want), (name, r)


@pytest.mark.parametrize("name", list(SMALL_DEQUANT))
def test_dequant_unpack_of_pack_equals_repack(name):
    w = SMALL_DEQUANT[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    c1 = np.full(O.cache_bytes(p), W.SENTINEL, dtype=np.uint8)
    O.repack(p, shards, c1, None, bt, stride)
    c2 = np.full(O.cache_bytes(p), W.SENTINEL, dtype=np.uint8)
    O.unpack(p, O.pack(p, shards), c2, None, bt, stride)
    assert np.array_equal(c1, c2)
    # and the transfer tensor is the e4m3fn one of a plain e4m3fn plan
    q = oracle_problem(O, w.replace(cache_dtype=""), lens)
    assert np.array_equal(O.pack(p, shards), O.pack(q, shards))


def test_dequant_round_trip_error_bound():
    """|q*s - x| <= 2^-4 |x| (e4m3 rounding, 3 fraction bits) + 2^-10 s (the
    subnormal step) + the fp32 product and 16-bit cast (2^-8 |x| for bf16)."""
    w = SMALL_DEQUANT["dequant_bf16_e4m3_bf16"]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    cache = np.full(O.cache_bytes(p), W.SENTINEL, dtype=np.uint8)
    O.repack(p, shards, cache, None, bt, stride)
    for r in range(len(lens)):
        got, _ = gather_pages(cache, w, lens, bt, r, w.layers)
        y = torch.from_numpy(got.reshape(-1).view(np.int16)).view(torch.bfloat16).float().numpy()
        x = torch.from_numpy(W.logical_values(w, lens, r, 0, w.layers)).to(torch.bfloat16).float()
        x = x.permute(0, 1, 3, 2, 4).reshape(-1, w.head_dim).numpy()
        y = y.reshape(x.shape)
        s = np.abs(x).max(axis=1, keepdims=True) / np.float32(448.0)
        bound = np.abs(x) * (2.0 ** -4 + 2.0 ** -8) * 1.001 + s * 2.0 ** -10 * 1.001
        assert np.all(np.abs(y - x) <= bound)


@pytest.mark.parametrize("cache", [O.FP16, O.BF16, O.E4M3FN])
def test_validate_cache_formats(cache):
    base = dict(layers=1, heads=8, head_dim=128, src_tp=1, dst_tp=1, dst_rank=0, src_fmt=O.BF16,
                src_order=O.TOKEN_MAJOR, block_size=16, num_blocks=8, seq_lens=[10])
    assert O.validate(O.OracleProblem(dst_fmt=O.E4M3FN, cache_fmt=cache, **base)) == 0
    # a cache format that differs from a 16-bit transfer format is not a conversion
    if cache != O.BF16:
        assert O.validate(O.OracleProblem(dst_fmt=O.BF16, cache_fmt=cache, **base)) == -2
