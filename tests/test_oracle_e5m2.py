"""Pins of the oracle's e5m2 transfer format (reading R26: the e4m3fn scheme
with OCP e5m2 codes, a per-(token, head) scale max|x| / 57344 and a
saturating round-to-nearest-even cast; precision alignment, Sec. I) to things
other than itself: hand-worked values of the format, torch's float8_e5m2
decode and conversion, whole rows against torch, the quantisation error
bound, the dequantisation of every code, and whole workloads against a
paged-attention reader built from torch."""
import numpy as np
import pytest
import torch

from cases import SMALL_E5M2, consumer_rows, gather_pages, inputs, oracle_problem
from conftest import golden_lines

import oracle as O
import workload as W

_TDT = {O.BF16: torch.bfloat16, O.FP16: torch.float16}


def _parse_float(tok):
    return float.fromhex(tok) if "0x" in tok.lower() else float(tok)


def _torch_e5m2(v32: np.ndarray) -> np.ndarray:
    """Library reference: torch's float8_e5m2 conversion (round to nearest
    even) after clamping to the finite range (torch maps magnitudes that round
    past 57344 to infinity rather than saturating)."""
    t = torch.from_numpy(v32).clamp(-57344.0, 57344.0).to(torch.float8_e5m2)
    return t.view(torch.uint8).numpy()


def test_decode_e5m2_matches_torch():
    bits = np.arange(256, dtype=np.uint8)
    ours = O.decode(O.E5M2, bits)
    ref = torch.from_numpy(bits).view(torch.float8_e5m2).double().numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    assert np.array_equal(np.signbit(ours[ok]), np.signbit(ref[ok]))
    # 0x7C / 0xFC are the infinities; 0x7D..0x7F and 0xFD..0xFF NaN
    assert np.isinf(ours[0x7C]) and ours[0xFC] == -np.inf
    assert np.isnan(ours[[0x7D, 0x7E, 0x7F, 0xFD, 0xFE, 0xFF]]).all()
    assert ours[0x7B] == 57344.0 and ours[0x01] == 2.0 ** -16 and ours[0x04] == 2.0 ** -14


def test_e5m2_golden():
    rows = golden_lines("e5m2_values.txt")
    assert len(rows) >= 26
    for ln in rows:
        v, b = ln.split()[:2]
        got = int(O.f32_to_e5m2(np.array([_parse_float(v)], dtype=np.float32))[0])
        assert got == int(b, 16), (ln, hex(got))


def test_e5m2_all_fp16_values_vs_torch():
    """Every finite fp16 value (e5m2 is fp16 with 8 fraction bits dropped)."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = bits.view(np.float16).astype(np.float32)
    fin = np.isfinite(v)
    assert np.array_equal(O.f32_to_e5m2(v[fin]), _torch_e5m2(v[fin]))


def test_e5m2_midpoints_and_neighbours_vs_torch():
    grid = O.decode(O.E5M2, np.arange(0, 0x7C, dtype=np.uint8))
    mids = ((grid[:-1] + grid[1:]) / 2).astype(np.float32)
    cases = [mids, np.nextafter(mids, np.float32(np.inf)), np.nextafter(mids, np.float32(0))]
    v = np.concatenate(cases + [grid.astype(np.float32)])
    v = np.concatenate([v, -v])
    assert np.array_equal(O.f32_to_e5m2(v), _torch_e5m2(v))


def test_e5m2_random_fp32_vs_torch():
    rng = np.random.default_rng(9)
    mant = rng.uniform(1.0, 2.0, 400_000)
    expo = rng.integers(-22, 18, 400_000)
    v = (mant * np.exp2(expo) * rng.choice([-1.0, 1.0], 400_000)).astype(np.float32)
    assert np.array_equal(O.f32_to_e5m2(v), _torch_e5m2(v))


def test_e5m2_rows_vs_torch_library_rows():
    """Whole rows: s = amax / 57344 (fp32 divide), q = e5m2(clamp(x / s))."""
    rng = np.random.default_rng(12)
    for src in (O.BF16, O.FP16):
        for _ in range(300):
            lim = 1e4 if src == O.FP16 else 1e30
            scale = min(10.0 ** rng.uniform(-6, 6), lim)
            x = torch.from_numpy((rng.standard_normal(128) * scale).astype(np.float32)).to(_TDT[src])
            out, s = O.convert_row(src, O.E5M2, x.view(torch.int16).numpy().view(np.uint16))
            xf = x.float()
            s_ref = xf.abs().max() / torch.tensor(57344.0)
            assert np.float32(s) == s_ref.item()
            if s_ref.item() == 0:
                continue
            assert np.array_equal(out, _torch_e5m2((xf / s_ref).numpy()))


def test_e5m2_row_error_bound():
    """|q*s - x| <= max(2^-3 |x|, 2^-17 s) + 2^-22 |x|: half a grid step of
    e5m2 (2 fraction bits, subnormal step 2^-16) after the fp32 divide."""
    rng = np.random.default_rng(6)
    for _ in range(200):
        x = torch.from_numpy((rng.standard_normal(128) * 10.0 ** rng.uniform(-3, 3))
                             .astype(np.float32)).to(torch.bfloat16)
        out, s = O.convert_row(O.BF16, O.E5M2, x.view(torch.int16).numpy().view(np.uint16))
        q = O.decode(O.E5M2, out)
        xd = x.double().numpy()
        err = np.abs(q * float(s) - xd)
        bound = np.maximum(2.0 ** -3 * np.abs(xd), 2.0 ** -17 * float(s)) + 2.0 ** -22 * np.abs(xd)
        assert np.all(err <= bound)
        assert np.max(np.abs(q)) == 57344.0


def test_e5m2_special_rows():
    """Zero rows keep signed zeros; a row holding +-Inf has scale Inf, its
    finite elements give signed zeros and the infinite ones the NaN code with
    the element's sign; a NaN element gives the NaN code."""
    zero = np.array([0x0000, 0x8000] * 4, dtype=np.uint16)
    out, s = O.convert_row(O.BF16, O.E5M2, zero)
    assert s == 0.0 and list(out) == [0x00, 0x80] * 4
    # bf16 bits: 1, -2, +Inf, -Inf, +0, -0, +NaN, -NaN
    row = np.array([0x3F80, 0xC000, 0x7F80, 0xFF80, 0x0000, 0x8000, 0x7FC0, 0xFFC1], np.uint16)
    out, s = O.convert_row(O.BF16, O.E5M2, row)
    assert np.isinf(s)
    assert list(out) == [0x00, 0x80, 0x7F, 0xFF, 0x00, 0x80, 0x7F, 0xFF]


@pytest.mark.parametrize("fmt", [O.BF16, O.FP16])
def test_e5m2_dequant_every_code_vs_torch(fmt):
    """All 256 codes under 200 scales: bits equal torch's q.float() * s then
    .to() (infinite codes give infinities); NaN codes give the quiet NaN with
    the code's sign."""
    rng = np.random.default_rng(8)
    scales = np.concatenate([2.0 ** rng.uniform(-40, 20, 190), 2.0 ** np.arange(-10, 0)])
    codes = np.arange(256, dtype=np.uint8)
    nan = ((codes & 0x7C) == 0x7C) & ((codes & 0x03) != 0)
    canon = 0x7FC0 if fmt == O.BF16 else 0x7E00
    for s in scales.astype(np.float32):
        got = O.dequant_row(fmt, codes, s, O.E5M2)
        q = torch.from_numpy(codes).view(torch.float8_e5m2).float()
        want = (q * torch.tensor(s, dtype=torch.float32)).to(_TDT[fmt]).view(torch.int16).numpy()
        assert np.array_equal(got[~nan], want.view(np.uint16)[~nan]), s
        assert np.array_equal(got[nan], ((codes[nan].astype(np.uint16) >> 7) << 15) | canon)
    # an infinite code under a zero scale: the product is NaN
    got = O.dequant_row(O.BF16, np.array([0x7C, 0xFC], np.uint8), np.float32(0.0), O.E5M2)
    assert list(got) == [0x7FC0, 0xFFC0]


@pytest.mark.parametrize("name", list(SMALL_E5M2))
def test_e5m2_workloads_match_paged_reader(name):
    w = SMALL_E5M2[name]
    lens, bt, stride, shards = inputs(w)
    p = oracle_problem(O, w, lens)
    assert O.validate(p) == 0
    cache = np.full(O.cache_bytes(p), W.SENTINEL, dtype=np.uint8)
    scales = None
    if w.cdt == "e5m2":
        scales = np.full(4 * O.scale_count(p), W.SENTINEL, dtype=np.uint8).view(np.float32)
    O.repack(p, shards, cache, scales, bt, stride)
    for r in range(len(lens)):
        want, want_s = consumer_rows(w, lens, r, 0, w.layers)
        got, got_s = gather_pages(cache, w, lens, bt, r, w.layers, scales)
        assert np.array_equal(got, want), (name, r)
        if want_s is not None:
            assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32)), (name, r)
    # unpack of pack is the repack
    c2 = np.full(O.cache_bytes(p), W.SENTINEL, dtype=np.uint8)
    s2 = None if scales is None else np.full_like(scales, np.nan)
    if s2 is not None:
        s2.view(np.uint8)[:] = W.SENTINEL
    O.unpack(p, O.pack(p, shards), c2, s2, bt, stride)
    assert np.array_equal(cache, c2)
    if scales is not None:
        assert np.array_equal(scales.view(np.uint32), s2.view(np.uint32))


def test_validate_e5m2():
    base = dict(layers=1, heads=8, head_dim=128, src_tp=1, dst_tp=1, dst_rank=0, src_fmt=O.BF16,
                src_order=O.TOKEN_MAJOR, block_size=16, num_blocks=8, seq_lens=[10])
    for cache in (0, O.E5M2, O.BF16, O.FP16):
        assert O.validate(O.OracleProblem(dst_fmt=O.E5M2, cache_fmt=cache, **base)) == 0
    assert O.validate(O.OracleProblem(dst_fmt=O.E5M2, cache_fmt=O.E4M3FN, **base)) == -2
    assert O.validate(O.OracleProblem(dst_fmt=O.E4M3FN, cache_fmt=O.E5M2, **base)) == -2
    assert O.validate(O.OracleProblem(dst_fmt=O.BF16, cache_fmt=O.E5M2, **base)) == -2
    assert O.validate(O.OracleProblem(dst_fmt=O.E5M2, **dict(base, src_fmt=O.E5M2))) == -2
