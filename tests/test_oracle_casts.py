"""Pins of the oracle's casts (precision alignment) to things other than itself:
hand-worked values of the formats, torch/numpy library conversions, and the
mathematical error bound of the e4m3fn quantisation."""
import numpy as np
import pytest
import torch

from conftest import golden_lines

import oracle as O


def _all16():
    return np.arange(65536, dtype=np.uint32).astype(np.uint16)


def test_decode_fp16_matches_numpy():
    bits = _all16()
    ours = O.decode(O.FP16, bits)
    ref = bits.view(np.float16).astype(np.float64)
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    assert np.array_equal(np.signbit(ours[ok]), np.signbit(ref[ok]))


def test_decode_bf16_matches_torch():
    bits = _all16()
    ours = O.decode(O.BF16, bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])


def test_decode_e4m3_matches_torch():
    bits = np.arange(256, dtype=np.uint8)
    ours = O.decode(O.E4M3FN, bits)
    ref = torch.from_numpy(bits).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    assert np.nanmax(ours) == 448.0 and ours[1] == 2.0 ** -9


def test_fp16_to_bf16_golden():
    rows = golden_lines("fp16_to_bf16.txt")
    assert len(rows) >= 15
    for ln in rows:
        a, b = ln.split()[:2]
        got = int(O.fp16_to_bf16(np.array([int(a, 16)], dtype=np.uint16))[0])
        assert got == int(b, 16), (ln, hex(got))


def test_fp16_to_bf16_exhaustive_vs_torch():
    bits = _all16()
    ours = O.fp16_to_bf16(bits)
    f16 = torch.from_numpy(bits.view(np.int16)).view(torch.float16)
    ref = f16.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(bits.view(np.float16))
    assert np.array_equal(ours[~nan], ref[~nan])


def test_fp16_to_bf16_nan_reading():
    bits = _all16()
    nan = np.isnan(bits.view(np.float16))
    ours = O.fp16_to_bf16(bits[nan])
    src = bits[nan]
    assert np.all((ours & 0x7F80) == 0x7F80)           # exponent all ones
    assert np.all(ours & 0x0040)                        # quiet
    assert np.array_equal(ours >> 15, src >> 15)        # sign kept
    assert np.array_equal(ours & 0x3F, (src & 0x3FF) >> 3 & 0x3F)  # payload top bits


def _parse_float(tok):
    return float.fromhex(tok) if "0x" in tok.lower() else float(tok)


def test_bf16_to_fp16_golden():
    rows = golden_lines("bf16_to_fp16.txt")
    assert len(rows) == 21
    for ln in rows:
        b, want = (int(x, 16) for x in ln.split()[:2])
        got = int(O.bf16_to_fp16(np.array([b], dtype=np.uint16))[0])
        assert got == want, (ln, hex(got))


def test_bf16_to_fp16_exhaustive_vs_torch():
    """Every non-NaN bf16 pattern against torch's conversion (round to
    nearest even through float32, overflow to infinity)."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = O.bf16_to_fp16(bits)
    t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
    want = t.to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    nan = torch.isnan(t).numpy()
    assert nan.sum() == 2 * 127
    assert np.array_equal(got[~nan], want[~nan])


def test_bf16_to_fp16_nan_reading():
    """NaN: sign kept, quiet bit set, the 7 bf16 fraction bits at the top of
    the fp16 fraction."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    nan = ((bits & 0x7F80) == 0x7F80) & ((bits & 0x7F) != 0)
    got = O.bf16_to_fp16(bits[nan]).astype(np.uint32)
    b = bits[nan].astype(np.uint32)
    assert np.array_equal(got >> 15, b >> 15)
    assert np.all((got & 0x7C00) == 0x7C00) and np.all(got & 0x0200)
    assert np.array_equal((got >> 3) & 0x3F, b & 0x3F)


def test_e4m3_golden_values():
    rows = golden_lines("e4m3_values.txt")
    assert len(rows) >= 19
    for ln in rows:
        v, b = ln.split()[:2]
        got = int(O.f32_to_e4m3fn(np.array([_parse_float(v)], dtype=np.float32))[0])
        assert got == int(b, 16), (ln, hex(got))


def _torch_e4m3(v32: np.ndarray) -> np.ndarray:
    """Library reference: torch's float8_e4m3fn conversion (round to nearest
    even) after clamping to the finite range (torch itself maps out-of-range
    values to NaN rather than saturating)."""
    t = torch.from_numpy(v32).clamp(-448.0, 448.0).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy()


def test_e4m3_all_bf16_values_vs_torch():
    bits = _all16()
    v = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    fin = np.isfinite(v)
    assert np.array_equal(O.f32_to_e4m3fn(v[fin]), _torch_e4m3(v[fin]))


def test_e4m3_midpoints_and_neighbours_vs_torch():
    # every e4m3 grid midpoint and its fp32 neighbours: the tie and near-tie cases
    grid = O.decode(O.E4M3FN, np.arange(0, 0x7F, dtype=np.uint8))
    mids = ((grid[:-1] + grid[1:]) / 2).astype(np.float32)
    cases = [mids, np.nextafter(mids, np.float32(np.inf)), np.nextafter(mids, np.float32(0))]
    v = np.concatenate(cases + [grid.astype(np.float32)])
    v = np.concatenate([v, -v])
    assert np.array_equal(O.f32_to_e4m3fn(v), _torch_e4m3(v))


def test_e4m3_random_fp32_vs_torch():
    rng = np.random.default_rng(7)
    mant = rng.uniform(1.0, 2.0, 400_000)
    expo = rng.integers(-20, 12, 400_000)
    v = (mant * np.exp2(expo) * rng.choice([-1.0, 1.0], 400_000)).astype(np.float32)
    assert np.array_equal(O.f32_to_e4m3fn(v), _torch_e4m3(v))


def test_e4m3_nan_and_saturation():
    v = np.array([np.nan, -np.nan, np.inf, -np.inf, 3e38, -3e38], dtype=np.float32)
    got = O.f32_to_e4m3fn(v)
    assert got[0] == 0x7F and got[1] == 0xFF
    assert list(got[2:]) == [0x7E, 0xFE, 0x7E, 0xFE]


def test_row_scale_matches_numpy():
    rng = np.random.default_rng(3)
    for _ in range(200):
        x = (rng.standard_normal(128) * 10.0 ** rng.uniform(-30, 30)).astype(np.float32)
        ref = np.float32(np.max(np.abs(x))) / np.float32(448.0)
        assert O.row_scale(x) == ref
    assert O.row_scale(np.zeros(128, np.float32)) == 0.0
    x = np.array([1.0, np.nan, -2.0], np.float32)
    assert O.row_scale(x) == np.float32(2.0) / np.float32(448.0)


def test_e4m3_rows_golden():
    rows = golden_lines("e4m3_rows.txt")
    assert len(rows) >= 11
    for ln in rows:
        amax, x, s_bits, q = ln.split()[:4]
        amax, x = _parse_float(amax), _parse_float(x)
        row = torch.tensor([amax, x] + [0.0] * 6, dtype=torch.float32).to(torch.bfloat16)
        assert row[0].item() == amax and row[1].item() == x, ln   # exact in bf16
        bits = row.view(torch.int16).numpy().view(np.uint16)
        out, s = O.convert_row(O.BF16, O.E4M3FN, bits)
        assert np.float32(s).view(np.uint32) == int(s_bits, 16), (ln, hex(np.float32(s).view(np.uint32)))
        assert out[1] == int(q, 16), (ln, hex(out[1]))
        assert out[0] == 0x7E        # the amax element is +448
        assert np.all(out[2:] == 0)  # zeros stay +0


def test_convert_row_vs_torch_library_rows():
    """Whole rows against torch: s = amax/448 (fp32), q = e4m3(clamp(x/s))."""
    rng = np.random.default_rng(11)
    for src in (O.BF16, O.FP16):
        tdt = torch.bfloat16 if src == O.BF16 else torch.float16
        for _ in range(300):
            lim = 1e4 if src == O.FP16 else 1e30
            scale = min(10.0 ** rng.uniform(-6, 6), lim)
            x = torch.from_numpy((rng.standard_normal(128) * scale).astype(np.float32)).to(tdt)
            bits = x.view(torch.int16).numpy().view(np.uint16)
            out, s = O.convert_row(src, O.E4M3FN, bits)
            xf = x.float()
            s_ref = xf.abs().max() / torch.tensor(448.0)
            assert np.float32(s) == s_ref.item()
            if s_ref.item() == 0:
                continue
            q_ref = _torch_e4m3((xf / s_ref).numpy())
            assert np.array_equal(out, q_ref)


def test_e4m3_row_dequant_error_bound():
    """|q*s - x| <= max(2^-4 |x|, 2^-10 s) + 2^-22 |x|: half a grid step of
    e4m3 (3 fraction bits, subnormal step 2^-9) after the fp32 divide."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        x = torch.from_numpy((rng.standard_normal(128) * 10.0 ** rng.uniform(-3, 3))
                             .astype(np.float32)).to(torch.bfloat16)
        bits = x.view(torch.int16).numpy().view(np.uint16)
        out, s = O.convert_row(O.BF16, O.E4M3FN, bits)
        q = O.decode(O.E4M3FN, out)
        xd = x.double().numpy()
        err = np.abs(q * float(s) - xd)
        bound = np.maximum(2.0 ** -4 * np.abs(xd), 2.0 ** -10 * float(s)) + 2.0 ** -22 * np.abs(xd)
        assert np.all(err <= bound)
        assert np.max(np.abs(q)) == 448.0


def test_e4m3_zero_row_keeps_signs():
    bits = np.array([0x0000, 0x8000] * 4, dtype=np.uint16)
    out, s = O.convert_row(O.BF16, O.E4M3FN, bits)
    assert s == 0.0
    assert list(out) == [0x00, 0x80] * 4


def test_same_type_is_bit_copy():
    bits = np.arange(0, 65536, 517, dtype=np.uint32).astype(np.uint16)
    for f in (O.FP16, O.BF16):
        out, _ = O.convert_row(f, f, bits)
        assert np.array_equal(out.view(np.uint16), bits)


def test_e4m3_infinite_row_maximum():
    """A row holding +-Inf has scale Inf: finite elements give signed zeros,
    the infinite ones an invalid quotient, whose NaN code takes the element's
    sign (platform NaN signs differ; the reading fixes it)."""
    row = torch.tensor([1.0, -2.0, float("inf"), float("-inf"), 0.0, -0.0, 3.0, 1.0],
                       dtype=torch.float32).to(torch.bfloat16)
    out, s = O.convert_row(O.BF16, O.E4M3FN, row.view(torch.int16).numpy().view(np.uint16))
    assert np.isinf(s)
    assert list(out) == [0x00, 0x80, 0x7F, 0xFF, 0x00, 0x80, 0x00, 0x00]
