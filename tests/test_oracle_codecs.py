"""Pins for the oracle's number-format codecs.

They are checked against the format definitions themselves (bit embedding of
bf16 into binary32, hand-computed e4m3 code values, round-half-to-even at
exact midpoints, saturation at 448) and cross-checked against torch's CPU
casts, an independent implementation of the same formats."""

import numpy as np
import pytest
import torch

from oracle.codecs import (bf16_decode, bf16_encode_rne, e4m3_decode,
                           e4m3_encode_rne_sat, f32_round)


def _all_bf16():
    return np.arange(65536, dtype=np.uint32).astype(np.uint16)


def test_bf16_decode_is_upper_half_of_binary32():
    b = _all_bf16()
    with np.errstate(invalid="ignore"):
        ref = (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    got = bf16_decode(b)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def test_bf16_roundtrip_every_finite_value():
    b = _all_bf16()
    v = bf16_decode(b)
    fin = np.isfinite(v)
    back = bf16_encode_rne(v[fin])
    # ±0 both encode to themselves
    assert np.array_equal(back, b[fin])


def test_bf16_midpoints_round_to_even():
    # around 1.0 the bf16 ulp is 2^-7
    cases = {
        1.0 + 2.0 ** -8: 1.0,                     # tie between 1 (even) and 1+2^-7
        1.0 + 3 * 2.0 ** -8: 1.0 + 2.0 ** -6,      # tie between 1+2^-7 (odd) and 1+2^-6
        1.0 + 2.0 ** -8 + 2.0 ** -30: 1.0 + 2.0 ** -7,  # just above the tie
        -(1.0 + 2.0 ** -8): -1.0,
        2.0 ** -134: 0.0,                          # half the smallest subnormal (2^-133): tie to 0
        2.0 ** -133: 2.0 ** -133,                  # the smallest subnormal itself
        3 * 2.0 ** -134: 2.0 ** -132,              # 1.5 subnormal ulps -> 2 ulps (even)
        3.4e38: np.inf,                            # beyond max + half ulp
    }
    for x, want in cases.items():
        assert bf16_decode(bf16_encode_rne(np.array([x])))[0] == want, x


def test_bf16_encode_matches_torch_cast():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(200000).astype(np.float32),
                        (rng.standard_normal(20000) * 1e-38).astype(np.float32),
                        (rng.standard_normal(20000) * 1e30).astype(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_encode_rne(x.astype(np.float64)), ref)


def test_e4m3_decode_definition_values():
    d = e4m3_decode(np.arange(256, dtype=np.uint8))
    assert d[0x00] == 0.0 and d[0x01] == 2.0 ** -9 and d[0x07] == 7 * 2.0 ** -9
    assert d[0x08] == 2.0 ** -6 and d[0x38] == 1.0 and d[0x3C] == 1.5
    assert d[0x7E] == 448.0 and np.isnan(d[0x7F]) and np.isnan(d[0xFF])
    assert d[0x80] == 0.0 and np.signbit(d[0x80]) and d[0xFE] == -448.0
    fin = np.isfinite(d)
    assert fin.sum() == 254
    pos = np.sort(d[:0x7F])
    assert np.all(np.diff(pos) > 0)          # strictly increasing over 0x00..0x7E


def test_e4m3_decode_matches_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = e4m3_decode(np.arange(256, dtype=np.uint8))
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def test_e4m3_roundtrip_and_midpoints():
    codes = np.arange(0x7F, dtype=np.uint8)              # 0 .. 448
    v = e4m3_decode(codes)
    assert np.array_equal(e4m3_encode_rne_sat(v), codes)
    assert np.array_equal(e4m3_encode_rne_sat(-v[1:]), codes[1:] | 0x80)
    mids = (v[:-1] + v[1:]) / 2
    got = e4m3_encode_rne_sat(mids)
    lo, hi = codes[:-1], codes[1:]
    want = np.where(lo % 2 == 0, lo, hi)                 # even mantissa wins a tie
    assert np.array_equal(got, want)


def test_e4m3_saturates():
    x = np.array([448.0, 460.0, 464.0, 500.0, 1e9, -1e9, -470.0])
    assert list(e4m3_decode(e4m3_encode_rne_sat(x))) == [448, 448, 448, 448, 448, -448, -448]


def test_e4m3_encode_matches_torch_inside_range():
    rng = np.random.default_rng(2)
    x = np.concatenate([rng.standard_normal(100000) * 50, rng.standard_normal(10000) * 0.01])
    x = np.clip(x, -447.0, 447.0)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = e4m3_encode_rne_sat(x.astype(np.float32).astype(np.float64))
    assert np.array_equal(got, ref)


def test_f32_round():
    assert f32_round(np.array([1.0 + 2.0 ** -24]))[0] == 1.0
    assert f32_round(np.array([1.0 + 3 * 2.0 ** -24]))[0] == 1.0 + 2.0 ** -22
