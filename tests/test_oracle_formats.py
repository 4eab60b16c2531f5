"""Pins of the oracle's number formats (CPU only).

bfloat16 rounding is checked against torch's CPU cast; the E4M3FN decoder
against the code table of the OCP FP8 specification (tests/golden) and
torch's float8_e4m3fn; the encoder exhaustively (round trip of every finite
code, every midpoint between neighbours) and against torch's cast on
in-range values.
"""
import json
import os

import numpy as np
import pytest
import torch

from oracle import formats

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_bf16_matches_torch_rne():
    rng = np.random.default_rng(11)
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32),
        (rng.standard_normal(20000) * 1e30).astype(np.float32),
        (rng.standard_normal(20000) * 1e-38).astype(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8], np.float32),
    ])
    mine = formats.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)


def test_bf16_ties_to_even():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7 in bf16 -> rounds to 1
    assert formats.bf16_bits_from_f32(np.float32(1.0 + 2 ** -8)) == 0x3F80
    # 1 + 3*2^-8 is halfway between 1+2^-7 and 1+2^-6 -> even = 1+2^-6
    assert formats.bf16_bits_from_f32(np.float32(1.0 + 3 * 2 ** -8)) == 0x3F82
    assert formats.bf16_bits_to_f64(np.uint16(0x3F82)) == 1.0 + 2 ** -6


def test_e4m3_table_matches_spec_golden():
    g = json.load(open(os.path.join(GOLD, "e4m3fn_codes.json")))
    for code_s, val in g["codes"]:
        c = int(code_s, 16)
        got = formats.E4M3_TABLE[c]
        if val == "nan":
            assert np.isnan(got)
        else:
            assert got == val and np.signbit(got) == np.signbit(val), (code_s, got, val)


def test_e4m3_table_matches_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mine = formats.E4M3_TABLE
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(mine))
    assert np.array_equal(ref[~nan], mine[~nan])
    assert int(nan.sum()) == 2


def test_e4m3_structure():
    t = formats.E4M3_TABLE
    pos = t[:0x7F]
    assert np.all(np.diff(pos) > 0)  # codes are monotone in value
    assert pos.max() == 448.0 and pos[1] == 2.0 ** -9
    assert np.array_equal(t[0x80:0xFF], -t[0x00:0x7F])


def test_e4m3_round_trip_every_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    assert np.array_equal(formats.e4m3_encode(formats.E4M3_TABLE[codes]), codes)


def test_e4m3_midpoints_tie_to_even():
    pos = formats.E4M3_TABLE[:0x7F]
    mids = (pos[:-1] + pos[1:]) / 2  # exact in float64
    codes = formats.e4m3_encode(mids)
    lo = np.arange(0x7E)
    expect = np.where(lo % 2 == 0, lo, lo + 1)
    assert np.array_equal(codes, expect.astype(np.uint8))
    # a hair either side of a midpoint goes to the nearer neighbour
    eps = np.spacing(mids)
    assert np.array_equal(formats.e4m3_encode(mids - eps), lo.astype(np.uint8))
    assert np.array_equal(formats.e4m3_encode(mids + eps), (lo + 1).astype(np.uint8))


def test_e4m3_golden_rounding():
    g = json.load(open(os.path.join(GOLD, "e4m3fn_codes.json")))
    for r in g["rounding"]:
        assert formats.e4m3_encode(np.float64(r["x"])) == int(r["code"], 16), r


def test_e4m3_encode_matches_torch_in_range():
    rng = np.random.default_rng(5)
    x = np.concatenate([
        rng.uniform(-448, 448, 100000),
        rng.standard_normal(100000) * 4,
        rng.standard_normal(100000) * 2 ** -7,
    ]).astype(np.float32)
    mine = formats.e4m3_encode(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(mine, ref)


def test_e4m3_encode_rejects_unclamped():
    with pytest.raises(ValueError):
        formats.e4m3_encode(np.float64(449.0))


def test_fp8_quantize_divides_in_binary32_and_saturates():
    x = np.array([1.0, 3.0, -1000.0, 1000.0, 0.0, -0.0], np.float32)
    s = np.array([3.0, 3.0, 1.0, 2.0, 5.0, 5.0], np.float32)
    got = formats.fp8_quantize(x, s)
    # fl32(1/3) = 0.3333333432674408 lies between 0.3125 (0x2A) and 0.34375
    # (0x2B) and is nearer the latter
    assert formats.E4M3_TABLE[0x2A] == 0.3125 and formats.E4M3_TABLE[0x2B] == 0.34375
    assert got[0] == 0x2B
    assert formats.E4M3_TABLE[got[1]] == 1.0
    assert got[2] == 0xFE and got[3] == 0x7E  # clamped to -448 / 448
    assert got[4] == 0x00 and got[5] == 0x80
    # a value at the edge of the saturation boundary: 464 / 1 is above 448
    assert formats.fp8_quantize(np.float32(464.0), np.float32(1.0)) == 0x7E
