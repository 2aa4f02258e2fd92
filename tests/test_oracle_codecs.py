"""Pins of the oracle's number formats against torch's casts and the OCP FP8 spec."""
import math

import numpy as np
import pytest
import torch

from oracle import bf16_bits_to_f64, e4m3fn_decode, e4m3fn_encode_rne


def test_e4m3fn_decode_matches_torch_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    mine = e4m3fn_decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(mine[ok], ref[ok])
    assert np.array_equal(np.signbit(mine[ok]), np.signbit(ref[ok]))


@pytest.mark.parametrize("code,value", [
    (0x00, 0.0), (0x01, 2.0 ** -9), (0x07, 7 * 2.0 ** -9), (0x08, 2.0 ** -6),
    (0x38, 1.0), (0x39, 1.125), (0x40, 2.0), (0x7E, 448.0), (0xB8, -1.0), (0xFE, -448.0),
])
def test_e4m3fn_known_values(code, value):
    # OCP 8-bit floating point spec: E4M3 bias 7, max normal 448, min subnormal 2^-9
    assert e4m3fn_decode(np.uint8(code)) == value


def test_e4m3fn_nan_codes_only():
    vals = e4m3fn_decode(np.arange(256, dtype=np.uint8))
    assert set(np.nonzero(np.isnan(vals))[0].tolist()) == {0x7F, 0xFF}
    assert not np.any(np.isinf(vals))


def test_e4m3fn_encode_roundtrip_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(e4m3fn_encode_rne(e4m3fn_decode(codes)), codes)


def test_e4m3fn_encode_ties_and_random_match_torch():
    finite = np.sort(np.unique(np.abs(e4m3fn_decode(np.arange(0x7F, dtype=np.uint8)))))
    mids = (finite[1:] + finite[:-1]) / 2  # exact ties (representable in fp32)
    rng = np.random.default_rng(7)
    rand = rng.uniform(-448, 448, size=20000)
    small = rng.uniform(-0.05, 0.05, size=20000)
    x = np.concatenate([mids, -mids, rand, small, finite, -finite]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    mine = e4m3fn_encode_rne(x.astype(np.float64))
    assert np.array_equal(mine, ref)


def test_e4m3fn_encode_tie_goes_to_even():
    # 1.0625 is halfway between 1.0 (0x38, even) and 1.125 (0x39)
    assert e4m3fn_encode_rne(np.array([1.0625]))[0] == 0x38
    # 1.1875 is halfway between 1.125 (0x39) and 1.25 (0x3A, even)
    assert e4m3fn_encode_rne(np.array([1.1875]))[0] == 0x3A
    assert e4m3fn_encode_rne(np.array([np.nan]))[0] == 0x7F
    with pytest.raises(ValueError):
        e4m3fn_encode_rne(np.array([449.0]))


def test_bf16_decode_matches_torch():
    bits = np.arange(0, 65536, 7, dtype=np.uint32).astype(np.uint16)
    mine = bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(mine[ok], ref[ok])
    assert bf16_bits_to_f64(np.uint16(0x3F80)) == 1.0
    assert bf16_bits_to_f64(np.uint16(0xC000)) == -2.0
    assert math.isnan(bf16_bits_to_f64(np.uint16(0x7FC0)))
