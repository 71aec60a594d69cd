"""Pins of the oracle's storage-format decode tables.

The tables are built from the formats' bit-field definitions; here they are
checked exhaustively against an independent library routine (torch's casts)
and at values the format definitions fix.
"""
import math

import numpy as np
import pytest
import torch

from oracle import numerics


def test_bf16_table_matches_torch_exhaustively():
    codes = np.arange(1 << 16, dtype=np.uint16)
    ref = torch.from_numpy(codes.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    ours = numerics.bf16_table()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    # signed zeros too
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


def test_e4m3_table_matches_torch_exhaustively():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = numerics.e4m3_table()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


@pytest.mark.parametrize("code,value", [
    (0x38, 1.0), (0x7E, 448.0), (0xFE, -448.0), (0x08, 2.0 ** -6), (0x01, 2.0 ** -9),
    (0x07, 7 * 2.0 ** -9), (0x40, 2.0), (0x3C, 1.5), (0x00, 0.0),
])
def test_e4m3_spot_values(code, value):
    assert numerics.e4m3_value(code) == value


def test_e4m3_nan_codes_only_s1111111():
    nans = [c for c in range(256) if math.isnan(numerics.e4m3_value(c))]
    assert nans == [0x7F, 0xFF]


@pytest.mark.parametrize("code,value", [
    (0x3F80, 1.0), (0xBF80, -1.0), (0x4000, 2.0), (0x3F00, 0.5), (0x0001, 2.0 ** -133),
    (0x0080, 2.0 ** -126), (0x7F7F, (2 - 2 ** -7) * 2.0 ** 127), (0x7F80, math.inf), (0xFF80, -math.inf),
])
def test_bf16_spot_values(code, value):
    assert numerics.bf16_value(code) == value


def test_decode_dispatch():
    assert numerics.decode(np.array([0x3F80], dtype=np.uint16), "bf16")[0] == 1.0
    assert numerics.decode(np.array([0x38], dtype=np.uint8), "fp8_e4m3")[0] == 1.0
    with pytest.raises(ValueError):
        numerics.decode(np.zeros(1, np.uint8), "int4")
