"""Exact decode of the storage formats the KV cache and queries use.

Test infrastructure only (see the package header).

The paper serves Llama-3-70B in BF16 (Sec. 4.1, "Model and hardware") and
Qwen3-235B-A22B with FP8 quantization (Sec. 4.7 case study).  It does not say
which FP8 variant; the reading taken here is OCP FP8 E4M3 ("e4m3fn": exponent
bias 7, no infinities, only S.1111.111 is NaN, largest finite 448), the format
gfx950's matrix and conversion units use natively.

Both tables are built from the bit-field definitions of the formats, in
float64, with no library conversion routine involved.  Pins (tests/):
exhaustive agreement with torch's own casts for all 65,536 bf16 and 256 e4m3
codes, plus spot values fixed by the format definitions.
"""
from __future__ import annotations

import math

import numpy as np

_BF16_TABLE: np.ndarray | None = None
_E4M3_TABLE: np.ndarray | None = None


def bf16_value(code: int) -> float:
    """Value of one bfloat16 bit pattern (1 sign, 8 exponent, 7 mantissa bits, bias 127)."""
    sign = -1.0 if (code >> 15) & 1 else 1.0
    exp = (code >> 7) & 0xFF
    man = code & 0x7F
    if exp == 0xFF:
        return sign * math.inf if man == 0 else math.nan
    if exp == 0:
        return sign * math.ldexp(man / 128.0, -126)
    return sign * math.ldexp(1.0 + man / 128.0, exp - 127)


def e4m3_value(code: int) -> float:
    """Value of one OCP E4M3 (e4m3fn) bit pattern (1 sign, 4 exponent, 3 mantissa bits, bias 7)."""
    sign = -1.0 if (code >> 7) & 1 else 1.0
    exp = (code >> 3) & 0xF
    man = code & 0x7
    if exp == 0xF and man == 0x7:
        return math.nan
    if exp == 0:
        return sign * math.ldexp(man / 8.0, -6)
    return sign * math.ldexp(1.0 + man / 8.0, exp - 7)


def bf16_table() -> np.ndarray:
    """float64[65536]: value of every bfloat16 code."""
    global _BF16_TABLE
    if _BF16_TABLE is None:
        _BF16_TABLE = np.array([bf16_value(c) for c in range(1 << 16)], dtype=np.float64)
    return _BF16_TABLE


def e4m3_table() -> np.ndarray:
    """float64[256]: value of every E4M3 code."""
    global _E4M3_TABLE
    if _E4M3_TABLE is None:
        _E4M3_TABLE = np.array([e4m3_value(c) for c in range(256)], dtype=np.float64)
    return _E4M3_TABLE


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """Decode an array of bf16 bit patterns (uint16 or int16) to float64."""
    return bf16_table()[np.asarray(bits).view(np.uint16)]


def decode_e4m3(bits: np.ndarray) -> np.ndarray:
    """Decode an array of E4M3 bit patterns (uint8) to float64."""
    return e4m3_table()[np.asarray(bits).view(np.uint8)]


def decode(bits: np.ndarray, fmt: str) -> np.ndarray:
    if fmt == "bf16":
        return decode_bf16(bits)
    if fmt == "fp8_e4m3":
        return decode_e4m3(bits)
    raise ValueError(f"unknown storage format {fmt!r}")
