"""Oracle helpers for the OCP 8-bit float operand formats E4M3 and E5M2.

TEST INFRASTRUCTURE ONLY -- never called by the product.

The paper keeps the data type a parameter of the method (Section III.A); the
8-bit variant of this build reads A and B as OCP FP8 E4M3 codes: 1 sign bit,
4 exponent bits with bias 7, 3 mantissa bits.  Exponent field 0 holds the
subnormals m/8 * 2^-6; the code with all exponent and mantissa bits set is
NaN; there are no infinities (the largest finite value is 448).  Every E4M3
value has at most 4 significant bits and an exponent in [-9, 8], so it is
exactly a bf16 value, and the fp64 GEMM oracle of gemm.py computes the
reference from the bf16 patterns of the decoded values.

E5M2: 1 sign bit, 5 exponent bits with bias 15, 2 mantissa bits, laid out as
an IEEE binary format: exponent field 0 holds the subnormals m/4 * 2^-14, the
all-ones exponent holds infinity (mantissa 0) and NaN (mantissa != 0), the
largest finite value is 57344.  Every finite E5M2 value has at most 3
significant bits and an exponent in [-16, 15], so it too is exactly a bf16
value (and the infinities are bf16 infinities).

Parity: pinned in tests/test_oracle_fp8.py against torch's float8_e4m3fn and
float8_e5m2 to float32 conversions (library routines) on all 256 codes, hand
values of each format (1, -1, the largest finite value, the smallest normal
and subnormal values, signed zeros, NaN, and for E5M2 the infinities), the
ordering of the positive codes, the exactness of the bf16 encoding, and
planted mistakes.
"""
from __future__ import annotations

import numpy as np

from oracle import bf16 as obf16

NAN_E4M3 = 0x7F


def e4m3_value(code: int) -> float:
    """Value of one E4M3 code, from the format's definition."""
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return s * (m / 8.0) * 2.0 ** -6
    return s * (1.0 + m / 8.0) * 2.0 ** (e - 7)


_TABLE = np.array([e4m3_value(c) for c in range(256)], dtype=np.float64)


def e4m3_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact values of an array of E4M3 codes (uint8)."""
    return _TABLE[np.asarray(bits, dtype=np.uint8)]


def e4m3_to_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """bf16 patterns of the decoded values (exact: no rounding happens)."""
    v = e4m3_to_f64(bits).astype(np.float32)
    return obf16.f32_to_bf16_rne(v)


NAN_E5M2 = 0x7F


def e5m2_value(code: int) -> float:
    """Value of one E5M2 code, from the format's definition."""
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 2) & 0x1F
    m = code & 0x3
    if e == 0x1F:
        return s * float("inf") if m == 0 else float("nan")
    if e == 0:
        return s * (m / 4.0) * 2.0 ** -14
    return s * (1.0 + m / 4.0) * 2.0 ** (e - 15)


_TABLE5 = np.array([e5m2_value(c) for c in range(256)], dtype=np.float64)


def e5m2_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact values of an array of E5M2 codes (uint8)."""
    return _TABLE5[np.asarray(bits, dtype=np.uint8)]


def e5m2_to_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """bf16 patterns of the decoded values (exact: no rounding happens)."""
    v = e5m2_to_f64(bits).astype(np.float32)
    return obf16.f32_to_bf16_rne(v)


def to_bf16_bits(bits: np.ndarray, fmt: str) -> np.ndarray:
    """bf16 patterns of fp8 codes of format fmt ("e4m3" or "e5m2")."""
    return {"e4m3": e4m3_to_bf16_bits, "e5m2": e5m2_to_bf16_bits}[fmt](bits)
