"""Oracle helpers for the bf16 storage format.

TEST INFRASTRUCTURE ONLY -- never called by the product.

bf16 keeps the upper 16 bits of an IEEE binary32 pattern (sign, 8 exponent
bits, 7 fraction bits).  The paper runs its GEMM in bf16 (Section IV.A) and
leaves the output type to the DType parameter (Section III.A); the readings of
this build are bf16 inputs, fp32 accumulation, and fp32 or bf16 output with
round-to-nearest-even (reading A8).

Parity: pinned in tests/test_oracle_gemm.py against torch's own fp32->bf16
conversion (a library routine) and against hand-picked ties, overflow,
subnormal, infinity and NaN cases.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of each bf16 pattern as fp64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact value of each bf16 pattern as fp32."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32)


def f32_to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round binary32 values to bf16, to nearest with ties to even.

    For values of one sign the binary32 patterns are ordered like the values
    they encode, and the bf16 values are exactly the patterns whose low 16 bits
    are zero.  The two bf16 neighbours of a pattern u are therefore
    (u >> 16) << 16 and the next pattern up, and their midpoint is the pattern
    with low half 0x8000.  Below the midpoint rounds down, above rounds up, at
    the midpoint the neighbour with an even upper half wins.  A carry out of the
    fraction moves into the exponent, which is the correct next value (up to
    infinity).  NaNs stay NaN with the quiet bit set.
    """
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    upper = u >> np.uint64(16)
    lower = u & np.uint64(0xFFFF)
    round_up = (lower > 0x8000) | ((lower == 0x8000) & ((upper & np.uint64(1)) == 1))
    out = upper + round_up.astype(np.uint64)
    is_nan = (u & np.uint64(0x7FFFFFFF)) > np.uint64(0x7F800000)
    out = np.where(is_nan, upper | np.uint64(0x0040), out)
    return out.astype(np.uint16)
