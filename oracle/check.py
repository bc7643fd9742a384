"""The parity bar for GEMM outputs.

TEST INFRASTRUCTURE ONLY.

An output C passes against the fp64 oracle C_ref when, for every element,
|C - C_ref| <= 1e-2 * R with R = |A| * |B|, and the relative Frobenius error
||C - C_ref||_F / ||C_ref||_F is at most 4e-3.  These bounds cover fp32
accumulation (about K * 2^-24 * R in the worst case) and a final bf16
rounding (2^-9 relative); an accumulation in bf16, a dropped or doubled tile
or K slice fails them.
"""
from __future__ import annotations

import numpy as np

ELEM_TOL = 1e-2
FROB_TOL = 4e-3


def gemm_errors(C, C_ref, R):
    C = np.asarray(C, dtype=np.float64)
    C_ref = np.asarray(C_ref, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    diff = np.abs(C - C_ref)
    bad = ~(diff <= ELEM_TOL * R)          # NaN counts as bad
    ref_norm = float(np.sqrt(np.sum(C_ref * C_ref)))
    err_norm = float(np.sqrt(np.sum(diff * diff))) if not np.isnan(diff).any() else float("inf")
    rel = err_norm / ref_norm if ref_norm > 0 else (0.0 if err_norm == 0 else float("inf"))
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(R > 0, diff / (ELEM_TOL * R), np.where(diff == 0, 0.0, np.inf))
    return {
        "n_bad": int(bad.sum()),
        "max_ratio": float(np.nanmax(ratio)) if ratio.size else 0.0,
        "rel_frob": rel,
    }


def assert_gemm_close(C, C_ref, R, what: str = ""):
    e = gemm_errors(C, C_ref, R)
    assert e["n_bad"] == 0 and e["rel_frob"] <= FROB_TOL, f"{what}: {e}"
    return e
