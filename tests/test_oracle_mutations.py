"""Plausible mistakes planted in copies of the oracle must fail its pins.

Each mutant is a textual edit of oracle/sfc_ref.py (or oracle/gemm_ref.c),
loaded or compiled on the CPU in a temporary place; the real oracle is not
touched."""
import importlib.util
import os
import subprocess
import sys
import types

import numpy as np
import pytest

import sfc_pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SFC_SRC = open(os.path.join(ROOT, "oracle", "sfc_ref.py")).read()

SFC_MUTANTS = {
    "long_test_ge": ("if 2 * major > 3 * minor:", "if 2 * major >= 3 * minor:"),
    "no_major_growth": ("if hmajor % 2 == 1 and major > 2:", "if False:"),
    "no_minor_growth": ("if hminor % 2 == 1 and minor > 2:", "if False:"),
    "third_start_off": ("y + (ay - say) + (hby - sby),", "y + (ay - say) + hby,"),
    "third_minor_sign": ("-hbx, -hby, -(ax - hax), -(ay - hay)", "-hbx, -hby, (ax - hax), (ay - hay)"),
    "second_axes_swapped": ("yield from _walk(x + hbx, y + hby, ax, ay, bx - hbx, by - hby, halving)",
                            "yield from _walk(x + hbx, y + hby, bx - hbx, by - hby, ax, ay, halving)"),
    "top_level_tie_to_y": ("if gm >= gn:\n        return list(_walk(0, 0, gm, 0, 0, gn, halving))",
                           "if gm > gn:\n        return list(_walk(0, 0, gm, 0, 0, gn, halving))"),
    "trunc_halving": ('def sfc_cells(gm: int, gn: int, halving: str = "floor")',
                      'def sfc_cells(gm: int, gn: int, halving: str = "trunc")'),
}


def _load_mutant(name, old, new):
    assert old in SFC_SRC, name
    mod = types.ModuleType("sfc_mutant_" + name)
    exec(compile(SFC_SRC.replace(old, new, 1), name, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(SFC_MUTANTS))
def test_sfc_mutant_fails_a_pin(name):
    mod = _load_mutant(name, *SFC_MUTANTS[name])

    def cells(a, b):
        try:
            return mod.sfc_cells(a, b)
        except RecursionError:
            return []
    fails = sfc_pins.all_pins(cells, sweep_max=24)
    if name == "trunc_halving":
        # floor vs trunc only differ on larger grids (reading A1); the pins cannot
        # prefer one reading, the frozen table can.
        fails = fails + ([] if mod.sfc_cells(10, 10) == __import__("oracle.sfc_ref").sfc_ref.sfc_cells(10, 10)
                         else ["differs from the frozen floor reading on 10x10"])
    assert fails, f"mutant {name} passed every pin"


GEMM_SRC = open(os.path.join(ROOT, "oracle", "gemm_ref.c")).read()
GEMM_MUTANTS = {
    "drop_last_k": ("for (k = 0; k < K; ++k) {\n            const double a = bf16_to_f64(A[i * lda + k]);\n            const double aa",
                    "for (k = 0; k < K - 1; ++k) {\n            const double a = bf16_to_f64(A[i * lda + k]);\n            const double aa"),
    "transposed_b": ("const uint16_t *brow = B + k * ldb;", "const uint16_t *brow = B + k;"),
    "wrong_decode": ("uint32_t u = ((uint32_t)h) << 16;", "uint32_t u = ((uint32_t)h) << 15;"),
    "lda_ignored": ("const double a = bf16_to_f64(A[i * lda + k]);\n            const double aa",
                    "const double a = bf16_to_f64(A[i * K + k]);\n            const double aa"),
    "sign_flip": ("c[j] += a * b;", "c[j] -= a * b;"),
}


def _compile_mutant(tmp_path, name, old, new):
    assert old in GEMM_SRC, name
    src = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    src.write_text(GEMM_SRC.replace(old, new, 1))
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", str(src), "-o", str(so), "-lm"], check=True)
    import ctypes
    lib = ctypes.CDLL(str(so))
    i64, p = ctypes.c_int64, ctypes.c_void_p
    lib.gemm_ref_rows.argtypes = [i64, i64, i64, i64, p, i64, p, i64, p, p]
    return lib


@pytest.mark.parametrize("name", sorted(GEMM_MUTANTS))
def test_gemm_mutant_fails_a_pin(tmp_path, name):
    import test_oracle_gemm as pins
    lib = _compile_mutant(tmp_path, name, *GEMM_MUTANTS[name])

    def rows(A, B, N, K, lda, ldb, M):
        A = np.ascontiguousarray(A, dtype=np.uint16)
        B = np.ascontiguousarray(B, dtype=np.uint16)
        C = np.empty((M, N))
        R = np.empty((M, N))
        lib.gemm_ref_rows(0, M, N, K, A.ctypes.data, lda, B.ctypes.data, ldb, C.ctypes.data, R.ctypes.data)
        return C, R
    assert pins.gemm_pin_failures(rows), f"mutant {name} passed every pin"
