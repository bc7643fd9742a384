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


MODEL_SRC = open(os.path.join(ROOT, "oracle", "model.py")).read()
MODEL_MUTANTS = {
    "no_patch_sharing": ("t_blk = brgemm_clk(G, gamma, beta / math.sqrt(patch),", "t_blk = brgemm_clk(G, gamma, beta,"),
    "panel_a_uses_bn": ("BM * BK * 2.0, BK * BN * 2.0)", "BN * BK * 2.0, BK * BN * 2.0)"),
    "gamma_ignores_occupancy": ("gamma = w / (FLOPS_PER_CLK_CU * RATE[shape])", "gamma = 1 / (FLOPS_PER_CLK_CU * RATE[shape])"),
    "sharing_ignores_grid_size": ("w = min(o, max(1, -(-active // num_cus)))", "w = o"),
    "copies_not_read_back": ("2 * c * M * N * 4 + M * N * out_bytes", "c * M * N * 4 + M * N * out_bytes"),
    "no_reduction_launch": ("launches = 1 if c == 1 else 2", "launches = 1"),
    "blocks_not_split": ("blocks = -(-nK // c)", "blocks = nK"),
    "rounds_floor": ("rounds = -(-tasks // slots)", "rounds = max(1, tasks // slots)"),
    "eq1_sum": ("return max(G * gamma, beta * (s_a + s_b))", "return G * gamma + beta * (s_a + s_b)"),
    "ties_keep_last": ("clk <= b_clk + tol and pad < b_pad)", "clk <= b_clk + tol and pad <= b_pad)"),
}


def _model_pins(mod):
    """The pins of tests/test_oracle_model.py, run on a mutant; returns failures."""
    fails = []
    occ = {(128, 128): 2, (256, 128): 1, (128, 256): 1, (256, 256): 1}
    if abs(mod.brgemm_clk(8388608, 1 / 3031.04, 0.01, 32768, 32768) - 2767.5676) > 1e-3:
        fails.append("eq1 compute")
    if abs(mod.brgemm_clk(8388608, 1 / 3031.04, 0.1, 32768, 32768) - 6553.6) > 1e-6:
        fails.append("eq1 memory")
    clk, pad = mod.estimate(1024, 1024, 65536, 4, 256, occ, (128, 256), 8)
    if abs(clk - 246330.85) > 246330.85 * 1e-8 or pad != 256 * 128 * 256:
        fails.append("worked estimate")
    rate = mod.RATE
    mod.RATE = {**rate, (256, 128): rate[(128, 256)]}   # symmetry holds for equal rates
    for (M, N, K) in [(3000, 7000, 2048), (1024, 4096, 8192), (8192, 512, 65536), (777, 5000, 1000)]:
        for s in mod.SHAPES:
            for c in mod.LAYERS:
                a = mod.estimate(M, N, K, 4, 256, occ, s, c)
                b = mod.estimate(N, M, K, 4, 256, occ, (s[1], s[0]), c)
                if abs(a[0] - b[0]) > 1e-12 * abs(a[0]) or a[1] != b[1]:
                    fails.append("symmetry")
    mod.RATE = rate
    if mod.choose(1024, 1024, 65536, out_bytes=4)[1] <= 1:
        fails.append("k-dominant layers")
    if mod.choose(8192, 8192, 8192, out_bytes=2)[:2] != ((256, 256), 1):
        fails.append("square")
    if mod.choose(512, 512, 128, layers=8)[1] != 2:
        fails.append("cap")
    r = mod.choose(0, 0, 64)
    if r[:2] != ((256, 256), 1) or r[2] != mod.LAUNCH_CLK:
        fails.append("ties")
    # worked tie case: the same M x N x K with one layer available twice
    if mod.choose(512, 512, 64, shape=(128, 128), layers=8)[1] != 1:
        fails.append("cap to one block")
    clk, _ = mod.estimate(8192, 8192, 8192, 4, 4096, occ, (128, 256), 1)
    if abs(clk - 316783.38) > 316783.38 * 1e-8:
        fails.append("memory-bound worked estimate")
    clk, _ = mod.estimate(512, 512, 512, 4, 256, occ, (128, 128), 1)
    if abs(clk - 19524.8184) > 19524.8184 * 1e-8:
        fails.append("small-grid worked estimate")
    clk, _ = mod.estimate(4096, 4096, 512, 4, 256, occ, (128, 128), 1)
    want = 10000 + 2 * 8 * max(2097152 * 2 / 1818.624, 512 / 3500 * 32768 / 8) + 4096 * 4096 * 4 / 3500
    if abs(clk - want) > want * 1e-9:
        fails.append("shared-CU worked estimate")
    return fails


@pytest.mark.parametrize("name", sorted(MODEL_MUTANTS))
def test_model_mutant_fails_a_pin(name):
    old, new = MODEL_MUTANTS[name]
    assert old in MODEL_SRC, name
    mod = types.ModuleType("model_mutant_" + name)
    exec(compile(MODEL_SRC.replace(old, new, 1), name, "exec"), mod.__dict__)
    assert _model_pins(mod), f"mutant {name} passed every pin"


def test_model_oracle_passes_its_pins():
    from oracle import model
    assert _model_pins(model) == []
