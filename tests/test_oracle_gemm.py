"""Pins of the GEMM, bf16 and CA oracles against exact arithmetic, library
routines and closed forms."""
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import ca as oca
from oracle import check as ocheck
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import NAN_BF16, draw


def _vals(bits):
    return obf16.bf16_to_f64(bits)


def gemm_pin_failures(rows_fn):
    """Run the closed-form pins against ``rows_fn(A, B, N, K, lda, ldb, M) -> (C, R)``."""
    fails = []
    # 1. Integer-valued inputs: every partial sum is an exact integer.
    for (M, N, K) in [(7, 5, 9), (16, 3, 33), (5, 8, 1), (3, 4, 64)]:
        A = draw(M, K, ("int", -4, 4), 11 + K)
        B = draw(K, N, ("int", -4, 4), 12 + K)
        C, R = rows_fn(A, B, N, K, K, N, M)
        Ai = _vals(A).astype(np.int64)
        Bi = _vals(B).astype(np.int64)
        if not np.array_equal(C, (Ai @ Bi).astype(np.float64)):
            fails.append(f"integer {M}x{N}x{K}: C differs from the exact integer product")
        if not np.array_equal(R, (np.abs(Ai) @ np.abs(Bi)).astype(np.float64)):
            fails.append(f"integer {M}x{N}x{K}: R differs from |A||B|")
    # 2. Identity B gives A exactly; lda and ldb padding (NaN) never leaks.
    M, K = 6, 10
    A = draw(M, K, ("uniform", -1, 1), 21, ld=16)
    I = np.full((K, 12), NAN_BF16, dtype=np.uint16)
    I[:, :K] = 0
    I[np.arange(K), np.arange(K)] = 0x3F80
    C, R = rows_fn(A, I, K, K, 16, 12, M)
    if not np.array_equal(C, _vals(A[:, :K])):
        fails.append("identity B: C != A")
    # 3. K = 1 is an exact outer product.
    a = draw(9, 1, ("normal", 0, 1), 31)
    b = draw(1, 7, ("normal", 0, 1), 32)
    C, R = rows_fn(a, b, 7, 1, 1, 7, 9)
    if not np.array_equal(C, np.outer(_vals(a[:, 0]), _vals(b[0]))):
        fails.append("K=1: not the outer product")
    # 4. Random values against exact rational arithmetic (tiny).
    M, N, K = 3, 4, 13
    A = draw(M, K, ("uniform", -1, 1), 41, ld=K + 3)
    B = draw(K, N, ("uniform", -1, 1), 42, ld=N + 2)
    C, R = rows_fn(A, B, N, K, K + 3, N + 2, M)
    av, bv = _vals(A), _vals(B)
    if not np.isfinite(C).all():
        return fails + ["non-finite output on finite inputs"]
    for i in range(M):
        for j in range(N):
            exact = sum(Fraction(float(av[i, k])) * Fraction(float(bv[k, j])) for k in range(K))
            if abs(Fraction(float(C[i, j])) - exact) > Fraction(K) * Fraction(2) ** -52 * Fraction(float(R[i, j])):
                fails.append(f"rational check failed at ({i},{j})")
    return fails


def test_gemm_pins():
    def rows(A, B, N, K, lda, ldb, M):
        return ogemm.gemm_ref_rows(A, B, N, K, lda, ldb, M=M)
    assert gemm_pin_failures(rows) == []


def test_gemm_against_library_matmul():
    M, N, K = 37, 29, 300
    A = draw(M, K, ("normal", 0, 1), 51)
    B = draw(K, N, ("normal", 0, 1), 52)
    C, R = ogemm.gemm_ref_rows(A, B, N, K, K, N, M=M)
    ref = _vals(A) @ _vals(B)
    scale = (np.abs(_vals(A)) @ np.abs(_vals(B))).max()
    assert np.allclose(C, ref, rtol=0, atol=1e-12 * scale)
    assert np.allclose(R, np.abs(_vals(A)) @ np.abs(_vals(B)), rtol=1e-13, atol=0)


def test_points_match_rows():
    M, N, K = 20, 30, 70
    A = draw(M, K, ("uniform", -1, 1), 61, ld=72)
    B = draw(K, N, ("uniform", -1, 1), 62, ld=32)
    C, R = ogemm.gemm_ref_rows(A, B, N, K, 72, 32, M=M)
    rng = np.random.default_rng(0)
    rows = rng.integers(0, M, 50)
    cols = rng.integers(0, N, 50)
    Cp, Rp = ogemm.gemm_ref_points(A, B, K, 72, 32, rows, cols)
    assert np.array_equal(Cp, C[rows, cols]) and np.array_equal(Rp, R[rows, cols])


def test_row_block_matches_full():
    M, N, K = 12, 9, 40
    A = draw(M, K, ("uniform", -1, 1), 71)
    B = draw(K, N, ("uniform", -1, 1), 72)
    C, _ = ogemm.gemm_ref_rows(A, B, N, K, K, N, M=M)
    Cb, _ = ogemm.gemm_ref_rows(A, B, N, K, K, N, row0=5, nrows=4)
    assert np.array_equal(Cb, C[5:9])


def test_k_zero_gives_zero():
    A = np.zeros((3, 1), np.uint16)
    B = np.zeros((1, 4), np.uint16)
    C, R = ogemm.gemm_ref_rows(A, B, 4, 0, 1, 4, M=3)
    assert (C == 0).all() and (R == 0).all()


# ---------------------------------------------------------------- bf16 rounding
def test_rne_matches_torch_conversion():
    rng = np.random.default_rng(5)
    x = np.concatenate([
        rng.normal(0, 1, 20000), rng.normal(0, 1e-38, 2000), rng.normal(0, 1e38, 2000),
        rng.uniform(-3e38, 3e38, 2000)]).astype(np.float32)
    x = np.concatenate([x, np.array([0.0, -0.0, np.inf, -np.inf, 3.4028235e38, -3.4028235e38,
                                     1e-45, -1e-45, 1.17549435e-38], np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(obf16.f32_to_bf16_rne(x), want)


def test_rne_ties_and_nan():
    # 1 + 2^-8 sits halfway between 1 and 1 + 2^-7: ties to the even pattern (1.0).
    # 1 + 3*2^-8 sits halfway between 1 + 2^-7 and 1 + 2^-6: ties to 1 + 2^-6.
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 1 + 2 ** -8 + 2 ** -20], np.float32)
    assert obf16.f32_to_bf16_rne(x).tolist() == [0x3F80, 0x3F82, 0xBF80, 0x3F81]
    big = np.array([np.float32(3.4028235e38)])          # rounds up past the largest bf16
    assert obf16.f32_to_bf16_rne(big).tolist() == [0x7F80]
    nan = np.array([np.float32("nan")])
    r = obf16.f32_to_bf16_rne(nan)[0]
    assert (r & 0x7F80) == 0x7F80 and (r & 0x7F) != 0


def test_bf16_decode_exact():
    bits = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F, 0x8000], np.uint16)
    v = obf16.bf16_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 2.0 ** -133 and v[4] == 0.0
    assert v[3] == (2 - 2 ** -7) * 2.0 ** 127


# ---------------------------------------------------------------- CA split
@pytest.mark.parametrize("K,c,bk", [(65536, 1, 64), (65536, 2, 64), (65536, 4, 64), (65536, 8, 64),
                                    (1000, 3, 64), (70, 8, 64), (64, 4, 64), (1, 2, 64), (0, 4, 64),
                                    (640, 3, 64)])
def test_k_slices_tile_k(K, c, bk):
    s = oca.k_slices(K, c, bk)
    assert s[0][0] == 0 and s[-1][1] == K
    assert all(a[1] == b[0] for a, b in zip(s, s[1:]))
    nk = -(-K // bk)
    assert len(s) == max(1, min(c, nk))
    blocks = [-(-(e - b) // bk) if e > b else 0 for b, e in s]
    if K > 0:
        assert max(blocks) - min(blocks) <= 1 and min(blocks) >= 1
    assert all(b % bk == 0 for b, _ in s)


def test_k_slices_even_split_matches_listing():
    # Listing 1: layer l starts at block l * Kb_per_layer when the blocks divide evenly.
    K, bk = 65536, 64
    for c in (1, 2, 4, 8):
        kb_per_layer = (K // bk) // c
        assert oca.k_slices(K, c, bk) == [(l * kb_per_layer * bk, (l + 1) * kb_per_layer * bk) for l in range(c)]


def test_layer_reduction_exact_on_integers_and_ordered():
    rng = np.random.default_rng(3)
    W = rng.integers(-1000, 1000, size=(5, 7, 9)).astype(np.float32)
    assert np.array_equal(oca.reduce_layers_f32(W), W.astype(np.int64).sum(0).astype(np.float32))
    # fp32 left-to-right: (1e8 + 1 - 1e8) = 0 in fp32 but 1 if summed in another order
    W2 = np.array([[[1e8]], [[1.0]], [[-1e8]]], np.float32)
    assert oca.reduce_layers_f32(W2)[0, 0] == np.float32(0.0)


# ---------------------------------------------------------------- parity bar
def test_check_accepts_rounding_and_rejects_dropped_work():
    M, N, K = 64, 64, 512
    A = draw(M, K, ("normal", 0, 1), 81)
    B = draw(K, N, ("normal", 0, 1), 82)
    C, R = ogemm.gemm_ref_rows(A, B, N, K, K, N, M=M)
    ocheck.assert_gemm_close(C.astype(np.float32), C, R)
    ocheck.assert_gemm_close(obf16.bf16_to_f64(obf16.f32_to_bf16_rne(C.astype(np.float32))), C, R)
    dropped = C.copy()
    dropped[:32, :32] = 0                             # a missing output tile
    assert ocheck.gemm_errors(dropped, C, R)["n_bad"] > 0
    # a missing K slice (half the contraction)
    Ch, _ = ogemm.gemm_ref_rows(A, B, N, K // 2, K, N, M=M)
    assert ocheck.gemm_errors(Ch, C, R)["n_bad"] > 0
    nan = C.copy()
    nan[3, 3] = np.nan
    assert ocheck.gemm_errors(nan, C, R)["n_bad"] == 1
