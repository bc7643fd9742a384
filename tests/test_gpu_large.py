"""Parity at the size limits, through the C ABI: operands, outputs and layer
workspaces larger than 4 GiB (every byte offset past 2^32 must be formed in
64 bits), and leading dimensions on both sides of the limits that decide
between the 16-byte load path and the element path.

Large operands are periodic along K: a seeded (M, P) block repeated K/P times,
so that the oracle needs only the sampled rows; rows differ, so an address
that lost its high bits would read another row and fail the check.  Outputs
are compared on sampled points and on whole rows, among them the rows that
straddle byte offset 2^32."""
import numpy as np
import pytest
import torch

from oracle import check as ocheck
from oracle import fp8 as of8
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import NAN_E4M3, draw, draw_e4m3
from gpu_util import raw_bits, sg, to_host

pytestmark = pytest.mark.gpu

U = ("uniform", -1.0, 1.0)
GiB4 = 1 << 32


def padded_bf16(bits, ld):
    """(rows, ld) bf16 CUDA tensor: bits in the first columns, NaN after."""
    rows, cols = bits.shape
    t = torch.full((rows, ld), float("nan"), dtype=torch.bfloat16, device="cuda")
    t[:, :cols] = sg().to_device_bf16(bits)
    return t


def periodic_bf16(block, reps, ld):
    """(rows, ld) bf16 CUDA tensor holding block repeated reps times along the
    columns, NaN after."""
    rows, p = block.shape
    t = torch.full((rows, ld), float("nan"), dtype=torch.bfloat16, device="cuda")
    t[:, :p * reps] = sg().to_device_bf16(block).repeat(1, reps)
    return t


def straddling_row(ld_bytes, nrows):
    """The row whose bytes include offset 2^32, if there is one."""
    r = GiB4 // ld_bytes
    return r if r < nrows else None


def check_rows(C_dev, rows, A_rows, B, N, K, what):
    """Whole rows of C against the oracle; A_rows[i] is row rows[i] of A."""
    Cr, R = ogemm.gemm_ref_rows(A_rows, B, N, K, A_rows.shape[1], B.shape[1], M=len(rows))
    got = to_host(C_dev[torch.tensor(rows, device="cuda")])
    ocheck.assert_gemm_close(got, Cr, R, what)


def check_points(C_dev, A, B, K, n_points, seed, what):
    """Sampled points of C (A and B whole on the host)."""
    M, N = C_dev.shape
    rng = np.random.default_rng(seed)
    rows, cols = rng.integers(0, M, n_points), rng.integers(0, N, n_points)
    Cp, Rp = ogemm.gemm_ref_points(A, B, K, A.shape[1], B.shape[1], rows, cols)
    got = to_host(C_dev[torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()])
    ocheck.assert_gemm_close(got, Cp, Rp, what)


def free():
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("ca_layers", [1, 0])
def test_a_beyond_4gib(ca_layers):
    """A is 5.25 GB (40000 x 65600 bf16); rows from 32736 on start past 2^32."""
    M, N, K, P, lda = 40000, 256, 65536, 1024, 65600
    blk = draw(M, P, U, 9101)
    B = draw(K, N, U, 9102)
    dA = periodic_bf16(blk, K // P, lda)
    dB = sg().to_device_bf16(B)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    sg().sfc_gemm_ex(dA[:, :K], dB, C, ca_layers=ca_layers)
    torch.cuda.synchronize()
    r_cross = straddling_row(lda * 2, M)
    rows = sorted({0, 1, r_cross - 1, r_cross, r_cross + 1, 32767, 32768, M - 2, M - 1})
    A_rows = np.tile(blk[rows], (1, K // P))
    check_rows(C, rows, A_rows, B, N, K, f"A > 4 GiB, c={ca_layers}")
    del dA, dB, C
    free()


@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_c_beyond_4gib(out):
    """C is 5.2 GB (36000^2 f32) or 4.6 GB (48000^2 bf16), K = 100 (a tail
    inside the second 64-deep block)."""
    M = N = 36000 if out == "f32" else 48000
    K = 100
    A = draw(M, K, U, 9201)
    B = draw(K, N, U, 9202)
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    C = torch.full((M, N), float("nan"), dtype=dtype, device="cuda")
    sg().sfc_gemm_ex(sg().to_device_bf16(A), sg().to_device_bf16(B), C)
    torch.cuda.synchronize()
    esz = 4 if out == "f32" else 2
    r_cross = straddling_row(N * esz, M)
    rows = [0, r_cross, r_cross + 1, M - 1]
    check_rows(C, rows, A[rows], B, N, K, f"C > 4 GiB ({out}) rows")
    check_points(C, A, B, K, 8192, 9203, f"C > 4 GiB ({out}) points")
    # no NaN left anywhere (every element written)
    assert not torch.isnan(C).any().item()
    del C
    free()


def test_workspace_beyond_4gib():
    """Four layer copies of an 18000^2 f32 output: 5.2 GB of workspace, layer 3
    crossing 2^32; the reduction reads all four."""
    M = N = 18000
    K, c = 256, 4
    A = draw(M, K, U, 9301)
    B = draw(K, N, U, 9302)
    assert sg().sfc_gemm_ws_size(M, N, K, c) > GiB4
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(sg().sfc_gemm_ws_size(M, N, K, c) // 4, dtype=torch.float32, device="cuda")
    sg().sfc_gemm_ex(sg().to_device_bf16(A), sg().to_device_bf16(B), C, ca_layers=c, workspace=ws)
    torch.cuda.synchronize()
    # rows of layer 3 around byte offset 2^32 of the workspace
    r_cross = (GiB4 - 3 * M * N * 4) // (N * 4)
    rows = [0, r_cross, r_cross + 1, M - 1]
    check_rows(C, rows, A[rows], B, N, K, "workspace > 4 GiB rows")
    check_points(C, A, B, K, 8192, 9303, "workspace > 4 GiB points")
    # layer 3's own partial, straddling row: the oracle over its K slice (the
    # last of four 64-deep blocks)
    W3 = ws[3 * M * N:4 * M * N].view(M, N)
    Cr, R = ogemm.gemm_ref_rows(np.ascontiguousarray(A[[r_cross], 192:256]), B[192:256], N, 64, 64, N, M=1)
    ocheck.assert_gemm_close(to_host(W3[r_cross:r_cross + 1]), Cr, R, "layer 3 partial at 2^32")
    del C, ws, W3
    free()


def test_f8_a_beyond_4gib():
    """fp8 A of 5.25 GB (40000 x 131200 E4M3 bytes)."""
    M, N, K, P, lda = 40000, 256, 131072, 2048, 131200
    blk = draw_e4m3(M, P, ("normal", 0.0, 0.1), 9401)
    B = draw_e4m3(K, N, ("normal", 0.0, 0.1), 9402)
    dA = torch.full((M, lda), NAN_E4M3, dtype=torch.uint8, device="cuda")
    dA[:, :K] = sg().to_device_u8(blk).repeat(1, K // P)
    dB = sg().to_device_u8(B)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    sg().sfc_gemm_f8_ex(dA[:, :K], dB, C)
    torch.cuda.synchronize()
    r_cross = straddling_row(lda, M)
    rows = sorted({0, r_cross, r_cross + 1, M - 1})
    A_rows = of8.e4m3_to_bf16_bits(np.tile(blk[rows], (1, K // P)))
    check_rows(C, rows, A_rows, of8.e4m3_to_bf16_bits(B), N, K, "fp8 A > 4 GiB")
    del dA, dB, C
    free()


@pytest.mark.parametrize("which", ["lda", "ldb"])
def test_leading_dimension_limits(which):
    """lda = 2^20 - 8 and ldb = 2^22 - 8 take the 16-byte load path, 2^20 and
    2^22 the element path: both correct and bitwise equal."""
    M, N, K = 300, 264, 136
    A = draw(M, K, U, 9501)
    B = draw(K, N, U, 9502)
    Cr, R = ogemm.gemm_ref_rows(A, B, N, K, K, N, M=M)
    limit = (1 << 20) if which == "lda" else (1 << 22)
    outs = []
    for ld in (limit - 8, limit):
        dA = padded_bf16(A, ld) if which == "lda" else sg().to_device_bf16(A)
        dB = padded_bf16(B, ld) if which == "ldb" else sg().to_device_bf16(B)
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        sg().sfc_gemm_ex(dA[:, :K], dB[:, :N], C, tile="256x256")
        torch.cuda.synchronize()
        ocheck.assert_gemm_close(to_host(C), Cr, R, f"{which} = {ld}")
        outs.append(raw_bits(C))
        del dA, dB, C
    assert np.array_equal(outs[0], outs[1])
    free()


@pytest.mark.parametrize("which", ["lda", "ldb"])
def test_f8_leading_dimension_limits(which):
    """fp8: lda = 2^21 - 16 and ldb = 2^23 - 16 are the largest accepted."""
    M, N, K = 300, 272, 400
    A = draw_e4m3(M, K, ("normal", 0.0, 0.1), 9601)
    B = draw_e4m3(K, N, ("normal", 0.0, 0.1), 9602)
    Cr, R = ogemm.gemm_ref_rows(of8.e4m3_to_bf16_bits(A), of8.e4m3_to_bf16_bits(B), N, K, K, N, M=M)
    ld = (1 << 21) - 16 if which == "lda" else (1 << 23) - 16
    rows = M if which == "lda" else K
    t = torch.full((rows, ld), NAN_E4M3, dtype=torch.uint8, device="cuda")
    src = A if which == "lda" else B
    t[:, :src.shape[1]] = sg().to_device_u8(src)
    dA = t if which == "lda" else sg().to_device_u8(A)
    dB = t if which == "ldb" else sg().to_device_u8(B)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    sg().sfc_gemm_f8_ex(dA[:, :K], dB[:, :N], C)
    torch.cuda.synchronize()
    ocheck.assert_gemm_close(to_host(C), Cr, R, f"fp8 {which} = {ld}")
    del t, dA, dB, C
    free()
