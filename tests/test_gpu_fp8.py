"""Parity of the fp8 (OCP E4M3) GEMM path (sfc_gemm_f8_ex, through the C ABI)
with the fp64 oracle over the decoded operands: ragged M, K tails inside a
128-deep block, several layer counts, both output types, both block shapes
(256x256 and 128x256, which give the same bits), exact integer inputs, the
bf16 output as RNE of the fp32 output, the model's choice of block shape, and
the argument checks."""
import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import check as ocheck
from oracle import fp8 as of8
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import NAN_E4M3, draw_e4m3, draw_fp8
from gpu_util import raw_bits, sg, to_host

pytestmark = pytest.mark.gpu


def up8(bits):
    return sg().to_device_u8(bits)


def ref(A8, B8, M, N, K):
    A = of8.e4m3_to_bf16_bits(A8[:, :K])
    B = of8.e4m3_to_bf16_bits(B8[:, :N])
    return ogemm.gemm_ref_rows(A, B, N, K, K, N, M=M)


def run8(A8, B8, M, N, K, out="f32", c=1, ldc=None, tile="auto"):
    ldc = N if ldc is None else ldc
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    Cfull = torch.full((M, ldc), float("nan"), dtype=dtype, device="cuda")
    dA, dB = up8(A8), up8(B8)
    sg().sfc_gemm_f8_ex(dA[:M, :K], dB[:K, :N], Cfull[:, :N], ca_layers=c, tile=tile)
    torch.cuda.synchronize()
    return Cfull


SHAPES = [(1, 16, 16), (7, 32, 48), (256, 256, 256), (300, 528, 400), (257, 512, 128), (513, 272, 1040),
          (130, 1024, 2064)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_ragged_shapes(M, N, K, out):
    A = draw_e4m3(M, K, ("normal", 0.0, 1.0), M + K)
    B = draw_e4m3(K, N, ("normal", 0.0, 1.0), N + K + 1)
    Cr, R = ref(A, B, M, N, K)
    for c in (1, 3):
        C = to_host(run8(A, B, M, N, K, out, c))
        ocheck.assert_gemm_close(C, Cr, R, f"fp8 {M}x{N}x{K} {out} c={c}")


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_ragged_shapes_128x256(M, N, K, out):
    """The 128x256 fp8 kernel (4 waves of 128x64, 8 MFMAs per 64-deep step)."""
    A = draw_e4m3(M, K, ("normal", 0.0, 1.0), 5 * M + K)
    B = draw_e4m3(K, N, ("normal", 0.0, 1.0), 5 * N + K + 1)
    Cr, R = ref(A, B, M, N, K)
    for c in (1, 3):
        C = to_host(run8(A, B, M, N, K, out, c, tile="128x256"))
        ocheck.assert_gemm_close(C, Cr, R, f"fp8 128x256 {M}x{N}x{K} {out} c={c}")


def test_block_shapes_give_the_same_bits():
    """Each output element takes the same MFMA products in the same K order on
    either block shape, so 128x256 and 256x256 blocks give identical bits (one
    layer), here on a grid with ragged edges in both directions."""
    M, N, K = 700, 912, 1296
    A = draw_e4m3(M, K, ("normal", 0.0, 1.0), 8801)
    B = draw_e4m3(K, N, ("normal", 0.0, 1.0), 8802)
    for out in ("f32", "bf16"):
        Cw = run8(A, B, M, N, K, out, tile="256x256")
        Cn = run8(A, B, M, N, K, out, tile="128x256")
        assert np.array_equal(raw_bits(Cw), raw_bits(Cn)), out


@pytest.mark.parametrize("M,N,K,c", [(8192, 640, 4096, 1), (1536, 2048, 1024, 1), (1024, 1024, 16384, 0),
                                     (300, 272, 1040, 0)])
def test_auto_block_shape_follows_the_model(M, N, K, c):
    """SFC_TILE_AUTO on fp8 operands: the block shape and layer count of the
    oracle's model over the two fp8 block shapes for the equivalent bf16
    problem (K' = 64*ceil(K/128)), at the fp8 kernels' occupancy."""
    from oracle import model as omodel
    plan = sg().sfc_gemm_f8_plan(M, N, K, c, "auto")
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    occ = {(128, 128): 1, (256, 128): 1,
           (128, 256): sg().sfc_gemm_f8_plan(8192, 8192, 128, 1, "128x256")["per_cu"],
           (256, 256): sg().sfc_gemm_f8_plan(8192, 8192, 128, 1, "256x256")["per_cu"]}
    k_eq = 64 * -(-K // 128)
    picks = [omodel.choose(M, N, k_eq, 4, cus, occ, shape=s, layers=c) for s in ((256, 256), (128, 256))]
    best = picks[1] if picks[1][2] < picks[0][2] else picks[0]
    assert (plan["BM"], plan["BN"]) == best[0]
    assert plan["layers"] == min(best[1], -(-K // 128))


@pytest.mark.parametrize("tile", ["auto", "256x256", "128x256"])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_k_zero_writes_zeros(tile, out):
    M, N = 70, 96
    A = np.zeros((M, 16), np.uint8)
    B = np.zeros((16, N), np.uint8)
    for c in (1, 0):
        C = to_host(run8(A, B, M, N, 0, out, c, tile=tile))
        assert (C == 0).all(), (tile, out, c)


@pytest.mark.parametrize("c", [1, 2, 5])
def test_integer_inputs_exact(c):
    M, N, K = 300, 272, 1040
    A = draw_e4m3(M, K, ("int", -4, 4), 31)
    B = draw_e4m3(K, N, ("int", -4, 4), 32)
    Ai = of8.e4m3_to_f64(A).astype(np.int64)
    Bi = of8.e4m3_to_f64(B).astype(np.int64)
    for tile in ("256x256", "128x256"):
        C = to_host(run8(A, B, M, N, K, "f32", c, tile=tile))
        assert np.array_equal(C, (Ai @ Bi).astype(np.float64)), tile


def test_bf16_output_is_rne_of_f32_output_and_padding_untouched():
    M, N, K = 333, 528, 656
    A = draw_e4m3(M, K, ("normal", 0.0, 1.0), 41)
    B = draw_e4m3(K, N, ("normal", 0.0, 1.0), 42)
    C32 = run8(A, B, M, N, K, "f32", ldc=544)
    C16 = run8(A, B, M, N, K, "bf16", ldc=544)
    want = obf16.f32_to_bf16_rne(C32[:, :N].contiguous().cpu().numpy())
    assert np.array_equal(raw_bits(C16[:, :N].contiguous()), want)
    assert np.isnan(to_host(C32)[:, N:]).all() and np.isnan(to_host(C16)[:, N:]).all()


def test_lda_ldb_padding_is_never_read():
    M, N, K = 200, 256, 384
    A = draw_e4m3(M, K, ("uniform", -1.0, 1.0), 51, ld=400)   # NaN codes beyond K
    B = draw_e4m3(K, N, ("uniform", -1.0, 1.0), 52, ld=272)   # NaN codes beyond N
    dA, dB = up8(A), up8(B)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    sg().sfc_gemm_f8_ex(dA[:, :K], dB[:, :N], C)
    torch.cuda.synchronize()
    Cr, R = ref(A, B, M, N, K)
    ocheck.assert_gemm_close(to_host(C), Cr, R, "fp8 padded operands")


def test_unsupported_arguments_are_rejected():
    A = up8(np.zeros((64, 48), np.uint8))
    B = up8(np.zeros((48, 64), np.uint8))
    C = torch.zeros((64, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(sg().SfcError) as e:
        sg().sfc_gemm_f8_ex(A[:, :40], B[:40, :], C)          # K not a multiple of 16
    assert e.value.code == sg().SFC_ERR_UNSUPPORTED
    with pytest.raises(sg().SfcError) as e:
        sg().sfc_gemm_f8_ex(A, B, C, tile="128x128")
    assert e.value.code == sg().SFC_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert (C == 0).all()


@pytest.mark.slow
def test_full_size_8192_sampled():
    M = N = K = 8192
    A = draw_e4m3(M, K, ("normal", 0.0, 1.0), 61)
    B = draw_e4m3(K, N, ("normal", 0.0, 1.0), 62)
    C = to_host(run8(A, B, M, N, K, "bf16"))
    Ab, Bb = of8.e4m3_to_bf16_bits(A), of8.e4m3_to_bf16_bits(B)
    rng = np.random.default_rng(63)
    rows, cols = rng.integers(0, M, 2048), rng.integers(0, N, 2048)
    Cp, Rp = ogemm.gemm_ref_points(Ab, Bb, K, K, N, rows, cols)
    ocheck.assert_gemm_close(C[rows, cols], Cp, Rp, "fp8 8192^3 points")
    for r in (0, 4095, 8191):
        Cr, Rr = ogemm.gemm_ref_rows(Ab, Bb, N, K, K, N, row0=r, nrows=1)
        ocheck.assert_gemm_close(C[r:r + 1], Cr, Rr, f"fp8 8192^3 row {r}")


@pytest.mark.parametrize("M,N,K", [(1024, 1024, 16384), (512, 768, 4096), (300, 272, 1040)])
def test_auto_layers(M, N, K):
    """SFC_CA_AUTO on fp8 operands: the model's layer count for the equivalent
    bf16 problem (K' = 64*ceil(K/128), 256x256 blocks); the result meets the
    bar whatever the count."""
    A = draw_e4m3(M, K, ("normal", 0.0, 0.1), 71 + M)
    B = draw_e4m3(K, N, ("normal", 0.0, 0.1), 72 + N)
    Cr, R = ref(A, B, M, N, K)
    C = to_host(run8(A, B, M, N, K, "f32", c=0))
    ocheck.assert_gemm_close(C, Cr, R, f"fp8 auto {M}x{N}x{K}")
    # the count the model picks for the equivalent bf16 problem is a K-dominant
    # choice with layers for the first shape
    pick = sg().sfc_gemm_model(M, N, 64 * -(-K // 128), out="f32", tile="256x256")
    if (M, N, K) == (1024, 1024, 16384):
        assert pick["layers"] > 1


# ---- OCP E5M2 and mixed formats (sfc_gemm_f8_fmt_ex) ---------------------------

FMT_PAIRS = [("e5m2", "e5m2"), ("e4m3", "e5m2"), ("e5m2", "e4m3")]


def ref_fmt(A8, B8, M, N, K, fa, fb):
    A = of8.to_bf16_bits(A8[:, :K], fa)
    B = of8.to_bf16_bits(B8[:, :N], fb)
    return ogemm.gemm_ref_rows(A, B, N, K, K, N, M=M)


@pytest.mark.parametrize("fa,fb", FMT_PAIRS)
@pytest.mark.parametrize("M,N,K,c,out", [(300, 528, 400, 1, "f32"), (513, 272, 1040, 3, "bf16"),
                                         (256, 256, 256, 2, "f32"), (7, 32, 48, 1, "bf16")])
def test_formats_against_oracle(fa, fb, M, N, K, c, out):
    seed = 9700 + M + 3 * K + (fa == "e5m2") + 2 * (fb == "e5m2")
    A = draw_fp8(M, K, ("normal", 0.0, 1.0), seed, fmt=fa)
    B = draw_fp8(K, N, ("normal", 0.0, 1.0), seed + 1, fmt=fb)
    Cr, R = ref_fmt(A, B, M, N, K, fa, fb)
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    for tile in ("256x256", "128x256"):
        C = torch.full((M, N), float("nan"), dtype=dtype, device="cuda")
        sg().sfc_gemm_f8_ex(up8(A), up8(B), C, ca_layers=c, tile=tile, a_format=fa, b_format=fb)
        torch.cuda.synchronize()
        ocheck.assert_gemm_close(to_host(C), Cr, R, f"{fa} x {fb} {M}x{N}x{K} c={c} {out} {tile}")


@pytest.mark.parametrize("fa,fb", FMT_PAIRS)
def test_formats_integers_exact(fa, fb):
    """Integers in [-8, 8] are exact in both formats; sums stay below 2^24."""
    M, N, K = 260, 304, 1024
    A = draw_fp8(M, K, ("int", -8, 8), 9801, fmt=fa)
    B = draw_fp8(K, N, ("int", -8, 8), 9802, fmt=fb)
    Cr, _ = ref_fmt(A, B, M, N, K, fa, fb)
    for c in (1, 4):
        for tile in ("256x256", "128x256"):
            C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
            sg().sfc_gemm_f8_ex(up8(A), up8(B), C, ca_layers=c, tile=tile, a_format=fa, b_format=fb)
            torch.cuda.synchronize()
            assert np.array_equal(to_host(C), Cr), f"{fa} x {fb} c={c} {tile}"


def test_format_codes_select_the_format():
    """The same bytes read as E4M3 and as E5M2 give the two oracles' results
    (a swapped or ignored format code fails one of them)."""
    M, N, K = 256, 256, 512
    A = draw_fp8(M, K, ("normal", 0.0, 0.5), 9901, fmt="e4m3")
    B = draw_fp8(K, N, ("normal", 0.0, 0.5), 9902, fmt="e4m3")
    # reinterpret B's bytes in the other format too (codes 0x7C-0x7F and
    # 0xFC-0xFF are infinities or NaN in E5M2: clear them to keep values finite)
    B5 = np.where((B & 0x7C) == 0x7C, B & 0x83, B).astype(np.uint8)
    for fb, Bx in (("e4m3", B5), ("e5m2", B5)):
        Cr, R = ref_fmt(A, Bx, M, N, K, "e4m3", fb)
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        sg().sfc_gemm_f8_ex(up8(A), up8(Bx), C, a_format="e4m3", b_format=fb)
        torch.cuda.synchronize()
        ocheck.assert_gemm_close(to_host(C), Cr, R, f"bytes read as {fb}")
