"""Parity of the HIP GEMM (through the C ABI) with the fp64 oracle on seeded
inputs: ragged shapes across several tiles, both load paths, every output
type, the CA layer split and its reduction, and the invariances the design
promises (tile order, schedule, run to run)."""
import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import ca as oca
from oracle import check as ocheck
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import draw
from gpu_util import raw_bits, run_gemm, sg, to_host, upload

pytestmark = pytest.mark.gpu

U = ("uniform", -1.0, 1.0)
TILES = ["128x128", "256x128", "128x256", "256x256"]


def oracle(A, B, M, N, K):
    return ogemm.gemm_ref_rows(A, B, N, K, A.shape[1], B.shape[1], M=M)


def operands(M, N, K, seed, dist=U, lda=None, ldb=None):
    return draw(M, K, dist, seed, lda), draw(K, N, dist, seed + 1, ldb)


SHAPES = [(1, 1, 1), (7, 7, 7), (31, 127, 129), (128, 128, 128), (129, 255, 300), (255, 129, 64),
          (300, 1000, 127), (1000, 300, 1000), (127, 31, 1000), (1, 1000, 255), (1000, 1, 31),
          (256, 256, 256), (257, 513, 200), (520, 264, 136)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("tile", ["auto", "128x128", "256x256"])
def test_ragged_shapes_f32(M, N, K, tile):
    A, B = operands(M, N, K, 100 + M + N + K)
    C = run_gemm(A, B, M, N, K, tile=tile)
    Cr, R = oracle(A, B, M, N, K)
    ocheck.assert_gemm_close(C, Cr, R, f"{M}x{N}x{K} {tile}")


@pytest.mark.parametrize("M,N,K", [(129, 255, 300), (300, 1000, 127), (520, 264, 136)])
@pytest.mark.parametrize("tile", TILES)
def test_ragged_shapes_bf16_out(M, N, K, tile):
    A, B = operands(M, N, K, 200 + M)
    C = run_gemm(A, B, M, N, K, out="bf16", tile=tile)
    Cr, R = oracle(A, B, M, N, K)
    ocheck.assert_gemm_close(C, Cr, R, f"bf16 {M}x{N}x{K} {tile}")


# K depths that give the fast path 1 .. 5 blocks per task, with and without a
# last block that runs past K (K % 64 in {8, 24, 32, 40}), split over 1-3 layers.
@pytest.mark.parametrize("K", [8, 24, 40, 64, 72, 96, 120, 136, 160, 200, 296, 320])
@pytest.mark.parametrize("tile", TILES)
def test_k_depths_and_tails_fast_path(K, tile):
    M, N = 264, 520
    A, B = operands(M, N, K, 700 + K)
    Cr, R = oracle(A, B, M, N, K)
    for c in (1, 2, 3):
        C = run_gemm(A, B, M, N, K, tile=tile, ca_layers=c)
        ocheck.assert_gemm_close(C, Cr, R, f"K={K} {tile} c={c}")


@pytest.mark.parametrize("tile", TILES)
def test_vector_and_element_loads_agree_bitwise(tile):
    # lda, ldb multiples of 8 take 128-bit loads; odd ones take element loads.
    M, N, K = 300, 264, 520
    A8, B8 = operands(M, N, K, 300, lda=528, ldb=272)
    A7 = np.ascontiguousarray(np.pad(A8[:, :K], ((0, 0), (0, 3)), constant_values=0x7FC0))
    B7 = np.ascontiguousarray(np.pad(B8[:, :N], ((0, 0), (0, 5)), constant_values=0x7FC0))
    c8 = run_gemm(A8, B8, M, N, K, tile=tile)
    c7 = run_gemm(A7, B7, M, N, K, tile=tile)
    assert np.array_equal(c8, c7)
    Cr, R = oracle(A8, B8, M, N, K)
    ocheck.assert_gemm_close(c8[:, :N], Cr, R)


@pytest.mark.parametrize("c", [1, 2, 3, 4, 8])
@pytest.mark.parametrize("tile", ["128x128", "256x256"])
def test_integer_inputs_exact_for_every_layer_count(c, tile):
    M, N, K = 300, 200, 1000
    A, B = operands(M, N, K, 400, dist=("int", -4, 4))
    C = run_gemm(A, B, M, N, K, ca_layers=c, tile=tile)
    exact = obf16.bf16_to_f64(A).astype(np.int64) @ obf16.bf16_to_f64(B).astype(np.int64)
    assert np.array_equal(C, exact.astype(np.float64))


def test_identity_and_outer_product():
    M, K = 200, 136
    A = draw(M, K, U, 500)
    I = np.zeros((K, K), np.uint16)
    I[np.arange(K), np.arange(K)] = 0x3F80
    assert np.array_equal(run_gemm(A, I, M, K, K), obf16.bf16_to_f64(A))
    a = draw(130, 1, U, 501)
    b = draw(1, 70, U, 502)
    assert np.array_equal(run_gemm(a, b, 130, 70, 1),
                          np.outer(obf16.bf16_to_f64(a[:, 0]), obf16.bf16_to_f64(b[0])))


@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_k_zero_writes_zeros(out):
    M, N = 70, 90
    A = np.zeros((M, 1), np.uint16)
    B = np.zeros((1, N), np.uint16)
    C = run_gemm(A, B, M, N, 0, out=out)
    assert (C == 0).all()


def test_padding_is_never_written_or_read():
    M, N, K = 150, 130, 200
    A, B = operands(M, N, K, 600, lda=216, ldb=136)       # NaN in the ld padding
    C = run_gemm(A, B, M, N, K, ldc=144)
    assert np.isnan(C[:, N:]).all()
    assert np.isfinite(C[:, :N]).all()
    Cr, R = oracle(A, B, M, N, K)
    ocheck.assert_gemm_close(C[:, :N], Cr, R)


@pytest.mark.parametrize("tile", ["128x128", "256x128", "256x256"])
def test_order_and_schedule_never_change_bits(tile):
    M, N, K = 1000, 1300, 300
    A, B = operands(M, N, K, 700)
    ref = run_gemm(A, B, M, N, K, tile=tile)
    for order in ("hilbert", "row_major"):
        for sched in ("interleaved", "block", "interleaved_plain"):
            assert np.array_equal(run_gemm(A, B, M, N, K, tile=tile, order=order, sched=sched), ref)
    assert np.array_equal(run_gemm(A, B, M, N, K, tile=tile), ref)   # run to run


@pytest.mark.parametrize("c", [1, 3])
def test_bf16_output_is_rne_of_f32_output(c):
    M, N, K = 333, 515, 600
    A, B = operands(M, N, K, 800, dist=("normal", 0, 1))
    dA, dB = upload(A), upload(B)
    C32 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    C16 = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    sg().sfc_gemm_ex(dA, dB, C32, ca_layers=c, tile="256x256")
    sg().sfc_gemm_ex(dA, dB, C16, ca_layers=c, tile="256x256")
    torch.cuda.synchronize()
    want = obf16.f32_to_bf16_rne(C32.cpu().numpy())
    assert np.array_equal(raw_bits(C16), want)


@pytest.mark.parametrize("c", [2, 3, 8])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_layer_copies_and_their_reduction(c, out):
    M, N, K = 260, 136, 1000
    A, B = operands(M, N, K, 900 + c, dist=("normal", 0, 1))
    dA, dB = upload(A), upload(B)
    ws_bytes = sg().sfc_gemm_ws_size(M, N, K, c)
    ce = oca.effective_layers(K, c, 64)
    assert ws_bytes == ce * M * N * 4
    ws = torch.full((ws_bytes // 4,), float("nan"), dtype=torch.float32, device="cuda")
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    C = torch.empty((M, N), dtype=dtype, device="cuda")
    sg().sfc_gemm_ex(dA, dB, C, ca_layers=c, tile="128x128", workspace=ws)
    torch.cuda.synchronize()
    W = ws.cpu().numpy().reshape(ce, M, N)
    # each layer is the product over its own K range
    for layer, (k0, k1) in enumerate(oca.k_slices(K, c, 64)):
        Cl, Rl = ogemm.gemm_ref_rows(np.ascontiguousarray(A[:, k0:k1]), np.ascontiguousarray(B[k0:k1]),
                                     N, k1 - k0, k1 - k0, N, M=M)
        ocheck.assert_gemm_close(W[layer], Cl, Rl, f"layer {layer}")
    # the reduction is the ordered fp32 sum, bit for bit
    red = oca.reduce_layers_f32(W)
    if out == "f32":
        assert np.array_equal(raw_bits(C), red.view(np.uint32))
    else:
        assert np.array_equal(raw_bits(C), obf16.f32_to_bf16_rne(red))
    Cr, R = oracle(A, B, M, N, K)
    ocheck.assert_gemm_close(to_host(C), Cr, R)


def test_small_workspace_rejected_and_c_untouched():
    M, N, K = 64, 64, 256
    A, B = operands(M, N, K, 1000)
    C = torch.full((M, N), 7.0, device="cuda")
    ws = torch.empty(10, dtype=torch.float32, device="cuda")
    with pytest.raises(sg().SfcError) as e:
        sg().sfc_gemm_ex(upload(A), upload(B), C, ca_layers=2, workspace=ws)
    assert e.value.code == sg().SFC_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (C.cpu() == 7.0).all()


def test_plain_entry_points():
    M, N, K = 300, 200, 500
    A, B = operands(M, N, K, 1100)
    dA, dB = upload(A), upload(B)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    sg().sfc_gemm(dA, dB, C, ca_layers=2)
    C16 = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    sg().sfc_gemm_bf16out(dA, dB, C16)
    torch.cuda.synchronize()
    Cr, R = oracle(A, B, M, N, K)
    ocheck.assert_gemm_close(to_host(C), Cr, R)
    ocheck.assert_gemm_close(to_host(C16), Cr, R)


def test_plan_reports_grid():
    p = sg().sfc_gemm_plan(3000, 7000, 2048, 1, "128x128")
    assert (p["BM"], p["BN"], p["gm"], p["gn"], p["layers"]) == (128, 128, 24, 55, 1)
    p = sg().sfc_gemm_plan(1024, 1024, 65536, 4, "128x128")
    assert (p["gm"], p["gn"], p["layers"]) == (8, 8, 4)
    assert p["workgroups"] == 256


def test_mfma_probe_runs():
    r = sg().sfc_probe_mfma(True, 2000)
    c = sg().sfc_probe_mfma(False, 2000)
    for v in (r, c):
        assert 100.0 < v["tflops"] < 3000.0 and 500.0 < v["mhz"] < 3000.0


@pytest.mark.parametrize("M,N,K,out", [(256, 192, 8192, "f32"), (300, 520, 4104, "bf16"), (64, 64, 20000, "f32")])
def test_auto_layers_match_oracle(M, N, K, out):
    """SFC_CA_AUTO: the model's block shape and layer count (row f1), checked
    against the fp64 oracle; on these K-dominant shapes it picks layers."""
    A, B = operands(M, N, K, 700 + M)
    C = run_gemm(A, B, M, N, K, out=out, ca_layers=0)
    Cr, R = oracle(A, B, M, N, K)
    ocheck.assert_gemm_close(C, Cr, R, f"auto {M}x{N}x{K} {out}")
    plan = sg().sfc_gemm_plan(M, N, K, 0, "auto")
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    # the model weighs the block shapes at their full-grid occupancy (a grid of
    # at most one 128x128 block per CU runs a one-per-CU kernel instead)
    occ = tuple(sg().sfc_gemm_plan(8192, 8192, 64, 1, t)["per_cu"] for t in TILES)
    model = sg().sfc_gemm_model(M, N, K, out="f32", ca_layers=0, num_cus=cus, occupancy=occ)
    assert (f"{plan['BM']}x{plan['BN']}", plan["layers"]) == (model["tile"], model["layers"])
    assert plan["layers"] > 1


@pytest.mark.parametrize("tile", TILES)
def test_bf16_store_paths_by_alignment(tile):
    """The bf16 epilogue has three store paths: 16-byte stores of paired
    fragments (C 16-byte aligned, ldc a multiple of 8), 8-byte stores (8-byte
    aligned, ldc a multiple of 4) and element stores (anything else).  Each must
    give the RNE of the fp32 result bit for bit and leave the padding alone."""
    M, N, K = 300, 520, 200
    A, B = operands(M, N, K, 1200, dist=("normal", 0, 1))
    dA, dB = upload(A), upload(B)
    C32 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    sg().sfc_gemm_ex(dA, dB, C32, tile=tile)
    torch.cuda.synchronize()
    want = obf16.f32_to_bf16_rne(C32.cpu().numpy())
    for offset, ldc in ((0, 520), (4, 524), (1, 523)):
        buf = torch.full((offset + M * ldc,), float("nan"), dtype=torch.bfloat16, device="cuda")
        C = buf[offset:].view(M, ldc)[:, :N]
        sg().sfc_gemm_ex(dA, dB, C, tile=tile)
        torch.cuda.synchronize()
        full = raw_bits(buf[offset:].view(M, ldc))
        assert np.array_equal(full[:, :N], want), (tile, offset, ldc)
        pad = to_host(buf[offset:].view(M, ldc))[:, N:]
        assert np.isnan(pad).all(), (tile, offset, ldc)
        assert np.isnan(to_host(buf[:offset])).all()


@pytest.mark.parametrize("K,out", [(2048, "f32"), (2000, "bf16")])
def test_deep_ring_matches_two_per_cu_kernel(K, out):
    """128x128 grids of at most one block per CU run the 4-deep ring kernel (one
    workgroup per CU), larger ones the 2-deep ring (two per CU).  The two run the
    same MFMA sequence per element, so the top-left 1024x1024 of a 4096x4096
    product (1024 blocks: 2-deep) equals the 1024x1024 product of the same rows
    and columns (64 blocks: 4-deep) bit for bit; both meet the bar on sampled
    rows.  K = 2000 ends in a masked block."""
    Mb, Ms = 4096, 1024
    A = draw(Mb, K, U, 1500 + K)
    B = draw(K, Mb, U, 1501 + K)
    dA, dB = upload(A), upload(B)
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    Cb = torch.full((Mb, Mb), float("nan"), dtype=dtype, device="cuda")
    Cs = torch.full((Ms, Ms), float("nan"), dtype=dtype, device="cuda")
    sg().sfc_gemm_ex(dA, dB, Cb, tile="128x128")
    sg().sfc_gemm_ex(dA[:Ms], dB[:, :Ms].contiguous(), Cs, tile="128x128")
    torch.cuda.synchronize()
    assert sg().sfc_gemm_plan(Ms, Ms, K, 1, "128x128")["per_cu"] == 1
    assert sg().sfc_gemm_plan(Mb, Mb, K, 1, "128x128")["per_cu"] == 2
    assert np.array_equal(raw_bits(Cb)[:Ms, :Ms], raw_bits(Cs))
    rows = [0, 127, 128, 640, 1023, 1024, 2047, 4095]
    Cr, R = ogemm.gemm_ref_rows(np.ascontiguousarray(A[rows]), B, Mb, K, K, Mb, M=len(rows))
    if out == "bf16":
        Cr = obf16.bf16_to_f64(obf16.f32_to_bf16_rne(Cr.astype(np.float32)))
    ocheck.assert_gemm_close(to_host(Cb)[rows], Cr, R, f"128x128 two per CU K={K} {out}")
    small = [r for r in rows if r < Ms]
    ocheck.assert_gemm_close(to_host(Cs)[small], Cr[:len(small), :Ms], R[:len(small), :Ms],
                             f"128x128 deep ring K={K} {out}")
