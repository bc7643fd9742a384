"""Special values and streams, through the C ABI: infinities and NaN in the
operands propagate as IEEE arithmetic says (inf * 0 = NaN, inf - inf = NaN),
element by element as the fp64 oracle gives them, for bf16 operands and for
E5M2 operands (the fp8 format with infinities), with one layer and with the
layer split; and GEMMs enqueued on two streams at once, with one layer and with
several (each stream with its own workspace), each meet the bar."""
import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import check as ocheck
from oracle import fp8 as of8
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import draw, draw_fp8
from gpu_util import sg, to_host, upload

pytestmark = pytest.mark.gpu

M, N, K = 64, 80, 160
# (row, k, kind) of the planted specials in A; column ZCOL of B is zero
PLANTS = [(3, 5, "+inf"), (10, 7, "-inf"), (20, 9, "nan"), (30, 1, "+inf"), (30, 2, "-inf"), (40, 150, "+inf")]
ZCOL = 11


def assert_same_specials(C, Cr, R, what):
    nan, nan_r = np.isnan(C), np.isnan(Cr)
    assert np.array_equal(nan, nan_r), f"{what}: NaN pattern differs"
    inf, inf_r = np.isinf(C), np.isinf(Cr)
    assert np.array_equal(inf, inf_r), f"{what}: infinity pattern differs"
    assert np.array_equal(np.sign(C[inf]), np.sign(Cr[inf_r])), f"{what}: infinity signs differ"
    fin = ~(nan | inf)
    assert fin.sum() > M * N // 2
    ocheck.assert_gemm_close(C[fin], Cr[fin], R[fin], f"{what} finite part")


def oracle(Ab, Bb):
    return ogemm.gemm_ref_rows(Ab, Bb, N, K, K, N, M=M)


@pytest.mark.parametrize("c,out", [(1, "f32"), (2, "f32"), (1, "bf16")])
def test_bf16_specials(c, out):
    A = draw(M, K, ("normal", 0.0, 1.0), 7101)
    B = draw(K, N, ("uniform", 0.5, 1.5), 7102)       # positive, no zeros
    B[:, ZCOL] = 0                                    # inf * 0 -> NaN in that column
    codes = {"+inf": 0x7F80, "-inf": 0xFF80, "nan": 0x7FC0}
    for r, k, kind in PLANTS:
        A[r, k] = codes[kind]
    Cr, R = oracle(A, B)
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    C = torch.zeros((M, N), dtype=dtype, device="cuda")
    sg().sfc_gemm_ex(upload(A), upload(B), C, ca_layers=c)
    torch.cuda.synchronize()
    if out == "bf16":
        Cr = obf16.bf16_to_f64(obf16.f32_to_bf16_rne(Cr.astype(np.float32)))
    assert_same_specials(to_host(C), Cr, R, f"bf16 specials c={c} {out}")


@pytest.mark.parametrize("c", [1, 2])
def test_e5m2_specials(c):
    A = draw_fp8(M, K, ("normal", 0.0, 1.0), 7201, fmt="e5m2")
    B = draw_fp8(K, N, ("uniform", 0.5, 1.5), 7202, fmt="e5m2")
    B[:, ZCOL] = 0
    codes = {"+inf": 0x7C, "-inf": 0xFC, "nan": 0x7F}
    for r, k, kind in PLANTS:
        A[r, k] = codes[kind]
    Cr, R = oracle(of8.e5m2_to_bf16_bits(A), of8.e5m2_to_bf16_bits(B))
    C = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    sg().sfc_gemm_f8_ex(sg().to_device_u8(A), sg().to_device_u8(B), C, ca_layers=c, a_format="e5m2",
                        b_format="e5m2")
    torch.cuda.synchronize()
    assert_same_specials(to_host(C), Cr, R, f"e5m2 specials c={c}")


def test_two_streams_at_once():
    """Two GEMMs (one layer each: no shared workspace) enqueued on two streams
    before either is waited for."""
    shapes = [(1000, 700, 900, "f32", 7301), (513, 1300, 640, "bf16", 7311)]
    ins, outs = [], []
    for Mx, Nx, Kx, out, seed in shapes:
        A = draw(Mx, Kx, ("uniform", -1.0, 1.0), seed)
        B = draw(Kx, Nx, ("uniform", -1.0, 1.0), seed + 1)
        dtype = torch.float32 if out == "f32" else torch.bfloat16
        ins.append((A, B, upload(A), upload(B)))
        outs.append(torch.full((Mx, Nx), float("nan"), dtype=dtype, device="cuda"))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for (A, B, dA, dB), C, s in zip(ins, outs, streams):
        sg().sfc_gemm_ex(dA, dB, C, stream=s)
    torch.cuda.synchronize()
    for (Mx, Nx, Kx, out, _), (A, B, _, _), C in zip(shapes, ins, outs):
        Cr, R = ogemm.gemm_ref_rows(A, B, Nx, Kx, Kx, Nx, M=Mx)
        if out == "bf16":
            Cr = obf16.bf16_to_f64(obf16.f32_to_bf16_rne(Cr.astype(np.float32)))
        ocheck.assert_gemm_close(to_host(C), Cr, R, f"stream GEMM {Mx}x{Nx}x{Kx}")


def test_two_streams_with_layers():
    """sfc_gemm with c = 2 and with SFC_CA_AUTO (layers chosen by the model,
    more than one on these K-dominant shapes), using the library's own
    workspace, enqueued on two default-priority streams before either is waited
    for; each stream also grows its workspace between its two calls.  Every
    result meets the bar against the oracle."""
    plan = [  # per stream: (M, N, K, ca_layers, seed), in enqueue order
        [(256, 192, 8192, 2, 7401), (320, 256, 16384, 0, 7411)],
        [(300, 200, 12288, 0, 7421), (512, 384, 6144, 2, 7431)],
    ]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    jobs = []
    for calls in plan:
        for Mx, Nx, Kx, c, seed in calls:
            A = draw(Mx, Kx, ("normal", 0.0, 1.0), seed)
            B = draw(Kx, Nx, ("normal", 0.0, 1.0), seed + 1)
            C = torch.full((Mx, Nx), float("nan"), dtype=torch.float32, device="cuda")
            jobs.append((Mx, Nx, Kx, c, A, B, upload(A), upload(B), C))
    torch.cuda.synchronize()
    k = 0
    for s, calls in zip(streams, plan):
        for _ in calls:
            Mx, Nx, Kx, c, _, _, dA, dB, C = jobs[k]
            sg().sfc_gemm(dA, dB, C, ca_layers=c, stream=s)
            k += 1
    torch.cuda.synchronize()
    for Mx, Nx, Kx, c, A, B, _, _, C in jobs:
        if c == 0:
            assert sg().sfc_gemm_plan(Mx, Nx, Kx, 0, "auto")["layers"] > 1
        Cr, R = ogemm.gemm_ref_rows(A, B, Nx, Kx, Kx, Nx, M=Mx)
        ocheck.assert_gemm_close(to_host(C), Cr, R, f"stream GEMM {Mx}x{Nx}x{Kx} c={c}")
