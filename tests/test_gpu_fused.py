"""The fused reduction (sfc_gemm_fused_ex): the workgroup that completes a
block's layer copies sums them inside the GEMM launch.  Through the C ABI,
against the oracle:
  * each layer copy left in the workspace is the product over its own K range
    (fp64 oracle, the bar), and C is the ordered fp32 sum of those copies bit
    for bit (the oracle's reduction, Listing 1's final add-reduce), for fp32
    and bf16 output, vector and element store paths, ragged edges;
  * C meets the bar against the fp64 oracle;
  * the arrival counters are left at zero: calls in a row (different grids,
    different layer counts, on one stream without a wait between) all meet
    the same bar, and the fused and separate reductions give the same bits,
    also when the two alternate on one workspace (so that chiplet caches may
    hold the previous call's copies of it)."""
import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import ca as oca
from oracle import check as ocheck
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import draw
from gpu_util import raw_bits, sg, to_host, upload

pytestmark = pytest.mark.gpu


def oracle(A, B, M, N, K):
    return ogemm.gemm_ref_rows(A, B, N, K, K, N, M=M)


def layer_oracle(A, B, N, K, c, layer):
    k0, k1 = oca.k_slices(K, c, 64)[layer]
    return ogemm.gemm_ref_rows(np.ascontiguousarray(A[:, k0:k1]), np.ascontiguousarray(B[k0:k1]),
                               N, k1 - k0, k1 - k0, N, M=A.shape[0])


CASES = [
    # M, N, K, c, tile, out
    (260, 136, 1000, 2, "128x128", "f32"),
    (260, 136, 1000, 3, "128x128", "bf16"),
    (300, 520, 1100, 8, "256x256", "f32"),
    (513, 264, 2048, 16, "256x128", "bf16"),
    (200, 390, 900, 5, "128x256", "f32"),     # N % 4 != 0 ... 390 % 4 = 2: element path
    (129, 255, 700, 4, "128x128", "bf16"),    # odd N: element path, K tail
]


@pytest.mark.parametrize("M,N,K,c,tile,out", CASES)
def test_fused_copies_and_sum(M, N, K, c, tile, out):
    A = draw(M, K, ("normal", 0.0, 1.0), 9100 + M)
    B = draw(K, N, ("normal", 0.0, 1.0), 9200 + N)
    dA, dB = upload(A), upload(B)
    ce = oca.effective_layers(K, c, 64)
    ws_bytes = sg().sfc_gemm_ws_size(M, N, K, c)
    assert ws_bytes == ce * M * N * 4
    ws = torch.full((ws_bytes // 4,), float("nan"), dtype=torch.float32, device="cuda")
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    C = torch.full((M, N), float("nan"), dtype=dtype, device="cuda")
    sg().sfc_gemm_fused_ex(dA, dB, C, ca_layers=c, tile=tile, workspace=ws)
    torch.cuda.synchronize()
    W = ws.cpu().numpy().reshape(ce, M, N)
    for layer in range(ce):
        Cl, Rl = layer_oracle(A, B, N, K, c, layer)
        ocheck.assert_gemm_close(W[layer], Cl, Rl, f"layer {layer}")
    red = oca.reduce_layers_f32(W)
    if out == "f32":
        assert np.array_equal(raw_bits(C), red.view(np.uint32))
    else:
        assert np.array_equal(raw_bits(C), obf16.f32_to_bf16_rne(red))
    Cr, R = oracle(A, B, M, N, K)
    ocheck.assert_gemm_close(to_host(C), Cr, R, f"fused {M}x{N}x{K} c={c} {tile} {out}")


def test_fused_equals_separate_and_counters_reset():
    """Calls in a row on one stream, no wait between: different grids and layer
    counts reuse the stream's counters, which must be back at zero after each
    launch; every result equals the separate reduction's bits."""
    runs = [(700, 600, 3000, 4, "128x128"), (700, 600, 3000, 4, "128x128"), (300, 1000, 5000, 16, "256x256"),
            (1024, 1024, 8192, 8, "256x256"), (700, 600, 3000, 2, "256x128")] * 3
    ins = {}
    outs = []
    for i, (M, N, K, c, tile) in enumerate(runs):
        key = (M, N, K)
        if key not in ins:
            A = draw(M, K, ("uniform", -1.0, 1.0), 9300 + M)
            B = draw(K, N, ("uniform", -1.0, 1.0), 9400 + N)
            ins[key] = (A, B, upload(A), upload(B))
        _, _, dA, dB = ins[key]
        Cf = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        Cs = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        sg().sfc_gemm_fused_ex(dA, dB, Cf, ca_layers=c, tile=tile)
        sg().sfc_gemm_ex(dA, dB, Cs, ca_layers=c, tile=tile)
        outs.append((key, c, tile, Cf, Cs))
    torch.cuda.synchronize()
    for (M, N, K), c, tile, Cf, Cs in outs:
        A, B, _, _ = ins[(M, N, K)]
        assert np.array_equal(raw_bits(Cf), raw_bits(Cs)), (M, N, K, c, tile)
        Cr, R = oracle(A, B, M, N, K)
        ocheck.assert_gemm_close(to_host(Cf), Cr, R, f"fused {M}x{N}x{K} c={c} {tile}")


def test_fused_one_layer_and_auto():
    M, N, K = 256, 192, 8192
    A = draw(M, K, ("normal", 0.0, 1.0), 9501)
    B = draw(K, N, ("normal", 0.0, 1.0), 9502)
    dA, dB = upload(A), upload(B)
    Cr, R = oracle(A, B, M, N, K)
    for c in (1, 0):
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        sg().sfc_gemm_fused_ex(dA, dB, C, ca_layers=c)
        Cs = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        sg().sfc_gemm_ex(dA, dB, Cs, ca_layers=c)
        torch.cuda.synchronize()
        assert np.array_equal(raw_bits(C), raw_bits(Cs)), c
        ocheck.assert_gemm_close(to_host(C), Cr, R, f"fused c={c}")


def test_fused_integer_inputs_exact():
    M, N, K = 300, 264, 4096
    A = draw(M, K, ("int", -4, 4), 9601)
    B = draw(K, N, ("int", -4, 4), 9602)
    Cr, _ = oracle(A, B, M, N, K)
    for c, tile in ((3, "128x128"), (16, "256x256"), (7, "128x256")):
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        sg().sfc_gemm_fused_ex(upload(A), upload(B), C, ca_layers=c, tile=tile)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(C), Cr), (c, tile)
