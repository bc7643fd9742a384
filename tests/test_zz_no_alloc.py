"""sfc_gemm_noalloc_ex (the entry point for callers that cannot allocate),
through the C ABI: two calls in a row, the second on a smaller problem, each
give the same bits as sfc_gemm_ex on the same arguments and meet the bar
against the fp64 oracle (on sampled rows for the large shapes).  Cases: layer
copies in the static workspace (a count the model picks, and a fixed one),
one layer, and the half-height strip that uses the second curve table."""
import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import check as ocheck
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import draw
from gpu_util import raw_bits, sg, to_host, upload

pytestmark = pytest.mark.gpu

SEQUENCES = [
    # two calls: (M, N, K, ca_layers, tile, out), the second smaller than the first
    [(1024, 1024, 16384, 0, "auto", "f32"), (300, 520, 4104, 3, "128x128", "bf16")],
    [(4096, 14336, 1024, 1, "auto", "bf16"), (2000, 3000, 512, 1, "auto", "f32")],
    [(2048, 2048, 8192, 4, "256x256", "f32"), (513, 264, 2048, 2, "auto", "f32")],
]


def sampled_rows(M):
    return sorted({0, 1, 127, 128, 255, 256, M // 2, M - 2, M - 1} & set(range(M)))


def check_against_oracle(A, B, C, M, N, K, out, what):
    rows = sampled_rows(M) if M * N * K > (1 << 31) else list(range(M))
    Cr, R = ogemm.gemm_ref_rows(np.ascontiguousarray(A[rows]), B, N, K, K, N, M=len(rows))
    if out == "bf16":
        Cr = obf16.bf16_to_f64(obf16.f32_to_bf16_rne(Cr.astype(np.float32)))
    ocheck.assert_gemm_close(to_host(C)[rows], Cr, R, what)


@pytest.mark.parametrize("seq", range(len(SEQUENCES)))
def test_noalloc_matches_ex_two_calls(seq):
    calls = SEQUENCES[seq]
    assert calls[1][0] * calls[1][1] < calls[0][0] * calls[0][1]
    for i, (M, N, K, c, tile, out) in enumerate(calls):
        A = draw(M, K, ("normal", 0.0, 1.0), 9700 + 10 * seq + i)
        B = draw(K, N, ("normal", 0.0, 1.0), 9800 + 10 * seq + i)
        dA, dB = upload(A), upload(B)
        dtype = torch.float32 if out == "f32" else torch.bfloat16
        Cn = torch.full((M, N), float("nan"), dtype=dtype, device="cuda")
        Ce = torch.full((M, N), float("nan"), dtype=dtype, device="cuda")
        sg().sfc_gemm_noalloc_ex(dA, dB, Cn, ca_layers=c, tile=tile)
        sg().sfc_gemm_ex(dA, dB, Ce, ca_layers=c, tile=tile)
        torch.cuda.synchronize()
        what = f"noalloc call {i} {M}x{N}x{K} c={c} {tile} {out}"
        assert np.array_equal(raw_bits(Cn), raw_bits(Ce)), what
        check_against_oracle(A, B, Cn, M, N, K, out, what)
    # the plan of the first sequence uses layer copies, the second a strip
    if seq == 0:
        assert sg().sfc_gemm_plan(1024, 1024, 16384, 0, "auto")["layers"] > 1


def test_noalloc_rejects_and_leaves_c_untouched():
    M, N, K = 2049, 4096, 128
    A = upload(draw(M, K, ("uniform", -1.0, 1.0), 9901))
    B = upload(draw(K, N, ("uniform", -1.0, 1.0), 9902))
    C = torch.full((M, N), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(sg().SfcError) as e:
        sg().sfc_gemm_noalloc_ex(A, B, C, ca_layers=2)
    assert e.value.code == sg().SFC_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (C == 7.0).all().item()
