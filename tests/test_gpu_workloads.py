"""The five measured workloads at full size, in the launch configuration the
benchmark times (tile shape, layer counts, curve order, interleaved
schedule), checked against the oracle on sampled elements: random points plus
whole rows and columns through the first, a middle and the last (ragged)
block."""
import numpy as np
import pytest
import torch

from oracle import check as ocheck
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import workloads
from gpu_util import sg, to_host, upload

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

WORKLOADS = {w.name: w for w in workloads()}


def sampled_check(A, B, C, M, N, K, seed, what):
    rng = np.random.default_rng(seed)
    rows = rng.integers(0, M, 4096)
    cols = rng.integers(0, N, 4096)
    Cp, Rp = ogemm.gemm_ref_points(A, B, K, K, N, rows, cols)
    ocheck.assert_gemm_close(C[rows, cols], Cp, Rp, what + " points")
    for r in sorted({0, min(M - 1, 127), min(M - 1, 128), M // 2, M - 1}):
        Cr, Rr = ogemm.gemm_ref_rows(A, B, N, K, K, N, row0=r, nrows=1)
        ocheck.assert_gemm_close(C[r:r + 1], Cr, Rr, f"{what} row {r}")
    for c in sorted({0, min(N - 1, 255), N // 2, N - 1}):
        rr = np.arange(M)
        Cc, Rc = ogemm.gemm_ref_points(A, B, K, K, N, rr, np.full(M, c))
        ocheck.assert_gemm_close(C[:, c], Cc, Rc, f"{what} col {c}")


def run(w, g, dA, dB, c, order="hilbert"):
    dtype = torch.float32 if g.out == "f32" else torch.bfloat16
    C = torch.full((g.M, g.N), float("nan"), dtype=dtype, device="cuda")
    sg().sfc_gemm_ex(dA, dB, C, ca_layers=c, tile=w.tile, order=order)
    torch.cuda.synchronize()
    return C


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_workload_full_size(name):
    w = WORKLOADS[name]
    for j, g in enumerate(w.gemms):
        A, B = g.operands()
        dA, dB = upload(A), upload(B)
        for c in w.ca_layers:
            print(f"[workload] {name} gemm {j} {g.M}x{g.N}x{g.K} c={c} tile={w.tile}", flush=True)
            C = to_host(run(w, g, dA, dB, c))
            assert np.isfinite(C).all()
            if g.M * g.N * g.K <= 512 ** 3:
                Cr, R = ogemm.gemm_ref_rows(A, B, g.N, g.K, g.K, g.N, M=g.M)
                ocheck.assert_gemm_close(C, Cr, R, name)
            else:
                sampled_check(A, B, C, g.M, g.N, g.K, 17 + j, f"{name} c={c}")
        del dA, dB
        torch.cuda.empty_cache()


def test_ragged_workload_order_invariance():
    w = WORKLOADS["ragged3000x7000x2048_f32out"]
    g = w.gemms[0]
    A, B = g.operands()
    dA, dB = upload(A), upload(B)
    a = run(w, g, dA, dB, 1, "hilbert")
    b = run(w, g, dA, dB, 1, "row_major")
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
