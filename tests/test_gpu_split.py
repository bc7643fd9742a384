"""When the library picks the block shape (SFC_TILE_AUTO), a partial last
round of 256-row blocks may go to a strip of half-height blocks in a second
launch.  The result is bitwise that of the single launch with the chosen
block shape, and meets the bar against the oracle on sampled points and whole
rows, on both sides of the strip boundary."""
import numpy as np
import pytest
import torch

from oracle import check as ocheck
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import draw
from gpu_util import sg, to_host, upload

pytestmark = pytest.mark.gpu

U = ("uniform", -1.0, 1.0)


def split_expected(M, N, K):
    """(tile name, strip width in block columns) when the split applies, else None."""
    pl = sg().sfc_gemm_plan(M, N, K, 1, "auto")
    if pl["layers"] != 1 or pl["BM"] != 256:
        return None
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    T, S = pl["gm"] * pl["gn"], cus * pl["per_cu"]
    r = T % S
    if T <= S or r == 0 or 2 * r > S:
        return None
    w = -(-r // pl["gm"])
    half_rows = -(-M // 128)
    if w >= pl["gn"] or half_rows * w > S:
        return None
    return f"{pl['BM']}x{pl['BN']}", w, pl["BN"]


@pytest.mark.parametrize("M,N,K,out,seed", [(4096, 14336, 4096, "bf16", 8101), (4000, 14000, 4096, "f32", 8201),
                                            (4000, 14000, 1000, "bf16", 8301), (4096, 14336, 2048, "f32", 8401)])
def test_strip_matches_single_launch(M, N, K, out, seed):
    exp = split_expected(M, N, K)
    if exp is None:
        pytest.skip("the split does not apply to this shape on this device")
    tile, w, bn = exp
    A = draw(M, K, U, seed)
    B = draw(K, N, U, seed + 1)
    dA, dB = upload(A), upload(B)
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    Ca = torch.full((M, N), float("nan"), dtype=dtype, device="cuda")
    Cb = torch.full((M, N), float("nan"), dtype=dtype, device="cuda")
    sg().sfc_gemm_ex(dA, dB, Ca, tile="auto")
    sg().sfc_gemm_ex(dA, dB, Cb, tile=tile)
    torch.cuda.synchronize()
    assert not torch.isnan(Ca).any().item()
    iview = torch.int32 if out == "f32" else torch.int16
    assert torch.equal(Ca.view(iview), Cb.view(iview))
    n1 = (-(-N // bn) - w) * bn                   # first column of the strip
    rng = np.random.default_rng(seed + 2)
    rows = rng.integers(0, M, 4096)
    cols = np.concatenate([rng.integers(0, n1, 2048), rng.integers(n1, N, 2048)])
    Cp, Rp = ogemm.gemm_ref_points(A, B, K, K, N, rows, cols)
    got = to_host(Ca[torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()])
    ocheck.assert_gemm_close(got, Cp, Rp, f"split {M}x{N}x{K} points")
    for r in (0, M - 1):
        Cr, Rr = ogemm.gemm_ref_rows(A, B, N, K, K, N, row0=r, nrows=1)
        ocheck.assert_gemm_close(to_host(Ca[r:r + 1]), Cr, Rr, f"split {M}x{N}x{K} row {r}")
