"""The 125-shape sweep (M, N, K in {512, ..., 8192}, bf16 out) in the launch
configuration the benchmark times -- the library's own block shape and layer
count (SFC_TILE_AUTO, SFC_CA_AUTO) -- checked against the oracle on sampled
elements: random points plus the last row and the last column."""
import numpy as np
import pytest
import torch

from oracle import check as ocheck
from oracle import gemm as ogemm
from paper_2601_16294_amd.inputs import draw, sweep_gemms
from gpu_util import sg, to_host, upload

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

_host, _dev = {}, {}


def _mat(rows, cols, dist, seed):
    if seed not in _host:
        _host[seed] = draw(rows, cols, dist, seed)
        _dev[seed] = upload(_host[seed])
    return _host[seed], _dev[seed]


@pytest.mark.parametrize("K", [512, 1024, 2048, 4096, 8192])
def test_sweep_shapes_auto_choice(K):
    for g in sweep_gemms():
        if g.K != K:
            continue
        A, dA = _mat(g.M, g.K, g.dist_a, g.seed_a)
        B, dB = _mat(g.K, g.N, g.dist_b, g.seed_b)
        print(f"[sweep] {g.M}x{g.N}x{g.K} auto", flush=True)
        C = torch.full((g.M, g.N), float("nan"), dtype=torch.bfloat16, device="cuda")
        sg().sfc_gemm_ex(dA, dB, C, ca_layers=0, tile="auto")
        torch.cuda.synchronize()
        Ch = to_host(C)
        del C
        rng = np.random.default_rng(g.M * 7 + g.N * 3 + g.K)
        rows = rng.integers(0, g.M, 512)
        cols = rng.integers(0, g.N, 512)
        Cp, Rp = ogemm.gemm_ref_points(A, B, g.K, g.K, g.N, rows, cols)
        ocheck.assert_gemm_close(Ch[rows, cols], Cp, Rp, f"{g.M}x{g.N}x{g.K} points")
        Cr, Rr = ogemm.gemm_ref_rows(A, B, g.N, g.K, g.K, g.N, row0=g.M - 1, nrows=1)
        ocheck.assert_gemm_close(Ch[g.M - 1:], Cr, Rr, f"{g.M}x{g.N}x{g.K} last row")
        rr = np.arange(g.M)
        Cc, Rc = ogemm.gemm_ref_points(A, B, g.K, g.K, g.N, rr, np.full(g.M, g.N - 1))
        ocheck.assert_gemm_close(Ch[:, g.N - 1], Cc, Rc, f"{g.M}x{g.N}x{g.K} last column")
    _host.clear()
    _dev.clear()
    torch.cuda.empty_cache()
