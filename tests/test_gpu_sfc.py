"""The device curve generator (sfc_tile_order, which also feeds the GEMM's
table cache) against the oracle, bit for bit."""
import numpy as np
import pytest

from oracle.sfc_ref import row_major_ref, sfc_ref

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sg():
    from paper_2601_16294_amd import sfcgemm
    return sfcgemm


def test_exhaustive_small_grids(sg):
    bad = []
    for gm in range(1, 65):
        for gn in range(1, 65):
            if sg.sfc_tile_order(gm, gn).tolist() != sfc_ref(gm, gn):
                bad.append((gm, gn))
    assert bad == []


@pytest.mark.parametrize("gm,gn", [(4, 4), (32, 32), (24, 55), (12, 55), (12, 28), (8, 8), (16, 56),
                                   (32, 112), (128, 128), (512, 32), (256, 64), (100, 100), (97, 203),
                                   (300, 7), (1, 1000), (1000, 1), (2, 999)])
def test_workload_and_large_grids(sg, gm, gn):
    assert sg.sfc_tile_order(gm, gn).tolist() == sfc_ref(gm, gn)


def test_row_major_mode(sg):
    assert sg.sfc_tile_order(7, 9, "row_major").tolist() == row_major_ref(7, 9)


def test_invalid_grid_raises(sg):
    with pytest.raises(sg.SfcError):
        sg.sfc_tile_order(0, 5)
