"""Pins of the SFC oracle (oracle/sfc_ref.py) against facts fixed outside it."""
import pytest

from oracle.sfc_ref import row_major_ref, sfc_cells, sfc_ref
import sfc_pins

CONFIG_GRIDS = [(4, 4), (32, 32), (24, 55), (12, 55), (12, 28), (8, 8), (16, 16), (16, 56),
                (32, 112), (16, 16), (4, 8), (8, 4), (2, 2), (1, 1)]


def test_textbook_hilbert_on_power_of_two_squares():
    # Section II.B: on power-of-two squares the generalized curve is the classical Hilbert curve.
    assert sfc_pins.check_textbook(sfc_cells, max_log2=8) == []


def test_paper_patch_statements():
    # Section II.B (Figure 2), Section II.D (Figure 3), Section II.E (Figure 4).
    assert sfc_pins.check_paper_patches(sfc_cells) == []


def test_invariants_exhaustive_small_grids():
    grids = [(a, b) for a in range(1, 65) for b in range(1, 65)]
    assert sfc_pins.check_invariants(sfc_cells, grids) == []


def test_invariants_on_workload_grids():
    assert sfc_pins.check_invariants(sfc_cells, CONFIG_GRIDS) == []


def test_brute_force_hamiltonian_tiny_grids():
    assert sfc_pins.check_brute_force(sfc_cells, max_cells=16) == []


def test_exception_grids_have_no_unit_step_walk_to_the_corner():
    # The chessboard argument behind the odd-major / even-minor exception.
    for gm, gn in [(3, 2), (5, 2), (2, 3), (2, 5), (5, 4), (4, 5), (7, 2)]:
        corner = (gm - 1, 0) if gm >= gn else (0, gn - 1)
        assert all(p[-1] != corner for p in sfc_pins.hamiltonian_paths(gm, gn))


def test_hand_traces():
    assert sfc_pins.check_hand_traces(sfc_cells) == []


def test_halving_reading_changes_some_curves():
    # Reading A1: floor and truncating halving both give valid curves but differ on 10x10.
    f = sfc_cells(10, 10, "floor")
    t = sfc_cells(10, 10, "trunc")
    assert f != t
    assert sfc_pins.check_invariants(lambda a, b: sfc_cells(a, b, "trunc"), [(10, 10)]) == []


def test_table_encoding():
    for gm, gn in [(3, 7), (7, 3), (4, 4)]:
        assert sfc_ref(gm, gn) == [x * gn + y for x, y in sfc_cells(gm, gn)]
    assert row_major_ref(3, 5) == list(range(15))


@pytest.mark.parametrize("gm,gn", [(0, 3), (3, 0), (-1, 2)])
def test_rejects_empty_grids(gm, gn):
    with pytest.raises(ValueError):
        sfc_cells(gm, gn)
