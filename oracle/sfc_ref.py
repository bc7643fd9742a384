"""Oracle: the generalized Hilbert ("SFC") order over an arbitrary gm x gn grid.

TEST INFRASTRUCTURE ONLY -- slow, plain, recursive; never called by the product.

What it follows
---------------
Section II.B of the paper adopts the generalized Hilbert curve for rectangles
of any size (its reference [gilbert]) and describes it as a recursion that cuts
the domain into parts and walks each part as a "U" before moving on.  Listing 1
(Section II.D) builds the map once from the (Mb, Nb) block grid and turns a 1D
position into the block pair (im, in).

The recursion, as implemented here (a rectangle is a start cell plus a "major"
vector along which the walk advances and a "minor" vector across it):

* a strip one cell thick is walked straight along its long side;
* a rectangle much longer than wide (2*major > 3*minor) is cut across its major
  axis into two halves walked one after the other, both keeping the orientation;
* otherwise it is cut into three parts: the near half of the minor side walked
  with the axes exchanged, then the far half of the minor side walked with the
  original axes, then the remaining block walked back towards the far corner;
* halving rounds toward minus infinity (reading A1), and when the half is odd
  (and the side longer than 2) it is grown by one cell so that sub-walks end on
  the corner where their successor starts.

Readings of the paper where it leaves a choice: the x coordinate is the block
row im and y the block column in; the longer side is the major axis at the top
level, ties going to x; the order is returned as ``cell = im * gn + in``.

Parity: pinned by tests/test_oracle_sfc.py against the textbook Hilbert
index->coordinate routine on 2^k x 2^k grids, the paper's patch statements
(Section II.B, Section II.D, Section II.E), exhaustive invariant sweeps and
brute-force Hamiltonian-path enumeration on tiny grids.
"""
from __future__ import annotations

from typing import Iterator, List, Tuple


def _sign(v: int) -> int:
    return (v > 0) - (v < 0)


def _half(v: int, halving: str) -> int:
    """Half of a signed extent.  'floor' is reading A1; 'trunc' exists only so a
    test can show that the choice changes some curves."""
    if halving == "floor":
        return v // 2
    if halving == "trunc":
        return int(v / 2)
    raise ValueError(halving)


def _walk(x: int, y: int, ax: int, ay: int, bx: int, by: int,
          halving: str) -> Iterator[Tuple[int, int]]:
    """Yield the cells of the rectangle with start (x, y), major vector (ax, ay)
    and minor vector (bx, by), in curve order."""
    major = abs(ax + ay)          # exactly one of ax, ay is non-zero
    minor = abs(bx + by)
    sax, say = _sign(ax), _sign(ay)
    sbx, sby = _sign(bx), _sign(by)

    if minor == 1:                # a strip along the major axis
        for i in range(major):
            yield (x + i * sax, y + i * say)
        return
    if major == 1:                # a strip along the minor axis
        for i in range(minor):
            yield (x + i * sbx, y + i * sby)
        return

    hax, hay = _half(ax, halving), _half(ay, halving)
    hbx, hby = _half(bx, halving), _half(by, halving)
    hmajor = abs(hax + hay)
    hminor = abs(hbx + hby)

    if 2 * major > 3 * minor:
        # Long rectangle: two halves along the major axis.
        if hmajor % 2 == 1 and major > 2:
            hax, hay = hax + sax, hay + say
        yield from _walk(x, y, hax, hay, bx, by, halving)
        yield from _walk(x + hax, y + hay, ax - hax, ay - hay, bx, by, halving)
        return

    # Three parts: up the near minor half, across, and back down.
    if hminor % 2 == 1 and minor > 2:
        hbx, hby = hbx + sbx, hby + sby
    yield from _walk(x, y, hbx, hby, hax, hay, halving)
    yield from _walk(x + hbx, y + hby, ax, ay, bx - hbx, by - hby, halving)
    yield from _walk(x + (ax - sax) + (hbx - sbx), y + (ay - say) + (hby - sby),
                     -hbx, -hby, -(ax - hax), -(ay - hay), halving)


def sfc_cells(gm: int, gn: int, halving: str = "floor") -> List[Tuple[int, int]]:
    """The (im, in) block pairs of a gm x gn grid in curve order."""
    if gm <= 0 or gn <= 0:
        raise ValueError("grid sides must be positive")
    if gm >= gn:
        return list(_walk(0, 0, gm, 0, 0, gn, halving))
    return list(_walk(0, 0, 0, gn, gm, 0, halving))


def sfc_ref(gm: int, gn: int, halving: str = "floor") -> List[int]:
    """The map of Listing 1 as a flat table: entry s is im * gn + in of the
    block visited at curve position s."""
    return [im * gn + jn for (im, jn) in sfc_cells(gm, gn, halving)]


def row_major_ref(gm: int, gn: int) -> List[int]:
    """The plain row-major block order that the SFC order is compared with."""
    return list(range(gm * gn))
