"""Pin checks for a generalized Hilbert order, shared by the oracle tests and
the mutation test.  Each check takes ``cells(gm, gn) -> [(im, in), ...]`` and
returns a list of failure strings (empty when the pin holds)."""
from __future__ import annotations

import json
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_patches.json")


def d2xy(n: int, d: int):
    """Textbook Hilbert index -> (x, y) on an n x n grid, n a power of two
    (the classical bit-by-bit construction)."""
    x = y = 0
    s = 1
    t = d
    while s < n:
        rx = 1 & (t // 2)
        ry = 1 & (t ^ rx)
        if ry == 0:
            if rx == 1:
                x = s - 1 - x
                y = s - 1 - y
            x, y = y, x
        x += s * rx
        y += s * ry
        t //= 4
        s *= 2
    return x, y


def check_textbook(cells, max_log2: int = 8):
    fails = []
    for e in range(0, max_log2 + 1):
        n = 1 << e
        got = cells(n, n)
        want = [d2xy(n, d) for d in range(n * n)]
        if got != want:
            fails.append(f"{n}x{n} differs from the textbook Hilbert curve")
    return fails


def _bbox(cs):
    xs = [c[0] for c in cs]
    ys = [c[1] for c in cs]
    return min(xs), max(xs) + 1, min(ys), max(ys) + 1


def _is_rect(cs):
    x0, x1, y0, y1 = _bbox(cs)
    return (x1 - x0) * (y1 - y0) == len(cs) and len(set(cs)) == len(cs), (x1 - x0, y1 - y0)


def check_paper_patches(cells):
    g = json.load(open(GOLDEN))
    fails = []
    p = g["grid16_patches"]
    c = cells(*p["grid"])
    patch = c[p["patch"]["first"]:p["patch"]["first"] + p["patch"]["count"]]
    ok, sides = _is_rect(patch)
    if not ok or sorted(sides) != sorted(p["patch"]["sides"]) or (0, 0) not in patch:
        fails.append(f"16x16: positions 0-31 are not an 8x4 patch at the origin ({sides})")
    sub = c[p["sub_patch"]["first"]:p["sub_patch"]["first"] + p["sub_patch"]["count"]]
    ok2, sides2 = _is_rect(sub)
    # "8x4" and "2x4" name the sides in the same axis order
    if ok and ok2:
        long_axis = 0 if sides[0] == 8 else 1
        if not (sides2[long_axis] == 2 and sides2[1 - long_axis] == 4 and set(sub) <= set(patch)):
            fails.append(f"16x16: positions 8-15 are not a 2x4 sub-patch ({sides2})")
    else:
        fails.append("16x16: positions 8-15 are not a rectangle")

    def chunk_check(grid, chunks, chunk_grid=None, chunk_sides=None, tag=""):
        cc = cells(*grid)
        size = len(cc) // chunks
        boxes = []
        for q in range(chunks):
            part = cc[q * size:(q + 1) * size]
            okq, sq = _is_rect(part)
            if not okq:
                return [f"{tag} {grid} / {chunks}: chunk {q} is not a rectangle"]
            if chunk_sides is not None and [sq[0], sq[1]] not in [list(s) for s in chunk_sides]:
                return [f"{tag} {grid} / {chunks}: chunk {q} has sides {sq}"]
            boxes.append(_bbox(part))
        if chunk_grid is not None:
            x_starts = sorted({b[0] for b in boxes})
            y_starts = sorted({b[2] for b in boxes})
            if [len(x_starts), len(y_starts)] != list(chunk_grid):
                return [f"{tag} {grid} / {chunks}: chunk grid {len(x_starts)}x{len(y_starts)}"]
        return []

    L = g["grid128_layers"]
    for case in L["cases"]:
        fails += chunk_check(L["grid"], case["chunks"], case.get("chunk_grid"), case.get("chunk_sides"),
                             "layers")
    A = g["aspect_ratio"]
    for case in A["cases"]:
        fails += chunk_check(case["grid"], A["chunks"], case["chunk_grid"], None, "aspect")
    return fails


def expected_exception(gm: int, gn: int) -> bool:
    """Odd major side and even minor side: no unit-step walk joins the two
    corners of the major side (chessboard colouring), so the construction may
    end elsewhere or take one diagonal step."""
    major, minor = (gm, gn) if gm >= gn else (gn, gm)
    return major % 2 == 1 and minor % 2 == 0


def check_invariants(cells, grids):
    fails = []
    for gm, gn in grids:
        c = cells(gm, gn)
        if len(c) != gm * gn or len(set(c)) != gm * gn or \
                not all(0 <= x < gm and 0 <= y < gn for x, y in c):
            fails.append(f"{gm}x{gn}: not a bijection onto the grid")
            continue
        if c[0] != (0, 0):
            fails.append(f"{gm}x{gn}: does not start at (0, 0)")
        diag = 0
        for (x0, y0), (x1, y1) in zip(c, c[1:]):
            dx, dy = abs(x1 - x0), abs(y1 - y0)
            if dx + dy == 1:
                continue
            if dx == 1 and dy == 1:
                diag += 1
            else:
                fails.append(f"{gm}x{gn}: jump {(x0, y0)} -> {(x1, y1)}")
                break
        exc = expected_exception(gm, gn)
        if diag > (1 if exc else 0):
            fails.append(f"{gm}x{gn}: {diag} diagonal steps")
        corner = (gm - 1, 0) if gm >= gn else (0, gn - 1)
        if not exc and c[-1] != corner:
            fails.append(f"{gm}x{gn}: ends at {c[-1]}, not {corner}")
        if gm == 1 or gn == 1:
            line = [(i, 0) for i in range(gm)] if gn == 1 else [(0, j) for j in range(gn)]
            if c != line:
                fails.append(f"{gm}x{gn}: a one-cell-thick grid is not walked straight")
    return fails


def hamiltonian_paths(gm: int, gn: int):
    """All unit-step walks from (0, 0) that visit every cell once (tiny grids)."""
    total = gm * gn
    seen = [[False] * gn for _ in range(gm)]
    path = [(0, 0)]
    seen[0][0] = True
    out = []

    def rec():
        if len(path) == total:
            out.append(list(path))
            return
        x, y = path[-1]
        for nx, ny in ((x + 1, y), (x - 1, y), (x, y + 1), (x, y - 1)):
            if 0 <= nx < gm and 0 <= ny < gn and not seen[nx][ny]:
                seen[nx][ny] = True
                path.append((nx, ny))
                rec()
                path.pop()
                seen[nx][ny] = False

    rec()
    return out


def check_brute_force(cells, max_cells: int = 16):
    fails = []
    for gm in range(1, max_cells + 1):
        for gn in range(1, max_cells // gm + 1):
            c = cells(gm, gn)
            paths = hamiltonian_paths(gm, gn)
            corner = (gm - 1, 0) if gm >= gn else (0, gn - 1)
            to_corner = [p for p in paths if p[-1] == corner]
            if c in paths:
                continue
            # not a unit-step walk: allowed only where no unit-step walk reaches the corner
            if to_corner or not expected_exception(gm, gn):
                fails.append(f"{gm}x{gn}: not a unit-step Hamiltonian walk although one exists")
    return fails


HAND_TRACES = {
    # Traced by hand from the recursion rules (strip / two halves / three parts,
    # floor halving, odd halves grown by one), independently of any code.
    (2, 2): [(0, 0), (0, 1), (1, 1), (1, 0)],
    (3, 2): [(0, 0), (0, 1), (1, 1), (2, 1), (2, 0), (1, 0)],
    (3, 3): [(0, 0), (0, 1), (0, 2), (1, 2), (2, 2), (2, 1), (1, 1), (1, 0), (2, 0)],
    (5, 4): [(0, 0), (1, 0), (1, 1), (0, 1), (0, 2), (0, 3), (1, 3), (1, 2), (2, 2), (2, 3),
             (3, 3), (4, 3), (4, 2), (3, 2), (4, 1), (3, 1), (2, 1), (2, 0), (3, 0), (4, 0)],
}


def check_hand_traces(cells):
    return [f"{g}: differs from the hand trace" for g, want in HAND_TRACES.items() if cells(*g) != want]


def all_pins(cells, sweep_max: int = 24):
    grids = [(a, b) for a in range(1, sweep_max + 1) for b in range(1, sweep_max + 1)]
    return (check_textbook(cells, 6) + check_paper_patches(cells) + check_invariants(cells, grids)
            + check_brute_force(cells, 12) + check_hand_traces(cells))
