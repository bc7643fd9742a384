"""Oracle for the choice of block shape and K-layer count (row f1).

TEST INFRASTRUCTURE ONLY -- never called by the product.

Section III.B models each BRGEMM of the critical path with a roofline:
Eq. 1 T = max(G*gamma, beta*(S_A + S_B)) when both panels come from slow
memory (Eq. 2-4 when one or both are already in fast memory), sums these over
the critical path, adds the reads/writes of C and, for 2.5D/3D runs, of the C
copies, and takes the decomposition with the smallest time (Section III.C,
second option).  The reading for this GPU:

* a core is a CU; it holds up to ``occ`` persistent workgroups; a workgroup
  gets 1/w of its CU's MFMA rate (gamma = w / (flops per clock x rate)), where
  w = min(occ, ceil(active / CUs)) is the number that actually share a CU: the
  dispatcher spreads a grid over the CUs before it doubles up (and a grid of at
  most one 128x128 block per CU runs a one-per-CU kernel);
* one BRGEMM is one 64-deep K block of one task (BM x BN output block):
  G = 2*BM*BN*64 flops, S_A = BM*64*2 and S_B = 64*BN*2 bytes;
* fast memory is an XCD's L2, slow memory is HBM.  The ``active`` tasks in
  flight split over the XCDs; each XCD's share forms a compact patch of about
  sqrt(P) x sqrt(P) blocks (P = active / XCDs, at least 1), whose panels are
  fetched once per patch, so a task pays beta*(S_A + S_B)/sqrt(P) per block,
  with beta = active / (HBM bytes per clock) (the bandwidth is shared);
* the critical path is ceil(tasks / slots) rounds of ceil(nK / c) blocks,
  plus C (M*N*out bytes) or, with c > 1, the fp32 copies written and read
  back (2*c*M*N*4) and then C, all at the HBM rate, plus one launch (two with
  a reduction);
* candidates: 256x256, 128x256, 256x128, 128x128 blocks, c in {1, 2, 4, 8, 16}
  capped at nK = ceil(K/64) (16 so that a K-dominant GEMM whose C grid has only
  16 blocks of 256x256 can still occupy 256 CUs: Section II.E lets the
  decomposition Tm x Tn x c follow the aspect ratio of the problem); times within a relative 1e-9 are ties, settled by
  fewer padded output elements, then by the order of evaluation (that block
  order, then ascending layer counts).

The calibration numbers are MI355X measurements (achieved MFMA rate per CU and
per block shape, loaded HBM bytes per clock, launch cost).

Parity: pinned in tests/test_oracle_model.py (Eq. 1 evaluated by hand on a
compute-bound and a memory-bound block, three whole estimates written out by
hand -- one of a grid smaller than the machine, where a workgroup has its CU
to itself -- the M <-> N symmetry, the K-dominant configuration of Section IV
needing layers while a large square does not, ties).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Tuple

FLOPS_PER_CLK_CU = 4096.0 * 0.74            # dense bf16 MFMA per CU per clock x achieved fraction
RATE = {(128, 128): 0.60, (256, 128): 0.80, (128, 256): 0.86, (256, 256): 1.0}
HBM_BYTES_PER_CLK = 3500.0
LAUNCH_CLK = 10000.0
XCDS = 8
BK = 64
SHAPES = [(256, 256), (128, 256), (256, 128), (128, 128)]   # tie order
LAYERS = [1, 2, 4, 8, 16]


def brgemm_clk(G: float, gamma: float, beta: float, s_a: float, s_b: float) -> float:
    """Eq. 1: both panels from slow memory."""
    return max(G * gamma, beta * (s_a + s_b))


def estimate(M: int, N: int, K: int, out_bytes: int, num_cus: int, occ: Dict[Tuple[int, int], int],
             shape: Tuple[int, int], c: int) -> Tuple[float, float]:
    """(estimated clocks, padded output elements) of one decomposition."""
    BM, BN = shape
    nK = -(-K // BK) if K > 0 else 0
    gm, gn = -(-M // BM), -(-N // BN)
    o = max(1, occ[shape])
    tasks = gm * gn * c
    slots = num_cus * o
    rounds = -(-tasks // slots)
    blocks = -(-nK // c)
    active = min(tasks, slots)
    G = 2.0 * BM * BN * BK
    w = min(o, max(1, -(-active // num_cus)))
    gamma = w / (FLOPS_PER_CLK_CU * RATE[shape])
    patch = max(1.0, active / XCDS)
    beta = active / HBM_BYTES_PER_CLK
    t_blk = brgemm_clk(G, gamma, beta / math.sqrt(patch), BM * BK * 2.0, BK * BN * 2.0)
    c_traffic = M * N * out_bytes if c == 1 else 2 * c * M * N * 4 + M * N * out_bytes
    launches = 1 if c == 1 else 2
    clk = launches * LAUNCH_CLK + rounds * blocks * t_blk + c_traffic / HBM_BYTES_PER_CLK
    return clk, float(tasks * BM * BN)


def candidates(K: int, shape: Optional[Tuple[int, int]], layers: int) -> List[Tuple[Tuple[int, int], int]]:
    nK = -(-K // BK) if K > 0 else 0
    out = []
    for s in SHAPES:
        if shape is not None and s != shape:
            continue
        seen = []
        for c in ([layers] if layers > 0 else LAYERS):
            ce = min(c, nK) if nK > 0 else 1
            if ce not in seen:
                seen.append(ce)
                out.append((s, ce))
    return out


def choose(M: int, N: int, K: int, out_bytes: int = 4, num_cus: int = 256,
           occ: Optional[Dict[Tuple[int, int], int]] = None, shape: Optional[Tuple[int, int]] = None,
           layers: int = 0) -> Tuple[Tuple[int, int], int, float]:
    """Fastest decomposition: (block shape, layer count, estimated clocks)."""
    if occ is None:
        occ = {(128, 128): 2, (256, 128): 1, (128, 256): 1, (256, 256): 1}
    best = None
    for s, c in candidates(K, shape, layers):
        clk, pad = estimate(M, N, K, out_bytes, num_cus, occ, s, c)
        if best is None:
            best = (clk, pad, c, s)
            continue
        b_clk, b_pad, b_c, _ = best
        tol = 1e-9 * b_clk
        if clk < b_clk - tol or (clk <= b_clk + tol and pad < b_pad):
            best = (clk, pad, c, s)
    return best[3], best[2], best[0]
