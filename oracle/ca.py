"""Oracle for the communication-avoiding (CA) split of Section II.C / II.D.

TEST INFRASTRUCTURE ONLY -- never called by the product.

Listing 1 replicates C into K_layers copies; copy l is produced from the l-th
contiguous range of K blocks (Kb_per_layer = Kb / K_layers blocks each) and the
copies are then summed by a strided add-reduce.

* ``k_slices`` gives those ranges in elements for block depth ``bk``.  Where K
  is not a multiple of bk, or the block count is not a multiple of the layer
  count, reading A4 applies: nK = ceil(K / bk) blocks, at most nK layers,
  layer l owning blocks [floor(l*nK/c), floor((l+1)*nK/c)).
* ``reduce_layers_f32`` is the reduction written out: fp32 sums in ascending
  layer order (reading A6), one rounding per addition.

Parity: pinned in tests/test_oracle_gemm.py (the slices tile [0, K) exactly,
are contiguous and ascending, differ in size by at most one block, and the
reduction of integer-valued layers is exact).
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np


def effective_layers(K: int, c: int, bk: int) -> int:
    nk = -(-K // bk) if K > 0 else 0
    return max(1, min(c, nk))


def k_slices(K: int, c: int, bk: int) -> List[Tuple[int, int]]:
    nk = -(-K // bk) if K > 0 else 0
    ce = effective_layers(K, c, bk)
    out = []
    for layer in range(ce):
        b0 = (layer * nk) // ce
        b1 = ((layer + 1) * nk) // ce
        out.append((min(K, b0 * bk), min(K, b1 * bk)))
    return out


def reduce_layers_f32(W: np.ndarray) -> np.ndarray:
    """Sum of W[0] + W[1] + ... + W[c-1] in fp32, left to right."""
    W = np.asarray(W, dtype=np.float32)
    acc = W[0].copy()
    for layer in range(1, W.shape[0]):
        acc = (acc + W[layer]).astype(np.float32)
    return acc
