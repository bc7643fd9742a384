"""Seeded synthetic inputs for the SFC-CA GEMM workloads.

This module only draws numbers: it holds none of the method's arithmetic, and
both the HIP path and the CPU oracle receive exactly the arrays it returns.

Matrices are drawn in fp32 with ``numpy.random.default_rng(seed)`` and
rounded to bf16 (round to nearest even, done by torch's CPU conversion); they
are returned as uint16 bit patterns, row-major with a chosen leading
dimension.  Padding columns (ld > cols) hold a NaN sentinel so that a kernel
that reads them shows it.

Workloads (the paper's shapes and roles: Section IV.A's cube sweep, the
Llama-3-8B prefill projections of Section IV.D) are synthetic stand-ins; no
dataset or trained weight is involved.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np
import torch

NAN_BF16 = 0x7FC0


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def draw(rows: int, cols: int, dist: Tuple, seed: int, ld: Optional[int] = None) -> np.ndarray:
    """A rows x ld uint16 array of bf16 patterns; columns >= cols are NaN.

    dist is ("uniform", lo, hi), ("normal", mean, std) or ("int", lo, hi)
    (integers drawn uniformly from [lo, hi], inclusive).
    """
    ld = cols if ld is None else ld
    if ld < cols:
        raise ValueError("ld < cols")
    rng = np.random.default_rng(seed)
    kind = dist[0]
    if kind == "uniform":
        x = rng.uniform(dist[1], dist[2], size=(rows, cols)).astype(np.float32)
    elif kind == "normal":
        x = rng.normal(dist[1], dist[2], size=(rows, cols)).astype(np.float32)
    elif kind == "int":
        x = rng.integers(dist[1], dist[2] + 1, size=(rows, cols)).astype(np.float32)
    else:
        raise ValueError(kind)
    out = np.full((rows, ld), NAN_BF16, dtype=np.uint16)
    if rows and cols:
        out[:, :cols] = _to_bf16_bits(x)
    return out


NAN_E4M3 = 0x7F
NAN_E5M2 = 0x7F


def draw_e4m3(rows: int, cols: int, dist: Tuple, seed: int, ld: Optional[int] = None) -> np.ndarray:
    """A rows x ld uint8 array of OCP FP8 E4M3 codes (drawn in fp32 as in draw()
    and converted by torch's float8_e4m3fn cast, round to nearest even);
    columns >= cols hold the NaN code."""
    return draw_fp8(rows, cols, dist, seed, ld, "e4m3")


def draw_fp8(rows: int, cols: int, dist: Tuple, seed: int, ld: Optional[int] = None,
             fmt: str = "e4m3") -> np.ndarray:
    """draw_e4m3 for either OCP format: fmt "e4m3" (torch.float8_e4m3fn) or
    "e5m2" (torch.float8_e5m2); columns >= cols hold that format's NaN code."""
    dtype = {"e4m3": torch.float8_e4m3fn, "e5m2": torch.float8_e5m2}[fmt]
    ld = cols if ld is None else ld
    if ld < cols:
        raise ValueError("ld < cols")
    rng = np.random.default_rng(seed)
    kind = dist[0]
    if kind == "uniform":
        x = rng.uniform(dist[1], dist[2], size=(rows, cols)).astype(np.float32)
    elif kind == "normal":
        x = rng.normal(dist[1], dist[2], size=(rows, cols)).astype(np.float32)
    elif kind == "int":
        x = rng.integers(dist[1], dist[2] + 1, size=(rows, cols)).astype(np.float32)
    else:
        raise ValueError(kind)
    out = np.full((rows, ld), NAN_E4M3 if fmt == "e4m3" else NAN_E5M2, dtype=np.uint8)
    if rows and cols:
        t = torch.from_numpy(np.ascontiguousarray(x)).to(dtype)
        out[:, :cols] = t.view(torch.uint8).numpy()
    return out


@dataclass
class Gemm:
    M: int
    N: int
    K: int
    dist_a: Tuple
    dist_b: Tuple
    seed_a: int
    seed_b: int
    out: str = "f32"                      # "f32" or "bf16"

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K

    def operands(self, lda: Optional[int] = None, ldb: Optional[int] = None):
        A = draw(self.M, self.K, self.dist_a, self.seed_a, lda)
        B = draw(self.K, self.N, self.dist_b, self.seed_b, ldb)
        return A, B


@dataclass
class Workload:
    name: str
    gemms: List[Gemm]
    tile: str = "auto"                    # "auto", "128x128", "256x128", "128x256", "256x256"
    ca_layers: List[int] = field(default_factory=lambda: [1])

    @property
    def flops(self) -> int:
        return sum(g.flops for g in self.gemms)


def workloads() -> List[Workload]:
    """The five measured workloads.  Seeds: workload k draws A with 1000k+1 and
    B with 1000k+2; GEMM j of the prefill batch uses 5000+10j+1 and +2."""
    U = ("uniform", -1.0, 1.0)
    return [
        Workload("cube512_f32out_t128", [Gemm(512, 512, 512, U, U, 1001, 1002)], tile="128x128"),
        Workload("square8192_bf16out_t256",
                 [Gemm(8192, 8192, 8192, ("normal", 0.0, 1.0), ("normal", 0.0, 1.0), 2001, 2002,
                       out="bf16")], tile="256x256"),
        Workload("ragged3000x7000x2048_f32out", [Gemm(3000, 7000, 2048, U, U, 3001, 3002)]),
        Workload("kdominant1024x1024x65536_f32out",
                 [Gemm(1024, 1024, 65536, ("normal", 0.0, 0.1), ("normal", 0.0, 0.1), 4001, 4002)],
                 ca_layers=[1, 2, 4, 8, 0]),     # 0: the count the library's model picks
        Workload("prefill4096_bf16out",
                 [Gemm(4096, n, k, ("normal", 0.0, 1.0), ("normal", 0.0, 0.02),
                       5000 + 10 * j + 1, 5000 + 10 * j + 2, out="bf16")
                  for j, (n, k) in enumerate([(4096, 4096), (14336, 4096), (4096, 14336)])]),
    ]


SWEEP_DIMS = (512, 1024, 2048, 4096, 8192)


def sweep_gemms() -> List[Gemm]:
    """The 125-shape sweep of Section IV.A: M, N, K each from {512, 1024, 2048,
    4096, 8192}, bf16 inputs U(-1, 1), bf16 output.  A depends only on (M, K)
    and B only on (K, N), so 25 A matrices and 25 B matrices serve every shape:
    A of (M, K) = (d_i, d_k) uses seed 700000 + 100i + 10k + 1, B of (K, N) =
    (d_k, d_n) uses 700000 + 100k + 10n + 2."""
    U = ("uniform", -1.0, 1.0)
    out = []
    for i, M in enumerate(SWEEP_DIMS):
        for j, N in enumerate(SWEEP_DIMS):
            for k, K in enumerate(SWEEP_DIMS):
                out.append(Gemm(M, N, K, U, U, 700000 + 100 * i + 10 * k + 1, 700000 + 100 * k + 10 * j + 2,
                                out="bf16"))
    return out


def workload(name: str) -> Workload:
    for w in workloads():
        if w.name == name:
            return w
    raise KeyError(name)
