"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and hand the result back as host arrays."""
from __future__ import annotations

import numpy as np
import torch

from oracle import bf16 as obf16


def sg():
    from paper_2601_16294_amd import sfcgemm
    return sfcgemm


def upload(bits: np.ndarray) -> torch.Tensor:
    return sg().to_device_bf16(bits)


def run_gemm(A_bits, B_bits, M, N, K, out="f32", ldc=None, ca_layers=1, tile="auto", order="hilbert",
             sched="interleaved", workspace=None, dev_A=None, dev_B=None):
    """C = A*B on the GPU.  A_bits is (M, lda) and B_bits is (K, ldb) uint16.
    Returns the whole (M, ldc) output buffer, initialised to NaN before the
    call, as float64 on the host."""
    A = upload(A_bits) if dev_A is None else dev_A
    B = upload(B_bits) if dev_B is None else dev_B
    ldc = N if ldc is None else ldc
    dtype = torch.float32 if out == "f32" else torch.bfloat16
    Cfull = torch.full((M, max(ldc, 1)), float("nan"), dtype=dtype, device="cuda")
    sg().sfc_gemm_ex(A[:M, :K], B[:K, :N], Cfull[:, :N], ca_layers=ca_layers, tile=tile, order=order,
                     sched=sched, workspace=workspace)
    torch.cuda.synchronize()
    return to_host(Cfull)


def to_host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return obf16.bf16_to_f64(t.cpu().view(torch.int16).numpy().view(np.uint16))
    return t.cpu().numpy().astype(np.float64)


def raw_bits(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.cpu().view(torch.int16).numpy().view(np.uint16)
    return t.cpu().numpy().view(np.uint32)
