"""Python binding of libsfcgemm.so (the C ABI in include/sfcgemm.h).

Argument marshalling only: every step of the GEMM runs in the library's HIP
kernels.  torch supplies device memory and the stream.  If the library is not
built, importing this module raises; there is no fallback.

Names follow the C ABI: ``sfc_tile_order``, ``sfc_gemm``, ``sfc_gemm_bf16out``,
``sfc_gemm_ex``, ``sfc_gemm_ws_size``, ``sfc_gemm_plan``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsfcgemm.so")

SFC_OK = 0
SFC_ERR_INVALID_ARG = -1
SFC_ERR_UNSUPPORTED = -2
SFC_ERR_WORKSPACE = -3
SFC_ERR_HIP = -4

SFC_OUT_F32 = 0
SFC_OUT_BF16 = 1

SFC_CA_AUTO = 0
TILES = {"auto": 0, "128x128": 1, "256x128": 2, "128x256": 3, "256x256": 4}
TILE_NAMES = {v: k for k, v in TILES.items()}
ORDERS = {"hilbert": 0, "row_major": 1}
SCHEDS = {"interleaved": 0, "block": 1, "interleaved_plain": 2}

# Every symbol include/sfcgemm.h declares.
EXPORTS = ["sfc_tile_order", "sfc_tile_order_ex", "sfc_gemm", "sfc_gemm_bf16out", "sfc_gemm_ws_size",
           "sfc_gemm_ex", "sfc_gemm_fused_ex", "sfc_gemm_noalloc_ex", "sfc_gemm_f8_ex", "sfc_gemm_f8_fmt_ex", "sfc_gemm_plan", "sfc_gemm_f8_plan", "sfc_gemm_model", "sfc_probe_mfma", "sfc_strerror",
           "sfc_last_error", "sfc_version"]


class SfcError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {code} ({strerror(code)}): {last_error()}")
        self.code = code


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2601_16294_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, p, sz = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t
    lib.sfc_tile_order.argtypes = [i32, i32, p]
    lib.sfc_tile_order.restype = i32
    lib.sfc_tile_order_ex.argtypes = [i32, i32, i32, p]
    lib.sfc_tile_order_ex.restype = i32
    gemm_args = [i64, i64, i64, p, i64, p, i64, p, i64, i32, p]
    lib.sfc_gemm.argtypes = gemm_args
    lib.sfc_gemm.restype = i32
    lib.sfc_gemm_bf16out.argtypes = gemm_args
    lib.sfc_gemm_bf16out.restype = i32
    lib.sfc_gemm_ex.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, i32, i32, i32, i32, i32, p, sz, p]
    lib.sfc_gemm_ex.restype = i32
    lib.sfc_gemm_fused_ex.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, i32, i32, i32, i32, i32, p, sz, p]
    lib.sfc_gemm_fused_ex.restype = i32
    lib.sfc_gemm_noalloc_ex.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, i32, i32, i32, i32, i32, p]
    lib.sfc_gemm_noalloc_ex.restype = i32
    lib.sfc_gemm_f8_ex.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, i32, i32, i32, i32, i32, p, sz, p]
    lib.sfc_gemm_f8_ex.restype = i32
    lib.sfc_gemm_f8_fmt_ex.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, i32, i32, i32, i32, i32, i32, i32, p,
                                       sz, p]
    lib.sfc_gemm_f8_fmt_ex.restype = i32
    lib.sfc_gemm_ws_size.argtypes = [i64, i64, i64, i32]
    lib.sfc_gemm_ws_size.restype = sz
    lib.sfc_gemm_plan.argtypes = [i64, i64, i64, i32, i32, ctypes.POINTER(ctypes.c_int64)]
    lib.sfc_gemm_plan.restype = i32
    lib.sfc_gemm_f8_plan.argtypes = [i64, i64, i64, i32, i32, ctypes.POINTER(ctypes.c_int64)]
    lib.sfc_gemm_f8_plan.restype = i32
    lib.sfc_gemm_model.argtypes = [i64, i64, i64, i32, i32, i32, i32, ctypes.POINTER(ctypes.c_int32),
                                   ctypes.POINTER(ctypes.c_int64)]
    lib.sfc_gemm_model.restype = i32
    lib.sfc_probe_mfma.argtypes = [i32, i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    lib.sfc_probe_mfma.restype = i32
    lib.sfc_strerror.argtypes = [i32]
    lib.sfc_strerror.restype = ctypes.c_char_p
    lib.sfc_last_error.argtypes = []
    lib.sfc_last_error.restype = ctypes.c_char_p
    lib.sfc_version.argtypes = []
    lib.sfc_version.restype = i32
    return lib


lib = _load()


def strerror(code: int) -> str:
    return lib.sfc_strerror(code).decode()


def last_error() -> str:
    return lib.sfc_last_error().decode()


def _check(code: int, what: str) -> None:
    if code != SFC_OK:
        raise SfcError(code, what)


def sfc_tile_order(gm: int, gn: int, order: str = "hilbert") -> np.ndarray:
    """Curve table of a gm x gn block grid: entry s = im*gn + in (host int32)."""
    out = np.empty(max(gm * gn, 1), dtype=np.int32)
    _check(lib.sfc_tile_order_ex(gm, gn, ORDERS[order], out.ctypes.data), "sfc_tile_order")
    return out[: gm * gn]


def sfc_gemm_ws_size(M: int, N: int, K: int, ca_layers: int) -> int:
    return int(lib.sfc_gemm_ws_size(M, N, K, ca_layers))


def sfc_gemm_plan(M: int, N: int, K: int, ca_layers: int = 1, tile: str = "auto") -> dict:
    plan = (ctypes.c_int64 * 7)()
    _check(lib.sfc_gemm_plan(M, N, K, ca_layers, TILES[tile], plan), "sfc_gemm_plan")
    keys = ["BM", "BN", "gm", "gn", "layers", "workgroups", "per_cu"]
    return dict(zip(keys, [int(v) for v in plan]))


def sfc_gemm_f8_plan(M: int, N: int, K: int, ca_layers: int = 1, tile: str = "auto") -> dict:
    """What sfc_gemm_f8_ex would launch (fp32 output), as sfc_gemm_plan."""
    plan = (ctypes.c_int64 * 7)()
    _check(lib.sfc_gemm_f8_plan(M, N, K, ca_layers, TILES[tile], plan), "sfc_gemm_f8_plan")
    keys = ["BM", "BN", "gm", "gn", "layers", "workgroups", "per_cu"]
    return dict(zip(keys, [int(v) for v in plan]))


def sfc_gemm_model(M: int, N: int, K: int, out: str = "f32", ca_layers: int = SFC_CA_AUTO,
                   tile: str = "auto", num_cus: int = 256, occupancy=(2, 1, 1, 1)) -> dict:
    """The model's (block shape, layer count) for given device parameters (host only)."""
    occ = (ctypes.c_int32 * 4)(*occupancy)
    ch = (ctypes.c_int64 * 3)()
    _check(lib.sfc_gemm_model(M, N, K, SFC_OUT_BF16 if out == "bf16" else SFC_OUT_F32, ca_layers, TILES[tile],
                              num_cus, occ, ch), "sfc_gemm_model")
    return {"tile": TILE_NAMES[int(ch[0])], "layers": int(ch[1]), "clk": int(ch[2])}


def sfc_probe_mfma(random_operands: bool = True, iterations: int = 20000) -> dict:
    """Register-only MFMA throughput and the shader clock during it."""
    tf, mhz = ctypes.c_double(), ctypes.c_double()
    _check(lib.sfc_probe_mfma(1 if random_operands else 0, iterations, ctypes.byref(tf), ctypes.byref(mhz)),
           "sfc_probe_mfma")
    return {"tflops": tf.value, "mhz": mhz.value}


def _matrix(t, name):
    """(pointer, rows, cols, ld) of a 2-D torch tensor with unit column stride."""
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    if t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError(f"{name} must have unit column stride")
    ld = t.stride(0) if t.shape[0] > 1 else max(t.shape[1], 1)
    return t.data_ptr(), t.shape[0], t.shape[1], ld


def _stream_handle(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _operands(A, B, C, what: str, in_types, in_name: str, out_types):
    """Checks shared by every GEMM wrapper, all made before the library is
    called: A (M, K), B (K, N) and C (M, N) are 2-D tensors with unit column
    stride and matching shapes, A and B hold `in_name` elements, C's dtype is
    one of `out_types`, and all three live on the current CUDA device.
    Returns (pa, lda, pb, ldb, pc, ldc, M, N, K, out_type)."""
    import torch
    for t, n in ((A, "A"), (B, "B"), (C, "C")):
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{what}: {n} must be a torch.Tensor")
    pa, M, K, lda = _matrix(A, "A")
    pb, K2, N, ldb = _matrix(B, "B")
    pc, M2, N2, ldc = _matrix(C, "C")
    if K2 != K or M2 != M or N2 != N:
        raise ValueError(f"{what}: shape mismatch: A {tuple(A.shape)} B {tuple(B.shape)} C {tuple(C.shape)}")
    for t, n in ((A, "A"), (B, "B")):
        if t.dtype not in in_types:
            raise TypeError(f"{what}: {n} must hold {in_name} (got {t.dtype})")
    if C.dtype not in out_types:
        raise TypeError(f"{what}: C must be " + " or ".join(str(d).replace("torch.", "") for d in out_types)
                        + f" (got {C.dtype})")
    out = SFC_OUT_F32 if C.dtype == torch.float32 else SFC_OUT_BF16
    for t, n in ((A, "A"), (B, "B"), (C, "C")):
        if not t.is_cuda:
            raise ValueError(f"{what}: {n} must be a CUDA tensor (got {t.device})")
    dev = torch.cuda.current_device()
    for t, n in ((A, "A"), (B, "B"), (C, "C")):
        if t.device.index != dev:
            raise ValueError(f"{what}: {n} is on {t.device}, the current device is cuda:{dev}")
    return pa, lda, pb, ldb, pc, ldc, M, N, K, out


def _bf16_types():
    import torch
    return (torch.bfloat16, torch.int16, torch.uint16)


def _f8_types():
    import torch
    return (torch.uint8, torch.int8, torch.float8_e4m3fn, torch.float8_e5m2)


def _out_types(*names):
    import torch
    return tuple(getattr(torch, n) for n in names)


def _workspace(workspace):
    if workspace is None:
        return None, 0
    if not workspace.is_cuda:
        raise ValueError("workspace must be a CUDA tensor")
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def sfc_gemm_ex(A, B, C, ca_layers: int = 1, tile: str = "auto", order: str = "hilbert",
                sched: str = "interleaved", workspace=None, stream=None) -> None:
    """C = A @ B on the GPU.  A: (M, K) bf16, B: (K, N) bf16, C: (M, N) float32
    or bfloat16 (the output type), all CUDA tensors with unit column stride."""
    pa, lda, pb, ldb, pc, ldc, M, N, K, out = _operands(A, B, C, "sfc_gemm_ex", _bf16_types(), "bf16 patterns",
                                                        _out_types("float32", "bfloat16"))
    ws_ptr, ws_bytes = _workspace(workspace)
    _check(lib.sfc_gemm_ex(M, N, K, pa, lda, pb, ldb, pc, ldc, out, ca_layers, TILES[tile],
                           ORDERS[order], SCHEDS[sched], ws_ptr, ws_bytes, _stream_handle(stream)),
           "sfc_gemm_ex")


def sfc_gemm_fused_ex(A, B, C, ca_layers: int = 1, tile: str = "auto", order: str = "hilbert",
                      sched: str = "interleaved", workspace=None, stream=None) -> None:
    """As sfc_gemm_ex, with the sum of the layer copies done inside the GEMM
    launch by the last workgroup to finish each block."""
    pa, lda, pb, ldb, pc, ldc, M, N, K, out = _operands(A, B, C, "sfc_gemm_fused_ex", _bf16_types(),
                                                        "bf16 patterns", _out_types("float32", "bfloat16"))
    ws_ptr, ws_bytes = _workspace(workspace)
    _check(lib.sfc_gemm_fused_ex(M, N, K, pa, lda, pb, ldb, pc, ldc, out, ca_layers, TILES[tile],
                                 ORDERS[order], SCHEDS[sched], ws_ptr, ws_bytes, _stream_handle(stream)),
           "sfc_gemm_fused_ex")


NOALLOC_WS_BYTES = 64 << 20
NOALLOC_MAX_BLOCKS = 1 << 17


def sfc_gemm_noalloc_ex(A, B, C, ca_layers: int = 1, tile: str = "auto", order: str = "hilbert",
                        sched: str = "interleaved", stream=None) -> None:
    """As sfc_gemm_ex without a workspace argument, for callers that cannot
    allocate: the library's static per-GPU array holds the layer copies (at
    most NOALLOC_WS_BYTES) and the curve tables.  Calls that overlap on one GPU
    race on that array."""
    pa, lda, pb, ldb, pc, ldc, M, N, K, out = _operands(A, B, C, "sfc_gemm_noalloc_ex", _bf16_types(),
                                                        "bf16 patterns", _out_types("float32", "bfloat16"))
    _check(lib.sfc_gemm_noalloc_ex(M, N, K, pa, lda, pb, ldb, pc, ldc, out, ca_layers, TILES[tile],
                                   ORDERS[order], SCHEDS[sched], _stream_handle(stream)),
           "sfc_gemm_noalloc_ex")


FP8_FORMATS = {"e4m3": 0, "e5m2": 1}


def sfc_gemm_f8_ex(A, B, C, ca_layers: int = 1, tile: str = "auto", order: str = "hilbert",
                   sched: str = "interleaved", workspace=None, stream=None, a_format: str = "e4m3",
                   b_format: str = "e4m3") -> None:
    """C = A @ B with OCP 8-bit float operands.  A: (M, K) and B: (K, N) CUDA
    tensors of fp8 bytes (torch.uint8, or torch.float8_e4m3fn / float8_e5m2),
    each in its format ("e4m3" or "e5m2"); C: (M, N) float32 or bfloat16, all
    with unit column stride.  Both formats E4M3 call sfc_gemm_f8_ex, any other
    pair sfc_gemm_f8_fmt_ex."""
    pa, lda, pb, ldb, pc, ldc, M, N, K, out = _operands(A, B, C, "sfc_gemm_f8_ex", _f8_types(), "fp8 bytes",
                                                        _out_types("float32", "bfloat16"))
    fa, fb = FP8_FORMATS[a_format], FP8_FORMATS[b_format]
    ws_ptr, ws_bytes = _workspace(workspace)
    if fa == 0 and fb == 0:
        _check(lib.sfc_gemm_f8_ex(M, N, K, pa, lda, pb, ldb, pc, ldc, out, ca_layers, TILES[tile],
                                  ORDERS[order], SCHEDS[sched], ws_ptr, ws_bytes, _stream_handle(stream)),
               "sfc_gemm_f8_ex")
    else:
        _check(lib.sfc_gemm_f8_fmt_ex(M, N, K, pa, lda, pb, ldb, pc, ldc, out, fa, fb, ca_layers, TILES[tile],
                                      ORDERS[order], SCHEDS[sched], ws_ptr, ws_bytes, _stream_handle(stream)),
               "sfc_gemm_f8_fmt_ex")


def to_device_u8(bits: np.ndarray, device="cuda"):
    """Upload a uint8 array (fp8 patterns) as a torch.uint8 CUDA tensor."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint8)).to(device)


def sfc_gemm(A, B, C, ca_layers: int = 1, stream=None) -> None:
    """C (float32) = A @ B with the default tile choice, curve order and schedule."""
    pa, lda, pb, ldb, pc, ldc, M, N, K, _ = _operands(A, B, C, "sfc_gemm", _bf16_types(), "bf16 patterns",
                                                      _out_types("float32"))
    _check(lib.sfc_gemm(M, N, K, pa, lda, pb, ldb, pc, ldc, ca_layers, _stream_handle(stream)), "sfc_gemm")


def sfc_gemm_bf16out(A, B, C, ca_layers: int = 1, stream=None) -> None:
    """C (bfloat16) = A @ B with the default tile choice, curve order and schedule."""
    pa, lda, pb, ldb, pc, ldc, M, N, K, _ = _operands(A, B, C, "sfc_gemm_bf16out", _bf16_types(),
                                                      "bf16 patterns", _out_types("bfloat16"))
    _check(lib.sfc_gemm_bf16out(M, N, K, pa, lda, pb, ldb, pc, ldc, ca_layers, _stream_handle(stream)),
           "sfc_gemm_bf16out")


def to_device_bf16(bits: np.ndarray, device="cuda"):
    """Upload a uint16 array of bf16 patterns as a torch.bfloat16 CUDA tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)
