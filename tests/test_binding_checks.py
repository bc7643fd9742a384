"""The Python binding rejects bad operands before it calls the library: a wrong
dtype, a shape that does not chain (M x K times K x N into M x N), a tensor
that is not 2-D or has a non-unit column stride, and host (CPU) tensors.  No
GPU is needed: every case raises before any HIP call, so a bad argument can
never reach a kernel as an out-of-range pointer or a host address."""
import pytest
import torch

from paper_2601_16294_amd import sfcgemm as sg

M, N, K = 8, 16, 24


def t(rows, cols, dtype=torch.bfloat16):
    return torch.zeros((rows, cols), dtype=dtype)


GEMMS = [
    ("sfc_gemm", torch.float32),
    ("sfc_gemm_bf16out", torch.bfloat16),
    ("sfc_gemm_ex", torch.float32),
    ("sfc_gemm_ex", torch.bfloat16),
]


@pytest.mark.parametrize("fn,cdt", GEMMS)
def test_shape_mismatch_raises(fn, cdt):
    f = getattr(sg, fn)
    with pytest.raises(ValueError, match="shape mismatch"):
        f(t(M, K), t(K - 1, N), t(M, N, cdt))          # B has fewer rows than K
    with pytest.raises(ValueError, match="shape mismatch"):
        f(t(M, K), t(K, N), t(M + 1, N, cdt))
    with pytest.raises(ValueError, match="shape mismatch"):
        f(t(M, K), t(K, N), t(M, N - 1, cdt))


@pytest.mark.parametrize("fn,good,bad", [
    ("sfc_gemm", torch.float32, torch.bfloat16),       # a bf16 C would be written as fp32 rows
    ("sfc_gemm_bf16out", torch.bfloat16, torch.float32),
    ("sfc_gemm_ex", torch.float32, torch.float16),
])
def test_output_dtype_raises(fn, good, bad):
    f = getattr(sg, fn)
    with pytest.raises(TypeError, match="C must be"):
        f(t(M, K), t(K, N), t(M, N, bad))


@pytest.mark.parametrize("fn,cdt", GEMMS)
def test_operand_dtype_raises(fn, cdt):
    f = getattr(sg, fn)
    with pytest.raises(TypeError, match="A must hold"):
        f(t(M, K, torch.float32), t(K, N), t(M, N, cdt))
    with pytest.raises(TypeError, match="B must hold"):
        f(t(M, K), t(K, N, torch.float16), t(M, N, cdt))


@pytest.mark.parametrize("fn,cdt", GEMMS)
def test_host_tensors_raise(fn, cdt):
    f = getattr(sg, fn)
    with pytest.raises(ValueError, match="must be a CUDA tensor"):
        f(t(M, K), t(K, N), t(M, N, cdt))


@pytest.mark.parametrize("fn,cdt", GEMMS)
def test_layout_raises(fn, cdt):
    f = getattr(sg, fn)
    with pytest.raises(ValueError, match="2-D"):
        f(torch.zeros((1, M, K), dtype=torch.bfloat16), t(K, N), t(M, N, cdt))
    with pytest.raises(ValueError, match="unit column stride"):
        f(t(K, M).t(), t(K, N), t(M, N, cdt))
    with pytest.raises(TypeError, match="torch.Tensor"):
        f(None, t(K, N), t(M, N, cdt))


def test_fp8_wrapper_checks():
    u8 = torch.uint8
    with pytest.raises(TypeError, match="A must hold"):
        sg.sfc_gemm_f8_ex(t(M, K), t(K, N, u8), t(M, N, torch.float32))
    with pytest.raises(ValueError, match="shape mismatch"):
        sg.sfc_gemm_f8_ex(t(M, K, u8), t(K + 1, N, u8), t(M, N, torch.float32))
    with pytest.raises(TypeError, match="C must be"):
        sg.sfc_gemm_f8_ex(t(M, K, u8), t(K, N, u8), t(M, N, torch.int32))
    with pytest.raises(ValueError, match="must be a CUDA tensor"):
        sg.sfc_gemm_f8_ex(t(M, K, u8), t(K, N, u8), t(M, N, torch.float32))
