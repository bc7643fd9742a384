"""The C-ABI library loads, exports what include/sfcgemm.h declares, and its
host-side checks answer without a GPU (every call here fails validation or is
a no-op, so no HIP call is made)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sfcgemm.h")


@pytest.fixture(scope="module")
def sg():
    from paper_2601_16294_amd import sfcgemm
    return sfcgemm


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sfc_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(sg):
    declared = declared_functions()
    assert sorted(sg.EXPORTS) == declared
    out = subprocess.run(["nm", "-D", "--defined-only", sg.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (sfc_[a-z0-9_]+)", out))
    assert set(declared) <= exported
    for name in declared:
        assert hasattr(sg.lib, name)


def test_version_and_strings(sg):
    assert sg.lib.sfc_version() == 1
    assert sg.strerror(0) == "success"
    assert sg.strerror(-1) == "invalid argument"
    assert sg.strerror(-3) == "workspace too small"
    assert sg.strerror(12345) == "unknown error code"


@pytest.mark.parametrize("M,N,K,c,want", [
    (1024, 1024, 65536, 1, 0),
    (1024, 1024, 65536, 2, 2 * 1024 * 1024 * 4),
    (1024, 1024, 65536, 8, 8 * 1024 * 1024 * 4),
    (100, 50, 64, 4, 0),                 # one K block: one layer
    (100, 50, 130, 4, 3 * 100 * 50 * 4),  # three K blocks: three layers
    (100, 50, 0, 4, 0),
    (-1, 5, 5, 2, 0),
    (5, 5, 500, 0, 8 * 5 * 5 * 4),       # SFC_CA_AUTO: the model's largest count (16), capped at the 8 K blocks
    (5, 5, 1500, 0, 16 * 5 * 5 * 4),     # ... or the largest count itself
    (5, 5, 100, 0, 2 * 5 * 5 * 4),       # ... capped at the K blocks
    (5, 5, 500, -1, 0),
    (5, 5, 500, 65, 0),
])
def test_ws_size(sg, M, N, K, c, want):
    assert sg.sfc_gemm_ws_size(M, N, K, c) == want


F32, BF16 = 0, 1
GOOD = dict(M=64, N=64, K=64, A=4096, lda=64, B=8192, ldb=64, C=16384, ldc=64, out=F32, c=1,
            tile=0, order=0, sched=0, ws=None, wsb=0)


def call_ex(sg, **kw):
    a = dict(GOOD)
    a.update(kw)
    return sg.lib.sfc_gemm_ex(a["M"], a["N"], a["K"], a["A"], a["lda"], a["B"], a["ldb"], a["C"], a["ldc"],
                              a["out"], a["c"], a["tile"], a["order"], a["sched"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(M=-1), -1), (dict(N=-2), -1), (dict(K=-3), -1),
    (dict(lda=63), -1), (dict(ldb=63), -1), (dict(ldc=63), -1),
    (dict(A=None), -1), (dict(B=None), -1), (dict(C=None), -1),
    (dict(c=-1), -1), (dict(c=65), -1), (dict(out=2), -1),
    (dict(tile=5), -1), (dict(tile=-1), -1), (dict(order=2), -1), (dict(sched=3), -1),
    (dict(A=4097), -2), (dict(B=8193), -2), (dict(C=16386), -2),
    (dict(M=1 << 31), -2), (dict(K=1 << 31, lda=1 << 31), -2),
    (dict(c=2, K=128, lda=128, ws=1 << 20, wsb=2 * 64 * 64 * 4 - 1), -3),
    (dict(c=2, K=128, lda=128, ws=(1 << 20) + 8, wsb=1 << 20), -2),
    # SFC_CA_AUTO with a caller workspace: it must hold the largest count the
    # model picks (16 layers, here capped at the 4 K blocks)
    (dict(c=0, K=256, lda=256, ws=1 << 20, wsb=4 * 64 * 64 * 4 - 1), -3),
])
def test_invalid_arguments_rejected_before_any_launch(sg, kw, code):
    assert call_ex(sg, **kw) == code
    assert sg.last_error() != ""


def test_empty_output_is_a_noop(sg):
    assert call_ex(sg, M=0, C=None, A=None) == 0
    assert call_ex(sg, N=0, C=None, B=None) == 0
    assert sg.lib.sfc_gemm(0, 10, 10, None, 10, None, 10, None, 10, 1, None) == 0
    assert sg.lib.sfc_gemm_bf16out(5, 0, 10, None, 10, None, 10, None, 10, 1, None) == 0


def test_simple_entry_points_validate(sg):
    assert sg.lib.sfc_gemm(4, 4, 4, None, 4, 4096, 4, 8192, 4, 1, None) == -1
    assert sg.lib.sfc_gemm(4, 4, 4, 4096, 4, 4096, 4, 8192, 3, 1, None) == -1
    assert sg.lib.sfc_gemm_bf16out(4, 4, 4, 4096, 4, 4096, 4, 8192, 4, -1, None) == -1


@pytest.mark.parametrize("gm,gn,order,code", [(0, 4, 0, -1), (4, -1, 0, -1), (4, 4, 7, -1),
                                             (1 << 16, 1 << 16, 0, -2)])
def test_tile_order_validation(sg, gm, gn, order, code):
    buf = (ctypes.c_int32 * 16)()
    assert sg.lib.sfc_tile_order_ex(gm, gn, order, buf) == code
    assert sg.lib.sfc_tile_order(4, 4, None) == -1


def test_plan_validation(sg):
    plan = (ctypes.c_int64 * 7)()
    assert sg.lib.sfc_gemm_plan(0, 4, 4, 1, 0, plan) == -1
    assert sg.lib.sfc_gemm_plan(4, 4, 4, 1, 0, None) == -1
    assert sg.lib.sfc_gemm_f8_plan(0, 4, 4, 1, 0, plan) == -1
    assert sg.lib.sfc_gemm_f8_plan(4, 4, 4, 1, 0, None) == -1
    for tile in (1, 2, 5):   # fp8 runs 128x256 and 256x256 blocks only
        assert sg.lib.sfc_gemm_f8_plan(64, 64, 64, 1, tile, plan) == -1


def test_probe_validation(sg):
    d = ctypes.c_double()
    assert sg.lib.sfc_probe_mfma(1, 0, ctypes.byref(d), ctypes.byref(d)) == -1
    assert sg.lib.sfc_probe_mfma(1, 10, None, ctypes.byref(d)) == -1


F8GOOD = dict(M=64, N=64, K=64, A=4096, lda=64, B=8192, ldb=64, C=16384, ldc=64, out=F32, c=1,
              tile=0, order=0, sched=0, ws=None, wsb=0)


def call_f8(sg, **kw):
    a = dict(F8GOOD)
    a.update(kw)
    return sg.lib.sfc_gemm_f8_ex(a["M"], a["N"], a["K"], a["A"], a["lda"], a["B"], a["ldb"], a["C"], a["ldc"],
                                 a["out"], a["c"], a["tile"], a["order"], a["sched"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(M=-1), -1), (dict(lda=63), -1), (dict(ldb=63), -1), (dict(A=None), -1), (dict(out=2), -1),
    (dict(c=65), -1), (dict(tile=5), -1),
    (dict(K=40, lda=64), -2),                 # K not a multiple of 16
    (dict(N=40, ldb=64, ldc=64), -2),         # N not a multiple of 16
    (dict(lda=72), -2), (dict(ldb=72), -2),   # leading dimensions not multiples of 16
    (dict(A=4096 + 8), -2), (dict(B=8192 + 8), -2),   # rows not 16-byte aligned
    (dict(tile=1), -2), (dict(tile=2), -2),    # no 128x128 or 256x128 fp8 kernel
    (dict(lda=1 << 21), -2), (dict(ldb=1 << 23), -2),   # past the 32-bit per-lane offsets; no element path
    (dict(c=2, K=256, lda=256, ws=1 << 20, wsb=2 * 64 * 64 * 4 - 1), -3),
])
def test_f8_invalid_arguments_rejected_before_any_launch(sg, kw, code):
    assert call_f8(sg, **kw) == code
    assert sg.last_error() != ""


def test_f8_empty_output_is_a_noop(sg):
    assert call_f8(sg, M=0, C=None, A=None) == 0
    assert call_f8(sg, N=0, C=None, B=None) == 0


def test_f8_format_codes_validated(sg):
    args = (64, 64, 64, 4096, 64, 8192, 64, 16384, 64, F32)
    tail = (1, 0, 0, 0, None, 0, None)
    for fa, fb in ((2, 0), (0, 2), (-1, 0), (0, 5)):
        assert sg.lib.sfc_gemm_f8_fmt_ex(*args, fa, fb, *tail) == -1
        assert "format" in sg.last_error()
    # valid codes reach the other checks: a misaligned A is still rejected
    assert sg.lib.sfc_gemm_f8_fmt_ex(64, 64, 64, 4096 + 8, 64, 8192, 64, 16384, 64, F32, 1, 1, *tail) == -2


def call_noalloc(sg, **kw):
    a = dict(GOOD)
    a.update(kw)
    return sg.lib.sfc_gemm_noalloc_ex(a["M"], a["N"], a["K"], a["A"], a["lda"], a["B"], a["ldb"], a["C"], a["ldc"],
                                      a["out"], a["c"], a["tile"], a["order"], a["sched"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(M=-1), -1), (dict(lda=63), -1), (dict(C=None), -1), (dict(c=65), -1), (dict(tile=5), -1),
    (dict(A=4097), -2),
    # layer copies beyond the static workspace (64 MiB): 2 x 2048 x 4096 x 4 B = 64 MiB fits, one more row does not
    (dict(M=2049, N=4096, ldc=4096, ldb=4096, K=128, lda=128, c=2), -3),
    (dict(M=1024, N=1024, ldc=1024, ldb=1024, K=65536, lda=65536, c=17), -3),
    # SFC_CA_AUTO is checked at the largest count the model picks (16)
    (dict(M=1025, N=1024, ldc=1024, ldb=1024, K=65536, lda=65536, c=0), -3),
])
def test_noalloc_rejected_before_any_launch(sg, kw, code):
    assert call_noalloc(sg, **kw) == code
    assert sg.last_error() != ""
    if code == -3:
        assert "workspace holds" in sg.last_error()


def test_noalloc_empty_output_is_a_noop(sg):
    assert call_noalloc(sg, M=0, C=None, A=None) == 0
    assert call_noalloc(sg, N=0, C=None, B=None) == 0
    assert sg.NOALLOC_WS_BYTES == 64 << 20
