"""The library's block-shape / layer-count model (sfc_gemm_model, host only)
against the oracle of the same model (oracle/model.py), on the configurations
of the benchmark and on seeded random shapes and device parameters.  The
choice must be identical; the estimate within 1e-9 relative."""
import numpy as np
import pytest

from oracle import model as om

SHAPE_OF = {"128x128": (128, 128), "256x128": (256, 128), "128x256": (128, 256), "256x256": (256, 256)}
NAME_OF = {v: k for k, v in SHAPE_OF.items()}


@pytest.fixture(scope="module")
def sg():
    from paper_2601_16294_amd import sfcgemm
    return sfcgemm


def _both(sg, M, N, K, out, layers, tile, cus, occ):
    lib = sg.sfc_gemm_model(M, N, K, out=out, ca_layers=layers, tile=tile, num_cus=cus,
                            occupancy=(occ[(128, 128)], occ[(256, 128)], occ[(128, 256)], occ[(256, 256)]))
    shape, c, clk = om.choose(M, N, K, out_bytes=2 if out == "bf16" else 4, num_cus=cus, occ=occ,
                              shape=None if tile == "auto" else SHAPE_OF[tile], layers=layers)
    return lib, (NAME_OF[shape], c, clk)


CONFIGS = [(512, 512, 512, "f32"), (8192, 8192, 8192, "bf16"), (3000, 7000, 2048, "f32"),
           (1024, 1024, 65536, "f32"), (4096, 4096, 4096, "bf16"), (4096, 14336, 4096, "bf16"),
           (4096, 4096, 14336, "bf16")]


@pytest.mark.parametrize("M,N,K,out", CONFIGS)
def test_benchmark_configs(sg, M, N, K, out):
    occ = {(128, 128): 2, (256, 128): 1, (128, 256): 1, (256, 256): 1}
    for layers in (0, 1, 2, 8):
        for tile in ("auto", "128x128", "256x256"):
            lib, ref = _both(sg, M, N, K, out, layers, tile, 256, occ)
            assert (lib["tile"], lib["layers"]) == ref[:2]
            assert lib["clk"] == pytest.approx(ref[2], rel=1e-9, abs=1.0)


def test_random_shapes_and_devices(sg):
    rng = np.random.default_rng(20260116)
    for _ in range(400):
        M, N = (int(x) for x in rng.integers(1, 20000, size=2))
        K = int(rng.choice([int(rng.integers(0, 300)), int(rng.integers(1, 70000))]))
        cus = int(rng.choice([1, 8, 80, 256, 304]))
        occ = {s: int(rng.integers(1, 3)) for s in SHAPE_OF.values()}
        out = "bf16" if rng.random() < 0.5 else "f32"
        layers = int(rng.choice([0, 0, 1, 3, 8, 64]))
        tile = str(rng.choice(["auto", "auto", "128x256", "256x128"]))
        lib, ref = _both(sg, M, N, K, out, layers, tile, cus, occ)
        assert (lib["tile"], lib["layers"]) == ref[:2], (M, N, K, out, layers, tile, cus, occ)
        assert lib["clk"] == pytest.approx(ref[2], rel=1e-9, abs=1.0)


def test_model_argument_checks(sg):
    import ctypes
    occ = (ctypes.c_int32 * 4)(1, 1, 1, 1)
    ch = (ctypes.c_int64 * 3)()
    assert sg.lib.sfc_gemm_model(-1, 4, 4, 0, 0, 0, 256, occ, ch) == -1
    assert sg.lib.sfc_gemm_model(4, 4, 4, 0, 0, 0, 0, occ, ch) == -1
    assert sg.lib.sfc_gemm_model(4, 4, 4, 0, 65, 0, 256, occ, ch) == -1
    assert sg.lib.sfc_gemm_model(4, 4, 4, 0, 0, 9, 256, occ, ch) == -1
    assert sg.lib.sfc_gemm_model(4, 4, 4, 0, 0, 0, 256, None, ch) == -1
    bad = (ctypes.c_int32 * 4)(1, 0, 1, 1)
    assert sg.lib.sfc_gemm_model(4, 4, 4, 0, 0, 0, 256, bad, ch) == -1
