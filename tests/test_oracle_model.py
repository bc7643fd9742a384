"""Pins of the block-shape / layer-count model oracle (oracle/model.py).

The model is the paper's Section III.B roofline (Eq. 1-4) evaluated over the
decompositions (Section III.C, second option), read for the GPU as the
oracle's docstring states.  The pins: Eq. 1 on hand-computed blocks, one whole estimate worked
out by hand, the M <-> N symmetry of the model, and the two facts the paper's
CA scheme rests on (Section II.C, Section IV.B): a K-dominant GEMM whose C grid
cannot fill the machine needs layers, a large square one does not.
"""
import pytest

from oracle import model as om


def test_eq1_compute_bound_block():
    # 256x256x64 block: 8,388,608 flops at 3031.04 flops per clock = 2767.5676 clk;
    # its panels (65,536 bytes) at 0.01 clk per byte = 655.36 clk
    g = 2 * 256 * 256 * 64
    assert g == 8388608
    t = om.brgemm_clk(g, 1 / 3031.04, 0.01, 32768, 32768)
    assert t == pytest.approx(2767.5676, rel=1e-7)


def test_eq1_memory_bound_block():
    # the same block with 0.1 clk per byte: 6553.6 clk of panel traffic
    t = om.brgemm_clk(8388608, 1 / 3031.04, 0.1, 32768, 32768)
    assert t == pytest.approx(6553.6, rel=1e-12)


def test_worked_estimate_kdominant_128x256_c8():
    # 1024 x 1024 x 65536, fp32 out, 128x256 blocks, 8 layers, 256 CUs, 1 per CU:
    # 8*4*8 = 256 tasks in 1 round; 1024 K blocks / 8 = 128 blocks per task;
    # block: 4,194,304 flops / (3031.04 * 0.86) = 1609.0509 clk (compute-bound:
    # panels 49,152 B * 256/3500 / sqrt(32) = 635.53 clk);
    # copies 2*8*1024*1024*4 + C 1024*1024*4 = 71,303,168 B / 3500 = 20,372.3 clk;
    # 2 launches = 20,000 clk.  Total 246,330.85 clk.
    occ = {(128, 128): 2, (256, 128): 1, (128, 256): 1, (256, 256): 1}
    clk, pad = om.estimate(1024, 1024, 65536, 4, 256, occ, (128, 256), 8)
    assert clk == pytest.approx(246330.85, rel=1e-8)
    assert pad == 256 * 128 * 256


@pytest.mark.parametrize("M,N,K", [(3000, 7000, 2048), (1024, 4096, 8192), (8192, 512, 65536), (777, 5000, 1000)])
def test_model_is_symmetric_in_m_and_n(M, N, K, monkeypatch):
    # the formula treats M and N alike; the calibrated rates of 128x256 and
    # 256x128 differ (two kernels), so the check runs with equal rates
    monkeypatch.setattr(om, "RATE", {**om.RATE, (256, 128): om.RATE[(128, 256)]})
    occ = {(128, 128): 2, (256, 128): 1, (128, 256): 1, (256, 256): 1}
    for (bm, bn) in om.SHAPES:
        for c in om.LAYERS:
            a = om.estimate(M, N, K, 4, 256, occ, (bm, bn), c)
            b = om.estimate(N, M, K, 4, 256, occ, (bn, bm), c)
            assert a[0] == pytest.approx(b[0], rel=1e-12) and a[1] == b[1]


def test_k_dominant_gemm_takes_layers():
    shape, c, _ = om.choose(1024, 1024, 65536, out_bytes=4)
    assert c > 1


def test_large_square_gemm_takes_one_layer():
    shape, c, _ = om.choose(8192, 8192, 8192, out_bytes=2)
    assert c == 1 and shape == (256, 256)


def test_fixed_knobs_are_respected():
    shape, c, _ = om.choose(1024, 1024, 65536, shape=(128, 128))
    assert shape == (128, 128)
    shape, c, _ = om.choose(1024, 1024, 65536, layers=2)
    assert c == 2
    # layer counts above the number of K blocks are capped
    shape, c, _ = om.choose(512, 512, 128, layers=8)
    assert c == 2


def test_ties_keep_the_first_candidate():
    # 256 x 256 x 64: every shape covers C exactly, one K block, c capped at 1;
    # 128x128 runs 4 tasks of a quarter of the work: no tie; but M = N = 0 makes
    # every candidate cost the same single launch, and the first shape wins
    shape, c, clk = om.choose(0, 0, 64)
    assert (shape, c) == ((256, 256), 1) and clk == om.LAUNCH_CLK


def test_worked_estimate_memory_bound():
    # 8192^3, fp32 out, 128x256 blocks, 1 layer, on a device of 4096 CUs:
    # 64*32 = 2048 tasks, all in flight (1 round), 256 per XCD (sqrt = 16);
    # block: panels 49,152 B * 2048/3500 / 16 = 1797.56 clk > compute 1609.05;
    # 128 blocks; C 8192*8192*4 B / 3500 = 76,695.4 clk; 1 launch.
    # Total 316,783.38 clk.
    occ = {(128, 128): 2, (256, 128): 1, (128, 256): 1, (256, 256): 1}
    clk, _ = om.estimate(8192, 8192, 8192, 4, 4096, occ, (128, 256), 1)
    assert clk == pytest.approx(316783.38, rel=1e-8)


def test_worked_estimate_grid_smaller_than_the_machine():
    # 512 x 512 x 512, fp32 out, 128x128 blocks, 1 layer, 256 CUs, 2 workgroups
    # per CU possible: 4*4 = 16 tasks, 1 round, 8 K blocks each.  16 workgroups
    # on 256 CUs have a CU each (w = min(2, ceil(16/256)) = 1):
    # block: 2,097,152 flops / (3031.04 * 0.60 = 1818.624) = 1153.15315 clk
    # (panels 32,768 B * 16/3500 / sqrt(16/8) = 105.92 clk: compute-bound);
    # 8 blocks = 9225.2252 clk; C 512*512*4 B / 3500 = 299.5931 clk; 1 launch.
    # Total 19,524.8184 clk.  Charged half a CU (w = 2), the same block would
    # take 2306.3 clk and the grid 28,749.7.
    occ = {(128, 128): 2, (256, 128): 1, (128, 256): 1, (256, 256): 1}
    clk, pad = om.estimate(512, 512, 512, 4, 256, occ, (128, 128), 1)
    assert clk == pytest.approx(19524.8184, rel=1e-8)
    assert pad == 16 * 128 * 128
    # 128x256 blocks: 8 tasks of 4,194,304 flops / (3031.04 * 0.86) = 1609.05 clk
    # per block: 10000 + 8 * 1609.05 + 299.59 = 23,172.0 clk -- slower, so the
    # model takes 128x128 here (the measured faster shape of this GEMM)
    clk2, _ = om.estimate(512, 512, 512, 4, 256, occ, (128, 256), 1)
    assert clk2 == pytest.approx(23172.0004, rel=1e-8)
    shape, c, _ = om.choose(512, 512, 512, out_bytes=4, occ=occ)
    assert shape == (128, 128) and c == 1
    # with more blocks than CUs two share a CU again
    clk3, _ = om.estimate(4096, 4096, 512, 4, 256, occ, (128, 128), 1)
    blk = 2097152 * 2 / 1818.624
    assert clk3 == pytest.approx(10000 + 2 * 8 * max(blk, 512 / 3500 * 32768 / 8) + 4096 * 4096 * 4 / 3500, rel=1e-9)
