"""Host-side planning rules that need no GPU (the half-height strip, the
deep-ring kernel choice), compiled with g++ straight from
the library's header-only checks (paper_2601_16294_amd/csrc/sfc_validate.h)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HARNESS = r'''
#include <stdio.h>
#include <stdlib.h>
#include "sfc_validate.h"
int main(int argc, char** argv) {
  for (int i = 1; i + 4 < argc; i += 5)
    printf("%d\n", sfc::strip_columns(atoi(argv[i]), atoi(argv[i + 1]), atoll(argv[i + 2]), atoll(argv[i + 3]),
                                      atoll(argv[i + 4])));
  return 0;
}
'''


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    d = tmp_path_factory.mktemp("rules")
    src, exe = d / "h.cpp", d / "h"
    src.write_text(HARNESS)
    subprocess.run(["g++", "-std=c++17", "-O1", f"-I{ROOT}/include", f"-I{ROOT}/paper_2601_16294_amd/csrc",
                    str(src), "-o", str(exe)], check=True)
    return str(exe)


def strip(harness, *cases):
    args = [str(v) for c in cases for v in c]
    out = subprocess.run([harness] + args, capture_output=True, text=True, check=True).stdout.split()
    return [int(x) for x in out]


def test_strip_columns(harness):
    # (gm, gn, slots, half_rows, half_slots) -> strip width in block columns
    cases = {
        (16, 56, 256, 32, 256): 8,    # 4096x14336 with 256x256 blocks: 3.5 rounds -> 3 + a half-height round
        (16, 64, 256, 32, 256): 0,    # whole rounds
        (16, 8, 256, 32, 256): 0,     # fewer blocks than workgroups
        (16, 60, 256, 32, 256): 0,    # last round 3/4 full
        (12, 28, 256, 24, 256): 7,    # 3000 rows: 80 blocks left over -> 7 columns of 24 half-height blocks
        (16, 55, 256, 32, 256): 7,    # 112 left over -> ceil(112/16) = 7
        (16, 56, 256, 40, 256): 0,    # the strip's half-height blocks would need two rounds
        (1, 300, 256, 2, 256): 44,    # one block row: r = 44 -> 44 columns of 2 half-height blocks
        (4, 65, 256, 8, 256): 1,      # r = 4 -> one column
        (0, 5, 256, 1, 256): 0,
    }
    assert strip(harness, *cases.keys()) == list(cases.values())


def test_strip_leaves_whole_rounds(harness):
    # whenever a strip is taken, the remaining blocks fit in floor(T/S) rounds
    # and the strip's half-height blocks in one round
    import itertools
    cases = [(gm, gn, 256, 2 * gm, 256) for gm, gn in itertools.product(range(1, 40), range(1, 80))]
    got = strip(harness, *cases)
    for (gm, gn, S, hr, hs), w in zip(cases, got):
        T = gm * gn
        if w == 0:
            continue
        assert 0 < w < gn
        assert gm * (gn - w) <= (T // S) * S
        assert hr * w <= hs
        assert 0 < T % S <= S // 2


DEEP = r'''
#include <stdio.h>
#include <stdlib.h>
#include "sfc_validate.h"
int main(int argc, char** argv) {
  for (int i = 1; i + 4 < argc; i += 5)
    printf("%d\n", (int)sfc::deep_ring(atoi(argv[i]), atoi(argv[i + 1]) != 0, atoi(argv[i + 2]), atoll(argv[i + 3]),
                                       atoll(argv[i + 4])));
  return 0;
}
'''


@pytest.fixture(scope="module")
def deep_harness(tmp_path_factory):
    d = tmp_path_factory.mktemp("deep")
    src, exe = d / "d.cpp", d / "d"
    src.write_text(DEEP)
    subprocess.run(["g++", "-std=c++17", "-O1", f"-I{ROOT}/include", f"-I{ROOT}/paper_2601_16294_amd/csrc",
                    str(src), "-o", str(exe)], check=True)
    return str(exe)


def test_deep_ring_rule(deep_harness):
    # (128x128 blocks?, fast path?, fp8?, tasks, CUs) -> the 4-deep ring kernel
    cases = {
        (1, 1, 0, 16, 256): 1,      # 512^3 at 128x128: 16 blocks on 256 CUs
        (1, 1, 0, 256, 256): 1,     # exactly one block per CU
        (1, 1, 0, 257, 256): 0,     # more blocks than CUs: two per CU at the 2-deep ring
        (1, 1, 0, 1320, 256): 0,
        (0, 1, 0, 16, 256): 0,      # other block shapes fill the LDS already
        (1, 0, 0, 16, 256): 0,      # element-load path
        (1, 1, 1, 16, 256): 0,      # fp8 operands have no 128x128 kernel
        (1, 1, 0, 0, 256): 0,
    }
    args = [str(v) for c in cases for v in c]
    out = subprocess.run([deep_harness] + args, capture_output=True, text=True, check=True).stdout.split()
    assert [int(x) for x in out] == list(cases.values())
