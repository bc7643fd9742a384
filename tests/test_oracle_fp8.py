"""Pins of the OCP FP8 E4M3 oracle (oracle/fp8.py): torch's float8_e4m3fn
conversion on every code, values fixed by the format's definition, ordering,
the exact bf16 encoding the GEMM oracle relies on, and planted mistakes."""
import math
import os
import types

import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import fp8 as of8

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CODES = np.arange(256, dtype=np.uint8)


def _fp8_pin_failures(mod):
    fails = []
    torch_vals = torch.from_numpy(CODES.copy()).view(torch.float8_e4m3fn).to(torch.float32).numpy().astype(np.float64)
    ours = np.array([mod.e4m3_value(int(c)) for c in CODES])
    same = (torch_vals == ours) | (np.isnan(torch_vals) & np.isnan(ours))
    if not same.all():
        fails.append(f"{int((~same).sum())} codes differ from torch")
    hand = {0x38: 1.0, 0xB8: -1.0, 0x7E: 448.0, 0x08: 2.0 ** -6, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9,
            0x40: 2.0, 0x3C: 1.5, 0x00: 0.0}
    for c, v in hand.items():
        if mod.e4m3_value(c) != v:
            fails.append(f"code {c:#x}")
    if not (math.copysign(1.0, mod.e4m3_value(0x80)) < 0 and mod.e4m3_value(0x80) == 0.0):
        fails.append("negative zero")
    if not (math.isnan(mod.e4m3_value(0x7F)) and math.isnan(mod.e4m3_value(0xFF))):
        fails.append("NaN codes")
    pos = [mod.e4m3_value(c) for c in range(0x7F)]
    if any(not (a < b) for a, b in zip(pos, pos[1:])):
        fails.append("positive codes not increasing")
    return fails


def test_oracle_passes_its_pins():
    assert _fp8_pin_failures(of8) == []


SRC = open(os.path.join(ROOT, "oracle", "fp8.py")).read()
MUTANTS = {
    "bias_8": ("* 2.0 ** (e - 7)", "* 2.0 ** (e - 8)"),
    "subnormal_exponent": ("(m / 8.0) * 2.0 ** -6", "(m / 8.0) * 2.0 ** -7"),
    "nan_on_exponent_only": ("if e == 0xF and m == 0x7:", "if e == 0xF:"),
    "mantissa_quarters": ("(1.0 + m / 8.0)", "(1.0 + m / 4.0)"),
    "sign_ignored": ("s = -1.0 if code & 0x80 else 1.0", "s = 1.0"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(name):
    old, new = MUTANTS[name]
    assert old in SRC
    mod = types.ModuleType("fp8_mutant_" + name)
    exec(compile(SRC.replace(old, new, 1), name, "exec"), mod.__dict__)
    assert _fp8_pin_failures(mod), f"mutant {name} passed every pin"


def test_every_value_is_exactly_a_bf16_value():
    ok = ~np.isnan(of8.e4m3_to_f64(CODES))
    back = obf16.bf16_to_f64(of8.e4m3_to_bf16_bits(CODES))
    assert np.array_equal(back[ok], of8.e4m3_to_f64(CODES)[ok])


def test_integers_up_to_16_are_exact():
    # the GPU tests' integer-valued inputs: |v| <= 16 round-trips through E4M3
    v = np.arange(-16, 17, dtype=np.float32)
    codes = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(of8.e4m3_to_f64(codes), v.astype(np.float64))


# ---- OCP E5M2 ---------------------------------------------------------------

def _e5m2_pin_failures(mod):
    fails = []
    torch_vals = torch.from_numpy(CODES.copy()).view(torch.float8_e5m2).to(torch.float32).numpy().astype(np.float64)
    ours = np.array([mod.e5m2_value(int(c)) for c in CODES])
    same = (torch_vals == ours) | (np.isnan(torch_vals) & np.isnan(ours))
    if not same.all():
        fails.append(f"{int((~same).sum())} codes differ from torch")
    hand = {0x3C: 1.0, 0xBC: -1.0, 0x7B: 57344.0, 0x04: 2.0 ** -14, 0x01: 2.0 ** -16, 0x03: 3 * 2.0 ** -16,
            0x40: 2.0, 0x3E: 1.5, 0x3D: 1.25, 0x00: 0.0, 0x7C: math.inf, 0xFC: -math.inf}
    for c, v in hand.items():
        if mod.e5m2_value(c) != v:
            fails.append(f"code {c:#x}")
    if not (math.copysign(1.0, mod.e5m2_value(0x80)) < 0 and mod.e5m2_value(0x80) == 0.0):
        fails.append("negative zero")
    if not all(math.isnan(mod.e5m2_value(c)) for c in (0x7D, 0x7E, 0x7F, 0xFD, 0xFE, 0xFF)):
        fails.append("NaN codes")
    pos = [mod.e5m2_value(c) for c in range(0x7D)]
    if any(not (a < b) for a, b in zip(pos, pos[1:])):
        fails.append("positive codes not increasing")
    return fails


def test_e5m2_oracle_passes_its_pins():
    assert _e5m2_pin_failures(of8) == []


MUTANTS5 = {
    "bias_16": ("* 2.0 ** (e - 15)", "* 2.0 ** (e - 16)"),
    "subnormal_exponent": ("(m / 4.0) * 2.0 ** -14", "(m / 4.0) * 2.0 ** -15"),
    "no_infinity": ("return s * float(\"inf\") if m == 0 else float(\"nan\")", "return float(\"nan\")"),
    "mantissa_eighths": ("(1.0 + m / 4.0)", "(1.0 + m / 8.0)"),
    "exponent_field_shift": ("e = (code >> 2) & 0x1F", "e = (code >> 3) & 0x1F"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS5))
def test_e5m2_planted_mistake_fails_a_pin(name):
    old, new = MUTANTS5[name]
    assert old in SRC
    mod = types.ModuleType("fp8_e5m2_mutant_" + name)
    exec(compile(SRC.replace(old, new, 1), name, "exec"), mod.__dict__)
    assert _e5m2_pin_failures(mod), f"mutant {name} passed every pin"


def test_every_e5m2_value_is_exactly_a_bf16_value():
    vals = of8.e5m2_to_f64(CODES)
    ok = ~np.isnan(vals)
    back = obf16.bf16_to_f64(of8.e5m2_to_bf16_bits(CODES))
    assert np.array_equal(back[ok], vals[ok])        # infinities included
    assert np.isnan(back[~ok]).all()


def test_e5m2_integers_up_to_8_are_exact():
    v = np.arange(-8, 9, dtype=np.float32)
    codes = torch.from_numpy(v).to(torch.float8_e5m2).view(torch.uint8).numpy()
    assert np.array_equal(of8.e5m2_to_f64(codes), v.astype(np.float64))
