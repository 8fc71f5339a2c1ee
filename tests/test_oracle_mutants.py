"""Planted mistakes: each mutant of the oracle (a dropped term, a wrong sign
or index, a transposed operand) must fail at least one pin.  The mutants are
built on the CPU from a patched copy of the oracle's C source; nothing here
touches the GPU or the product library."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
from oracle import build as obuild

from test_oracle_pins import brute_force_int, tiny_cases

MUTANTS = {
    "filter_flipped": ("* R + r) * S + s]", "* R + (R - 1 - r)) * S + s]"),
    "bias_dropped": ("b ? b[k] : 0.0", "0.0"),
    "group_offset_dropped": ("(n * C + g * Cg + c)", "(n * C + c)"),
    "dilation_ignored_rows": ("+ r * dh", "+ r"),
    "pad_axes_swapped": ("p * sh - ph", "p * sh - pw"),
    "stride_axes_swapped": ("q * sw", "q * sh"),
    "relu_dropped": ("out[i] > 0.0 ? out[i] : 0.0", "out[i]"),
}


def _build_mutant(tmp_path, name, old, new):
    src = open(obuild.SRC).read()
    assert old in src, name
    mutated = src.replace(old, new)
    path = tmp_path / ("%s.c" % name)
    path.write_text(mutated)
    lib = tmp_path / ("lib%s.so" % name)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", str(path), "-o", str(lib)],
                   check=True)
    return str(lib)


def _pins_pass():
    for x, w, b, stride, pad, dil, G in tiny_cases(60, seed=11):
        ref = brute_force_int(x, w, b, stride, pad, dil, G)
        if not np.array_equal(oracle.conv2d(x, w, b, stride, pad, dil, G), ref):
            return False
        if not np.array_equal(oracle.conv2d(x, w, b, stride, pad, dil, G, relu=True), np.maximum(ref, 0)):
            return False
    return True


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_oracle_mistake(tmp_path, name, monkeypatch):
    old, new = MUTANTS[name]
    path = _build_mutant(tmp_path, name, old, new)
    saved = oracle._load()
    mutant = ctypes.CDLL(path)
    mutant.oracle_conv2d_f64.argtypes = saved.oracle_conv2d_f64.argtypes
    mutant.oracle_conv2d_f64.restype = ctypes.c_int
    mutant.oracle_conv2d_points_f64.argtypes = saved.oracle_conv2d_points_f64.argtypes
    mutant.oracle_conv2d_points_f64.restype = ctypes.c_int
    monkeypatch.setattr(oracle, "_lib", mutant)
    assert not _pins_pass(), "mutant %s survived the pins" % name


def test_unmutated_oracle_passes_the_same_pins():
    assert _pins_pass()


@pytest.mark.parametrize("which,index", [("WINO_BT", (1, 2)), ("WINO_G", (2, 1)), ("WINO_AT", (1, 3)),
                                         ("WINO_G", (1, 0))])
def test_winograd_pin_catches_wrong_matrix_entry(monkeypatch, which, index):
    m = getattr(oracle, which).copy()
    m[index] = -m[index] if m[index] != 0 else 1.0
    monkeypatch.setattr(oracle, which, m)
    rng = np.random.default_rng(12)
    x = rng.standard_normal((1, 3, 6, 6))
    w = rng.standard_normal((2, 3, 3, 3))
    got = oracle.winograd_conv2d(x, w, None, padding=1)
    ref = oracle.conv2d(x, w, None, 1, 1, 1)
    assert np.max(np.abs(got - ref)) > 1e-6
