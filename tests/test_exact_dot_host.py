"""Host build of the GPU path's long-accumulator exact dot product, checked
against the oracle's exact router keys (an expansion sum, a different method)
and against exact rationals.  Runs on the CPU: the routine is plain C++."""
import ctypes
import os
import subprocess
import tempfile
from fractions import Fraction

import numpy as np
import pytest

import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR_DIR = os.path.join(ROOT, "paper_2505_00315_amd", "csrc")

SRC = r"""
#include "exact_dot.h"
extern "C" double t_dot_bf16(const uint16_t* x, const uint16_t* w, int n) { return mosa::exact_dot_bf16(x, w, n); }
extern "C" double t_dot_f32(const uint32_t* x, const uint32_t* w, int n) { return mosa::exact_dot_f32(x, w, n); }
"""


@pytest.fixture(scope="module")
def dotlib():
    d = tempfile.mkdtemp(prefix="mosa_exact_dot_")
    src = os.path.join(d, "t.cpp")
    so = os.path.join(d, "t.so")
    with open(src, "w") as f:
        f.write(SRC)
    subprocess.check_call(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-I", HDR_DIR, src, "-o", so])
    L = ctypes.CDLL(so)
    for n in ("t_dot_bf16", "t_dot_f32"):
        getattr(L, n).restype = ctypes.c_double
        getattr(L, n).argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    return L


def _dot(L, x, w):
    x, w = np.ascontiguousarray(x), np.ascontiguousarray(w)
    if x.dtype == np.uint16:
        return L.t_dot_bf16(x.ctypes.data, w.ctypes.data, x.size)
    return L.t_dot_f32(x.view(np.uint32).ctypes.data, w.view(np.uint32).ctypes.data, x.size)


def _exact(x, w):
    xf, wf = wl.as_f32(x).astype(np.float64), wl.as_f32(w).astype(np.float64)
    return float(sum((Fraction(float(a)) * Fraction(float(b)) for a, b in zip(xf, wf)), Fraction(0)))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_long_accumulator_matches_oracle_keys(orc, dotlib, dtype):
    rng = np.random.default_rng(3)
    X = rng.standard_normal((2, 50, 96)).astype(np.float32)
    W = (rng.standard_normal((3, 96)) / 10).astype(np.float32)
    if dtype == "bf16":
        X, W = wl.f32_to_bf16_bits(X), wl.f32_to_bf16_bits(W)
    keys = orc.router_keys(X, W)
    for b in range(2):
        for h in range(3):
            for t in range(50):
                assert _dot(dotlib, X[b, t], W[h]) == keys[b, h, t]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_long_accumulator_extreme_ranges(dotlib, dtype):
    rng = np.random.default_rng(8)
    for trial in range(400):
        n = int(rng.integers(1, 40))
        mant = rng.uniform(-2, 2, n)
        ex = rng.integers(-149 if dtype == "f32" else -133, 127, n)
        x = (mant * np.exp2(ex.astype(np.float64))).astype(np.float32)
        w = (rng.uniform(-2, 2, n) * np.exp2(rng.integers(-60, 60, n).astype(np.float64))).astype(np.float32)
        if trial % 3 == 0:  # exact cancellation plus a tiny remainder
            x = np.concatenate([x, -x[:-1]])
            w = np.concatenate([w, w[:-1]])
        if dtype == "bf16":
            x, w = wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(w)
        assert _dot(dotlib, x, w) == _exact(x, w)


def test_long_accumulator_ties_round_to_even(dotlib):
    # 2^53 + 1 (exactly half-way) rounds to even 2^53; 2^53 + 3 rounds up to 2^53 + 4.
    for extra, want in [(1.0, 2.0 ** 53), (3.0, 2.0 ** 53 + 4), (-1.0, 2.0 ** 53 - 1)]:
        x = np.array([2.0 ** 26, extra], dtype=np.float32)
        w = np.array([2.0 ** 27, 1.0], dtype=np.float32)
        assert _dot(dotlib, x, w) == want
    # sticky bit below the half-way point
    x = np.array([2.0 ** 26, 1.0, 2.0 ** -40], dtype=np.float32)
    w = np.array([2.0 ** 27, 1.0, 1.0], dtype=np.float32)
    assert _dot(dotlib, x, w) == 2.0 ** 53 + 2
