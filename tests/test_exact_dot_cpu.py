"""The library's exact fallback for the transform (csrc/exact_dot.h), built for the host
with g++, against the oracle's rational definition of h = fl32(sum_j x_j T_jc)."""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest

from oracle import aatc as ora

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    d = tempfile.mkdtemp(prefix="aatc_exact_dot_")
    so = os.path.join(d, "libexactdot.so")
    subprocess.run(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-ffp-contract=off",
                    "-I", os.path.join(ROOT, "paper_2608_14191_amd", "csrc"),
                    os.path.join(ROOT, "tests", "native", "exact_dot_harness.cpp"), "-o", so],
                   check=True)
    L = ctypes.CDLL(so)
    L.exact_dot_q22_host.restype = ctypes.c_float
    L.exact_dot_q22_host.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    return L


def _call(L, x, tq):
    x = np.ascontiguousarray(x, dtype=np.float32)
    tq = np.ascontiguousarray(tq, dtype=np.int32)
    return np.float32(L.exact_dot_q22_host(x.ctypes.data, tq.ctypes.data, x.size))


def _want(x, tq):
    return ora.exact_dot_f32(np.asarray(x, np.float32),
                             np.ldexp(np.asarray(tq, np.float64), -22).astype(np.float32))


def _same(a, b):
    return (a == b and np.signbit(a) == np.signbit(b)) or (a == 0 and b == 0)


def test_near_ties_and_signs(lib):
    tq = np.array([1 << 22, 1, 1, 1], dtype=np.int32)
    for x in ([1.0, 0.25, 2.0 ** -40, 0.0], [1.0, 0.25, -2.0 ** -40, 0.0], [1.0, 0.25, 0, 0],
              [1.0, 0.75, 0, 0], [-1.0, -0.25, -2.0 ** -40, 0], [0, 0, 0, 0],
              [1.0, 0, 0, 0], [-3.0, 0, 0, 0]):
        got, want = _call(lib, x, tq), _want(x, tq)
        assert _same(got, want), (x, got, want)


def test_subnormal_and_extreme_ranges(lib):
    rng = np.random.default_rng(11)
    for trial in range(300):
        n = int(rng.integers(1, 129))
        e = rng.integers(-160, 100, n)
        x = (rng.standard_normal(n) * np.exp2(e)).astype(np.float32)
        if trial % 3 == 0:                               # subnormal inputs
            x[: n // 2] = (rng.standard_normal(n // 2) * 2.0 ** -140).astype(np.float32)
        tq = rng.integers(-(1 << 22), (1 << 22) + 1, n).astype(np.int32)
        if trial % 5 == 0:
            tq[:] = rng.integers(-3, 4, n)               # tiny transform entries
        got, want = _call(lib, x, tq), _want(x, tq)
        assert _same(got, want), (trial, got, want)


def test_cancellation_and_overflow(lib):
    rng = np.random.default_rng(12)
    for trial in range(200):
        n = 64
        x = (rng.standard_normal(n) * 2.0 ** rng.integers(-30, 30)).astype(np.float32)
        x = np.concatenate([x, -x]).astype(np.float32)          # exact cancellation ...
        tq = np.concatenate([rng.integers(-(1 << 22), 1 << 22, n)] * 2).astype(np.int32)
        x[int(rng.integers(0, 2 * n))] *= np.float32(1 + 2.0 ** -20)   # ... but for one
        got, want = _call(lib, x, tq), _want(x, tq)
        assert _same(got, want), (trial, got, want)
    big = np.full(128, 3.0e38, dtype=np.float32)
    assert np.isinf(_call(lib, big, np.full(128, 1 << 22, np.int32)))
