"""The decode-attention work split on the host: the header the kernels
compile (paper_2510_15330_amd/csrc/work_split.h), built for the CPU, against
a plain restatement here.  Wave w of W takes the units [C(w) P / C(W),
C(w + 1) P / C(W)) (floors), C the cumulative weight with 256 + k for the
waves of even-XCD workgroups (w / 4 even) and 256 - k for the others, and the
merge kernel must find, for every unit x, the one wave whose range holds it.
The reference below sums the weights one wave at a time and inverts the
bounds by binary search; no formula is shared with the header."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SHIM = os.path.join(ROOT, "tests", "native", "work_split_shim.cpp")


@pytest.fixture(scope="module")
def lib(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("ws") / "libws.so")
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    subprocess.check_call([hipcc, "-x", "hip", "--offload-host-only", "-O2", "-std=c++17", "-shared", "-fPIC",
                           SHIM, "-o", out])
    L = ctypes.CDLL(out)
    i32, P = ctypes.c_int, ctypes.c_void_p
    L.ws_skew.argtypes = [i32, i32, i32, i32]
    L.ws_skew.restype = i32
    L.ws_bounds.argtypes = [i32, i32, i32, P]
    L.ws_bounds.restype = None
    L.ws_waves.argtypes = [i32, i32, i32, P, ctypes.c_long, P]
    L.ws_waves.restype = None
    return L


def ref_bounds(P, W, skew):
    w = np.arange(W)
    wts = np.where((w // 4) % 2 == 0, 256 + skew, 256 - skew).astype(np.int64)
    C = np.concatenate([[0], np.cumsum(wts)])          # at most 2^9 W, times P < 2^31: fits int64
    return C * P // C[-1]


def lib_bounds(lib, P, W, skew):
    out = np.zeros(W + 1, dtype=np.int32)
    lib.ws_bounds(P, W, skew, out.ctypes.data)
    return out.astype(np.int64)


def lib_waves(lib, P, W, skew, xs):
    xs = np.ascontiguousarray(xs, dtype=np.int32)
    out = np.zeros(len(xs), dtype=np.int32)
    lib.ws_waves(P, W, skew, xs.ctypes.data, len(xs), out.ctypes.data)
    return out.astype(np.int64)


def check(lib, P, W, skew, xs=None):
    b = lib_bounds(lib, P, W, skew)
    ref = ref_bounds(P, W, skew)
    assert np.array_equal(b, ref), (P, W, skew)
    assert b[0] == 0 and b[W] == P and np.all(np.diff(b) >= 0)
    if xs is None:
        xs = np.arange(P)
    got = lib_waves(lib, P, W, skew, xs)
    want = np.searchsorted(ref, xs, side="right") - 1   # the last wave starting at or before x
    assert np.array_equal(got, want), (P, W, skew, xs[got != want][:5])
    # the wave found holds a non-empty range containing x
    assert np.all(b[got] <= xs) and np.all(xs < b[got + 1])
    return got.size


def test_skew_applies_to_long_shares_only(lib):
    # from 384 pages a wave: P steps of PP pages each
    for W in (1, 7, 1024, 2048):
        for PP in (1, 2, 4):
            n = 384 * W // PP + (1 if (384 * W) % PP else 0)   # fewest steps reaching 384 W pages
            assert lib.ws_skew(10, n - 1, W, PP) == 0
            assert lib.ws_skew(10, n, W, PP) == 10
        assert lib.ws_skew(0, 1 << 29, W, 4) == 0


def test_exhaustive_small(lib):
    n = 0
    for skew in (0, 1, 10, 128, 255):
        for W in range(1, 41):
            for P in range(1, 301):
                n += check(lib, P, W, skew)
    assert n > 2_000_000


def test_random_large(lib):
    rng = np.random.default_rng(0)
    n = 0
    for _ in range(1500):
        W = int(rng.integers(1, 16385))
        P = int(rng.integers(1, 2**31))
        skew = int(rng.choice([0, 10, int(rng.integers(0, 256))]))
        b = ref_bounds(P, W, skew)
        # every range edge, its neighbours, and random units
        xs = np.concatenate([b[:-1], b[1:] - 1, np.minimum(b[:-1] + 1, P - 1), rng.integers(0, P, 64)])
        xs = np.unique(np.clip(xs, 0, P - 1))
        n += check(lib, P, W, skew, xs)
    assert n > 1_000_000


def test_device_shapes(lib):
    # the launch shapes: 256 CUs x 4 waves (one workgroup per CU) or x 8, on
    # the step counts of the summarization (~140k) and stress (~250k) batches
    for W in (1024, 2048):
        for P in (139_811, 256 * 1024, 262_144 + 7, 253_955):
            for skew in (0, 10):
                check(lib, P, W, skew)
