"""The decode-attention work split on the host: the header the kernels
compile (paper_2510_15330_amd/csrc/work_split.h), built for the CPU, against
a plain restatement here.  Wave w of W takes the units [C(w) P / C(W),
C(w + 1) P / C(W)) (floors), C the cumulative weight, wave v weighing the
weight of its XCD (v / 4) mod 8, and the merge kernel must find, for every
unit x, the one wave whose range holds it.  The reference below sums the
weights one wave at a time and inverts the bounds by binary search; no
formula is shared with the header."""
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
    L.ws_in_force.argtypes = [P, i32, i32, P]
    L.ws_skew_weights.argtypes = [i32, P]
    L.ws_bounds.argtypes = [i32, i32, P, P]
    L.ws_waves.argtypes = [i32, i32, P, P, ctypes.c_long, P]
    L.ws_all_units.argtypes = [i32, i32, P]
    L.ws_all_units.restype = i32
    for f in (L.ws_in_force, L.ws_skew_weights, L.ws_bounds, L.ws_waves):
        f.restype = None
    return L


def arr(w):
    return np.ascontiguousarray(w, dtype=np.int32)


def skew_weights(k):
    return arr([256 - k if x % 2 else 256 + k for x in range(8)])


def ref_bounds(P, W, wts8):
    v = np.arange(W)
    wts = np.asarray(wts8, dtype=np.int64)[(v // 4) % 8]
    C = np.concatenate([[0], np.cumsum(wts)])          # at most 1023 W, times P < 2^31: fits int64
    return C * P // C[-1]


def lib_bounds(lib, P, W, w8):
    w8 = arr(w8)
    out = np.zeros(W + 1, dtype=np.int32)
    lib.ws_bounds(P, W, w8.ctypes.data, out.ctypes.data)
    return out.astype(np.int64)


def lib_waves(lib, P, W, w8, xs):
    w8 = arr(w8)
    xs = np.ascontiguousarray(xs, dtype=np.int32)
    out = np.zeros(len(xs), dtype=np.int32)
    lib.ws_waves(P, W, w8.ctypes.data, xs.ctypes.data, len(xs), out.ctypes.data)
    return out.astype(np.int64)


def check(lib, P, W, w8, xs=None):
    b = lib_bounds(lib, P, W, w8)
    ref = ref_bounds(P, W, w8)
    assert np.array_equal(b, ref), (P, W, list(w8))
    assert b[0] == 0 and b[W] == P and np.all(np.diff(b) >= 0)
    if xs is None:
        xs = np.arange(P)
    got = lib_waves(lib, P, W, w8, xs)
    want = np.searchsorted(ref, xs, side="right") - 1   # the last wave starting at or before x
    assert np.array_equal(got, want), (P, W, list(w8), xs[got != want][:5])
    # the wave found holds a non-empty range containing x
    assert np.all(b[got] <= xs) and np.all(xs < b[got + 1])
    # the merge's shortcut: when it says every wave holds units, they do
    w8a = arr(w8)
    if lib.ws_all_units(P, W, w8a.ctypes.data):
        assert np.all(np.diff(ref) >= 1), (P, W, list(w8))
    return got.size


def test_weights_apply_to_long_shares_only(lib):
    out = np.zeros(8, dtype=np.int32)
    lib.ws_skew_weights(10, out.ctypes.data)
    assert list(out) == [266, 246] * 4
    w8 = arr([300, 200, 280, 230, 256, 256, 400, 100])
    for W in (1, 7, 1024, 2048):
        lib.ws_in_force(w8.ctypes.data, 256 * W - 1, W, out.ctypes.data)
        assert len(set(out)) == 1
        lib.ws_in_force(w8.ctypes.data, 256 * W, W, out.ctypes.data)
        assert np.array_equal(out, w8)


WEIGHT_SETS = [skew_weights(k) for k in (0, 1, 10, 128, 255)] + [
    arr([300, 200, 280, 230, 256, 256, 400, 100]),
    arr([1] * 8), arr([1023] * 8), arr([1, 1023] * 4), arr([1023, 1, 1, 1, 1, 1, 1, 1]),
]


def test_exhaustive_small(lib):
    n = 0
    for w8 in WEIGHT_SETS:
        for W in range(1, 41):
            for P in range(1, 301):
                n += check(lib, P, W, w8)
    assert n > 4_000_000


def test_random_large(lib):
    rng = np.random.default_rng(0)
    n = 0
    for _ in range(1500):
        W = int(rng.integers(1, 16385))
        P = int(rng.integers(1, 2**31))
        pick = int(rng.integers(0, 3))
        w8 = (skew_weights(int(rng.integers(0, 256))) if pick == 0 else
              arr(rng.integers(1, 1024, 8)) if pick == 1 else arr(rng.integers(128, 513, 8)))
        b = ref_bounds(P, W, w8)
        # every range edge, its neighbours, and random units
        xs = np.concatenate([b[:-1], b[1:] - 1, np.minimum(b[:-1] + 1, P - 1), rng.integers(0, P, 64)])
        xs = np.unique(np.clip(xs, 0, P - 1))
        n += check(lib, P, W, w8, xs)
    assert n > 1_000_000


def test_device_shapes(lib):
    # the launch shapes: 256 CUs x 4 waves (one workgroup per CU) or x 8, on
    # the step counts of the summarization (~140k) and stress (~250k) batches
    for W in (1024, 2048):
        for P in (139_811, 256 * 1024, 262_144 + 7, 253_955):
            for w8 in (skew_weights(0), skew_weights(10), arr([278, 262, 252, 242, 248, 236, 268, 250])):
                check(lib, P, W, w8)
