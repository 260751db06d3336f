"""Pins of the oracle's e4m3fn quantiser (used by the quantising append):
every bf16 input under several scales against torch's float8_e4m3fn cast of
the clamped binary32 quotient (torch rounds to nearest even but does not
saturate, hence the clamp), the format's corner values, the quantising
append's bytes, and planted mistakes."""
from __future__ import annotations

import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
import torch

import oracle

ORACLE_C = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")
SCALES = [1.0, 0.37, 1.0 / 448.0, 3.7e-3, 25.0, 2.0 ** -7]


def all_bf16_values():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()


def torch_codes(x, scale):
    # every bf16 pattern, inf and NaN included: their quotients are meant
    with np.errstate(over="ignore", invalid="ignore"):
        q = (x.astype(np.float32) / np.float32(scale)).astype(np.float32)
    t = torch.from_numpy(q).clamp(-448.0, 448.0).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy()


def oracle_codes(lib, x, scale):
    f = lib.oracle_quantize_e4m3fn
    return np.array([f(float(v), float(scale)) for v in x], dtype=np.uint8)


def pin_against_torch(lib):
    x = all_bf16_values()
    for s in SCALES:
        s32 = float(np.float32(s))
        got = oracle_codes(lib, x, s32)
        ref = torch_codes(x, s32)
        nan = np.isnan(x)
        if not np.array_equal(got[~nan], ref[~nan]):
            bad = np.nonzero(got[~nan] != ref[~nan])[0][:5]
            return f"scale {s}: {len(bad)} mismatches, e.g. x={x[~nan][bad]} got={got[~nan][bad]} ref={ref[~nan][bad]}"
        if not np.all((got[nan] & 0x7F) == 0x7F):
            return f"scale {s}: NaN not kept"
    return None


def pin_corners(lib):
    q = lambda v: lib.oracle_quantize_e4m3fn(float(v), 1.0)
    cases = [                              # (value, code); +0.0 and -0.0 both listed
        (0.0, 0x00), (-0.0, 0x80), (448.0, 0x7E), (1e30, 0x7E), (-1e30, 0xFE), (float("inf"), 0x7E),
        (464.0, 0x7E),                     # tie between 448 and 480: even mantissa, then saturation
        (2.0 ** -9, 0x01),                 # smallest subnormal
        (2.0 ** -10, 0x00),                # tie with zero: even
        (3 * 2.0 ** -10, 0x02),            # 1.5 ulp: tie to even (2)
        (2.0 ** -6, 0x08),                 # smallest normal
        (1.0, 0x38), (1.0625, 0x38),       # tie between 1 and 1.125: even (1)
        (1.1875, 0x3A),                    # tie between 1.125 and 1.25: even (1.25)
        (-2.5, 0xC2),
    ]
    for v, c in cases:
        if q(v) != c:
            return f"{v}: {q(v):#x} != {c:#x}"
    return None


def pin_append_quant_bytes(lib):
    rng = np.random.default_rng(31)
    B, H_kv, D, NP, maxP = 3, 2, 64, 12, 3
    lens = np.array([0, 17, 5], dtype=np.int32)
    bt = rng.permutation(NP).astype(np.int32)[:B * maxP].reshape(B, maxP).copy()
    kp = rng.integers(0, 256, size=(NP, H_kv, D // 16, 16, 16)).astype(np.uint8)
    vp = rng.integers(0, 256, size=(NP, H_kv, D, 16)).astype(np.uint8)
    kn = torch.from_numpy(rng.standard_normal((B, H_kv, D)).astype(np.float32) * 30).to(torch.bfloat16)
    vn = torch.from_numpy(rng.standard_normal((B, H_kv, D)).astype(np.float32) * 30).to(torch.bfloat16)
    ks = rng.uniform(0.01, 0.2, size=(B, H_kv)).astype(np.float32)
    vs = rng.uniform(0.01, 0.2, size=(B, H_kv)).astype(np.float32)
    k0, v0, sl = kp.copy(), vp.copy(), lens.copy()
    oracle.kv_append(kn.view(torch.int16).numpy().view(np.uint16), vn.view(torch.int16).numpy().view(np.uint16),
                     kp, vp, bt, sl, oracle.FP8_E4M3FN, ks, vs, lib=lib)
    if not np.array_equal(sl, lens + 1):
        return "lengths"
    kexp, vexp = k0.copy(), v0.copy()
    for b in range(B):
        pg, slot = bt[b, lens[b] // 16], lens[b] % 16
        for g in range(H_kv):
            kc = torch_codes(kn[b, g].float().numpy(), ks[b, g])
            vc = torch_codes(vn[b, g].float().numpy(), vs[b, g])
            kexp[pg, g, :, slot, :] = kc.reshape(D // 16, 16)
            vexp[pg, g, :, slot] = vc
    if not (np.array_equal(kp, kexp) and np.array_equal(vp, vexp)):
        return "pool bytes"
    return None


PINS = [pin_against_torch, pin_corners, pin_append_quant_bytes]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_quant_pin(oracle_lib, pin):
    assert pin(oracle_lib) is None


MUTANTS = {
    "no saturation": ("    if (a >= 448.0)\n        return (uint8_t)(sign | 0x7E);\n    if (a < ldexp(1.0, -6)) {\n        step",
                      "    if (a >= 480.0)\n        return (uint8_t)(sign | 0x7F);\n    if (a < ldexp(1.0, -6)) {\n        step"),
    "ties away from zero": ("if (r > 0.5 || (r == 0.5 && fmod(fl, 2.0) != 0.0))", "if (r >= 0.5)"),
    "truncation": ("if (r > 0.5 || (r == 0.5 && fmod(fl, 2.0) != 0.0))", "if (r > 1.0)"),
    "multiply by scale": ("float v = x / scale;", "float v = x * scale;"),
    "subnormal spacing": ("step = ldexp(1.0, -9);                         /* subnormal spacing */",
                          "step = ldexp(1.0, -8);                         /* subnormal spacing */"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_quant_mutants_are_caught(name):
    src = open(ORACLE_C).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name!r} not found exactly once"
    d = tempfile.mkdtemp()
    try:
        c = os.path.join(d, "m.c")
        so = os.path.join(d, "libm.so")
        open(c, "w").write(src.replace(old, new))
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-std=c99", "-shared", "-fPIC", c, "-o", so, "-lm"])
        lib = oracle.load(so)
        fails = [r for r in (p(lib) for p in PINS) if r is not None]
        assert fails, f"mutant {name!r} passed every pin"
    finally:
        shutil.rmtree(d, ignore_errors=True)
