"""Pins of the binary64 oracle against things other than itself: exhaustive
format tables from torch, dense brute force (numpy and torch's fp64
scaled_dot_product_attention), closed forms and invariants of attention, and
byte-level checks of the append.  ``test_mutants_are_caught`` plants plausible
mistakes in copies of the oracle source and checks that these pins catch each.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from tests import _dense as dn

ORACLE_C = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")


# ---------------------------------------------------------------- formats ---

def test_bf16_decode_exhaustive(oracle_lib):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = dn.bits_to_f64_bf16(bits)
    got = np.array([oracle_lib.oracle_bf16_to_f64(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def test_e4m3fn_decode_exhaustive(oracle_lib):
    codes = np.arange(256, dtype=np.uint16).astype(np.uint8)
    ref = dn.codes_to_f64_fp8(codes)
    got = np.array([oracle_lib.oracle_e4m3fn_to_f64(int(c)) for c in codes])
    nan = np.isnan(ref)
    assert nan.sum() == 2                      # 0x7F and 0xFF only
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert got[0x7E] == 448.0 and got[0x01] == 2.0 ** -9


# ----------------------------------------------------- dense brute force ---

SHAPES = [
    # B, H_q, H_kv, D, lens, kv
    (3, 8, 2, 64, [1, 17, 200], "bf16"),
    (4, 4, 4, 128, [16, 15, 33, 64], "bf16"),
    (2, 8, 1, 64, [31, 5], "bf16"),
    (3, 16, 2, 128, [1, 48, 129], "fp8"),
    (2, 4, 2, 64, [7, 40], "fp8"),
]


def _run(lib, case, scale, kv):
    kvd = oracle.BF16 if kv == "bf16" else oracle.FP8_E4M3FN
    return oracle.decode_attention(case["q_bits"], case["k_pages"], case["v_pages"],
                                   case["block_table"], case["seq_lens"], scale, kvd,
                                   case["k_scale"], case["v_scale"], lib=lib)


def pin_dense_numpy(lib):
    for i, (B, H_q, H_kv, D, lens, kv) in enumerate(SHAPES):
        rng = np.random.default_rng(100 + i)
        case = dn.random_case(rng, B, H_q, H_kv, D, lens, kv)
        scale = 1.0 / np.sqrt(D)
        got = _run(lib, case, scale, kv)
        ref = dn.dense_reference(case, scale, kv)
        err = np.abs(got - ref).max()
        if not err <= 1e-12:
            return f"dense numpy {i}: {err}"
    return None


def pin_dense_torch_sdpa(lib):
    for i, (B, H_q, H_kv, D, lens, kv) in enumerate(SHAPES):
        rng = np.random.default_rng(200 + i)
        case = dn.random_case(rng, B, H_q, H_kv, D, lens, kv)
        scale = float(np.float32(1.0 / np.sqrt(D)))
        got = _run(lib, case, scale, kv)
        q = torch.from_numpy(dn.bits_to_f64_bf16(case["q_bits"]))
        for b, L in enumerate(lens):
            if kv == "bf16":
                ks = dn.bits_to_f64_bf16(case["dense_k"][b])
                vs = dn.bits_to_f64_bf16(case["dense_v"][b])
            else:
                ks = dn.codes_to_f64_fp8(case["dense_k"][b]) * case["k_scale"][b][None, :, None].astype(np.float64)
                vs = dn.codes_to_f64_fp8(case["dense_v"][b]) * case["v_scale"][b][None, :, None].astype(np.float64)
            kt = torch.from_numpy(ks).permute(1, 0, 2)[None]      # [1, H_kv, L, D]
            vt = torch.from_numpy(vs).permute(1, 0, 2)[None]
            qt = q[b][None, :, None, :]                            # [1, H_q, 1, D]
            ref = F.scaled_dot_product_attention(qt, kt, vt, scale=scale, enable_gqa=True)[0, :, 0, :]
            err = (torch.from_numpy(got[b]) - ref).abs().max().item()
            if not err <= 1e-12:
                return f"sdpa {i} b={b}: {err}"
    return None


# ------------------------------------------------ closed forms/invariants ---

def _bf16_bits(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def pin_single_token(lib):
    rng = np.random.default_rng(1)
    case = dn.random_case(rng, 2, 8, 2, 64, [1, 1])
    got = _run(lib, case, 0.125, "bf16")
    for b in range(2):
        for h in range(8):
            v = dn.bits_to_f64_bf16(case["dense_v"][b][0, h // 4])
            if not np.array_equal(got[b, h], v):
                return f"single token b={b} h={h}"
    return None


def pin_constant_v(lib):
    rng = np.random.default_rng(2)
    case = dn.random_case(rng, 2, 8, 2, 64, [50, 77])
    const = _bf16_bits(rng.standard_normal((2, 2, 64)))
    for b in range(2):
        case["dense_v"][b][:] = const[b][None]
    kp, vp = dn.write_pools(case["dense_k"], case["dense_v"], [50, 77], case["page_lists"],
                            case["num_pages"], 2, 64, 8, np.uint16(0x7FC0))
    case["k_pages"], case["v_pages"] = kp, vp
    got = _run(lib, case, 0.125, "bf16")
    for b in range(2):
        for h in range(8):
            ref = dn.bits_to_f64_bf16(const[b][h // 4])
            if not np.abs(got[b, h] - ref).max() <= 1e-14:
                return f"constant v b={b} h={h}"
    return None


def pin_page_permutation(lib):
    rng = np.random.default_rng(3)
    lens = [37, 200, 16]
    case = dn.random_case(rng, 3, 8, 2, 64, lens)
    a = _run(lib, case, 0.125, "bf16")
    perm = rng.permutation(case["num_pages"]).astype(np.int32)       # new place of page p
    kp = np.empty_like(case["k_pages"])
    vp = np.empty_like(case["v_pages"])
    kp[perm] = case["k_pages"]
    vp[perm] = case["v_pages"]
    bt = case["block_table"].copy()
    bt[bt >= 0] = perm[bt[bt >= 0]]
    case2 = dict(case, k_pages=kp, v_pages=vp, block_table=bt)
    b = _run(lib, case2, 0.125, "bf16")
    return None if np.array_equal(a, b) else "page permutation"


def pin_weights_sum_to_one(lib):
    rng = np.random.default_rng(4)
    lens = [3, 100, 257]
    case = dn.random_case(rng, 3, 8, 2, 64, lens)
    one = _bf16_bits(np.ones(1))[0]
    for b in range(3):
        case["dense_v"][b][:, :, 5] = one
    kp, vp = dn.write_pools(case["dense_k"], case["dense_v"], lens, case["page_lists"],
                            case["num_pages"], 2, 64, 8, np.uint16(0x7FC0))
    case["k_pages"], case["v_pages"] = kp, vp
    got = _run(lib, case, 0.125, "bf16")
    err = np.abs(got[:, :, 5] - 1.0).max()
    return None if err <= 1e-13 else f"weights sum {err}"


def pin_scale_zero_is_mean(lib):
    rng = np.random.default_rng(5)
    lens = [9, 130]
    case = dn.random_case(rng, 2, 8, 2, 64, lens)
    got = _run(lib, case, 0.0, "bf16")
    for b, L in enumerate(lens):
        vs = dn.bits_to_f64_bf16(case["dense_v"][b])          # [L, H_kv, D]
        mean = vs.mean(axis=0)
        for h in range(8):
            if not np.abs(got[b, h] - mean[h // 4]).max() <= 1e-13:
                return f"scale 0 b={b} h={h}"
    return None


def pin_identical_keys_is_mean(lib):
    rng = np.random.default_rng(6)
    lens = [40, 3]
    case = dn.random_case(rng, 2, 8, 2, 64, lens)
    for b in range(2):
        case["dense_k"][b][:] = case["dense_k"][b][0][None]
    kp, vp = dn.write_pools(case["dense_k"], case["dense_v"], lens, case["page_lists"],
                            case["num_pages"], 2, 64, 8, np.uint16(0x7FC0))
    case["k_pages"], case["v_pages"] = kp, vp
    got = _run(lib, case, 0.125, "bf16")
    for b in range(2):
        mean = dn.bits_to_f64_bf16(case["dense_v"][b]).mean(axis=0)
        for h in range(8):
            if not np.abs(got[b, h] - mean[h // 4]).max() <= 1e-13:
                return f"identical keys b={b} h={h}"
    return None


def pin_batch_independence(lib):
    rng = np.random.default_rng(7)
    lens = [20, 300, 45]
    case = dn.random_case(rng, 3, 8, 2, 64, lens)
    full = _run(lib, case, 0.125, "bf16")
    for b in range(3):
        sub = dict(case, q_bits=case["q_bits"][b:b + 1], block_table=case["block_table"][b:b + 1],
                   seq_lens=case["seq_lens"][b:b + 1])
        one = _run(lib, sub, 0.125, "bf16")
        if not np.array_equal(one[0], full[b]):
            return f"batch independence b={b}"
    return None


def pin_two_tokens_closed_form(lib):
    """L = 2: out = sigmoid(s0 - s1) v0 + sigmoid(s1 - s0) v1, written out."""
    rng = np.random.default_rng(8)
    case = dn.random_case(rng, 1, 2, 1, 64, [2])
    scale = 0.125
    got = _run(lib, case, scale, "bf16")
    q = dn.bits_to_f64_bf16(case["q_bits"])[0]
    k = dn.bits_to_f64_bf16(case["dense_k"][0])[:, 0]
    v = dn.bits_to_f64_bf16(case["dense_v"][0])[:, 0]
    for h in range(2):
        s0 = scale * float(q[h] @ k[0])
        s1 = scale * float(q[h] @ k[1])
        a0 = 1.0 / (1.0 + np.exp(s1 - s0))
        ref = a0 * v[0] + (1.0 - a0) * v[1]
        if not np.abs(got[0, h] - ref).max() <= 1e-14:
            return f"two tokens h={h}"
    return None


def pin_large_scores(lib):
    """Scores in the hundreds: the weights must come from shifted exponentials
    (finite, close to one-hot), matching dense brute force."""
    rng = np.random.default_rng(10)
    lens = [40, 90]
    case = dn.random_case(rng, 2, 8, 2, 64, lens)
    scale = 60.0
    got = _run(lib, case, scale, "bf16")
    ref = dn.dense_reference(case, scale)
    if not np.all(np.isfinite(got)):
        return "large scores not finite"
    err = np.abs(got - ref).max()
    return None if err <= 1e-12 else f"large scores {err}"


def pin_zero_length(lib):
    rng = np.random.default_rng(9)
    case = dn.random_case(rng, 2, 4, 2, 64, [0, 5])
    got = _run(lib, case, 0.125, "bf16")
    return None if np.all(got[0] == 0.0) and np.all(np.isfinite(got[1])) else "zero length"


ATTENTION_PINS = [pin_dense_numpy, pin_dense_torch_sdpa, pin_single_token, pin_constant_v,
                  pin_page_permutation, pin_weights_sum_to_one, pin_scale_zero_is_mean,
                  pin_identical_keys_is_mean, pin_batch_independence, pin_two_tokens_closed_form,
                  pin_large_scores, pin_zero_length]


@pytest.mark.parametrize("pin", ATTENTION_PINS, ids=lambda f: f.__name__)
def test_attention_pin(oracle_lib, pin):
    assert pin(oracle_lib) is None


# -------------------------------------------------------------- append ----

def pin_append_bytes(lib, kv="bf16"):
    """Append into pools whose every byte is random poison: exactly the target
    slot's bytes change, to the new row's bytes, and lengths advance by one."""
    rng = np.random.default_rng(11)
    B, H_kv, D = 4, 2, 64
    x = 8 if kv == "bf16" else 16
    code = np.uint16 if kv == "bf16" else np.uint8
    NP, maxP = 24, 5
    lens = np.array([0, 15, 16, 63], dtype=np.int32)
    perm = rng.permutation(NP).astype(np.int32)
    bt = perm[:B * maxP].reshape(B, maxP).copy()
    info = np.iinfo(code)
    kp = rng.integers(0, info.max + 1, size=(NP, H_kv, D // x, 16, x)).astype(code)
    vp = rng.integers(0, info.max + 1, size=(NP, H_kv, D, 16)).astype(code)
    kn = rng.integers(0, info.max + 1, size=(B, H_kv, D)).astype(code)
    vn = rng.integers(0, info.max + 1, size=(B, H_kv, D)).astype(code)
    k0, v0, sl = kp.copy(), vp.copy(), lens.copy()
    oracle.kv_append(kn, vn, kp, vp, bt, sl, oracle.BF16 if kv == "bf16" else oracle.FP8_E4M3FN, lib=lib)
    if not np.array_equal(sl, lens + 1):
        return "lengths"
    kexp, vexp = k0.copy(), v0.copy()
    for b in range(B):
        pg, slot = bt[b, lens[b] // 16], lens[b] % 16
        kexp[pg, :, :, slot, :] = kn[b].reshape(H_kv, D // x, x)
        vexp[pg, :, :, slot] = vn[b]
    if not (np.array_equal(kp, kexp) and np.array_equal(vp, vexp)):
        return "pool bytes"
    return None


def pin_append_then_attend(lib):
    """Fill an all-NaN pool token by token with the append, then attend: equals
    dense attention over the appended rows."""
    rng = np.random.default_rng(12)
    B, H_q, H_kv, D = 2, 8, 2, 64
    lens = [19, 33]
    case = dn.random_case(rng, B, H_q, H_kv, D, lens)
    kp = np.full_like(case["k_pages"], 0x7FC0)
    vp = np.full_like(case["v_pages"], 0x7FC0)
    sl = np.zeros(B, dtype=np.int32)
    for t in range(max(lens)):
        active = [b for b in range(B) if t < lens[b]]
        kn = np.stack([case["dense_k"][b][t] for b in active])
        vn = np.stack([case["dense_v"][b][t] for b in active])
        sub_sl = sl[active].copy()
        oracle.kv_append(kn, vn, kp, vp, case["block_table"][active], sub_sl, lib=lib)
        sl[active] = sub_sl
    if not np.array_equal(sl, np.array(lens, dtype=np.int32)):
        return "append lengths"
    case2 = dict(case, k_pages=kp, v_pages=vp)
    got = _run(lib, case2, 0.125, "bf16")
    ref = dn.dense_reference(case, 0.125)
    err = np.abs(got - ref).max()
    return None if err <= 1e-12 else f"append then attend {err}"


APPEND_PINS = [pin_append_bytes, lambda lib: pin_append_bytes(lib, "fp8"), pin_append_then_attend]


@pytest.mark.parametrize("i", range(len(APPEND_PINS)))
def test_append_pin(oracle_lib, i):
    assert APPEND_PINS[i](oracle_lib) is None


def test_out_of_range_inputs_rejected(oracle_lib):
    rng = np.random.default_rng(13)
    case = dn.random_case(rng, 2, 4, 2, 64, [5, 20])
    bad = dict(case, block_table=case["block_table"].copy())
    bad["block_table"][1, 1] = case["num_pages"]
    with pytest.raises(ValueError):
        _run(oracle_lib, bad, 0.125, "bf16")
    bad = dict(case, seq_lens=np.array([5, 16 * case["block_table"].shape[1] + 1], dtype=np.int32))
    with pytest.raises(ValueError):
        _run(oracle_lib, bad, 0.125, "bf16")


# ------------------------------------------------------------- mutants ----

MUTANTS = {
    "gqa head modulo": ("const int g = h / G;", "const int g = h % H_kv;"),
    "drops last token": ("for (int t = 0; t < L; ++t) {\n        int64_t pg = block_table[(int64_t)b * max_pages + t / ORACLE_PAGE];\n        int slot = t % ORACLE_PAGE;\n        double w",
                         "for (int t = 0; t < L - 1; ++t) {\n        int64_t pg = block_table[(int64_t)b * max_pages + t / ORACLE_PAGE];\n        int slot = t % ORACLE_PAGE;\n        double w"),
    "scale ignored": ("s[t] = (double)scale * dot;", "s[t] = dot;"),
    "normalised by length": ("double w = s[t] / Z;", "double w = s[t] / L;"),
    "max taken from first score": ("if (s[t] > m)\n            m = s[t];", "if (s[t] > m)\n            m = m;"),
    "k chunk index transposed": ("return (chunk * ORACLE_PAGE + slot) * x + d % x;",
                                 "return (chunk * ORACLE_PAGE + (d % x) % ORACLE_PAGE) * x + slot % x;"),
    "v slot/dim swapped": ("return (tile * D + d) * ORACLE_PAGE + slot;",
                           "return tile * D * ORACLE_PAGE + slot * D + d;"),
    "fp8 exponent bias": ("mag = ldexp(1.0 + (double)m / 8.0, e - 7);", "mag = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    "fp8 subnormal": ("mag = ldexp((double)m / 8.0, 1 - 7);", "mag = ldexp((double)m / 8.0, -7);"),
    "v scale dropped": ("vs = (double)v_scale[(int64_t)b * H_kv + g];", "vs = 1.0;"),
    "append slot off by one": ("int slot = L % ORACLE_PAGE;\n        for (int g",
                               "int slot = (L + 1) % ORACLE_PAGE;\n        for (int g"),
    "append keeps length": ("seq_lens[b] = L + 1;", "seq_lens[b] = L;"),
}


def _all_pins(lib):
    fails = []
    for pin in ATTENTION_PINS + APPEND_PINS:
        try:
            r = pin(lib)
        except Exception as e:  # a crash in a mutant counts as caught
            r = f"raised {e!r}"
        if r is not None:
            fails.append(r)
    return fails


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutants_are_caught(name):
    src = open(ORACLE_C).read()
    old, new = MUTANTS[name]
    # a site shared by the decode and prefill entry points is mutated in both
    assert src.count(old) >= 1, f"mutation site for {name!r} not found"
    d = tempfile.mkdtemp()
    try:
        c = os.path.join(d, "m.c")
        so = os.path.join(d, "libm.so")
        open(c, "w").write(src.replace(old, new))
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-std=c99", "-shared", "-fPIC", c, "-o", so, "-lm"])
        lib = oracle.load(so)
        assert _all_pins(lib), f"mutant {name!r} passed every pin"
    finally:
        shutil.rmtree(d, ignore_errors=True)
