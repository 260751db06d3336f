"""Pins of the oracle's prompt (prefill) attention and prompt KV write against
things other than itself: dense causal attention in numpy and torch's fp64
scaled_dot_product_attention(is_causal=True), pools laid out by reshapes
(tests/_dense.py), and invariants.  ``test_prefill_mutants_are_caught``
plants plausible mistakes in copies of the oracle source."""
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

# B, H_q, H_kv, D, total lengths, query tokens per request (the last n of L)
CASES = [
    (2, 8, 2, 64, [40, 17], [40, 17]),        # whole prompts
    (3, 4, 1, 128, [33, 64, 5], [9, 64, 5]),   # a chunk after a cached prefix
    (1, 16, 2, 128, [130], [50]),
]


def _case(seed, B, H_q, H_kv, D, lens, nq, kv="bf16"):
    rng = np.random.default_rng(seed)
    c = dn.random_case(rng, B, H_q, H_kv, D, lens, kv)
    T = int(sum(nq))
    q = rng.standard_normal((T, H_q, D)).astype(np.float32)
    c["pq_bits"] = torch.from_numpy(q).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    c["q_start"] = np.concatenate([[0], np.cumsum(nq)]).astype(np.int32)
    return c


def _prefill(lib, c, scale):
    return oracle.prefill_attention(c["pq_bits"], c["k_pages"], c["v_pages"], c["block_table"],
                                    c["seq_lens"], c["q_start"], scale, lib=lib)


def pin_prefill_dense_numpy(lib):
    for i, (B, H_q, H_kv, D, lens, nq) in enumerate(CASES):
        c = _case(300 + i, B, H_q, H_kv, D, lens, nq)
        scale = 1.0 / np.sqrt(D)
        got = _prefill(lib, c, scale)
        q = dn.bits_to_f64_bf16(c["pq_bits"])
        for b in range(B):
            ks = dn.bits_to_f64_bf16(c["dense_k"][b])
            vs = dn.bits_to_f64_bf16(c["dense_v"][b])
            for j in range(nq[b]):
                t = c["q_start"][b] + j
                p = lens[b] - nq[b] + j                  # position of this query token
                ref = dn.dense_attention(q[t], ks[:p + 1], vs[:p + 1], scale)
                err = np.abs(got[t] - ref).max()
                if not err <= 1e-12:
                    return f"prefill dense case {i} b={b} j={j}: {err}"
    return None


def pin_prefill_dense_fp8(lib):
    # fp8 pools: codes decoded by torch's float8_e4m3fn, times the request's
    # per-head scales, then dense causal attention
    for i, (B, H_q, H_kv, D, lens, nq) in enumerate(CASES):
        c = _case(320 + i, B, H_q, H_kv, D, lens, nq, kv="fp8")
        scale = 1.0 / np.sqrt(D)
        got = oracle.prefill_attention(c["pq_bits"], c["k_pages"], c["v_pages"], c["block_table"], c["seq_lens"],
                                       c["q_start"], scale, kv_dtype=oracle.FP8_E4M3FN, k_scale=c["k_scale"],
                                       v_scale=c["v_scale"], lib=lib)
        q = dn.bits_to_f64_bf16(c["pq_bits"])
        for b in range(B):
            ks = dn.codes_to_f64_fp8(c["dense_k"][b]) * c["k_scale"][b][None, :, None].astype(np.float64)
            vs = dn.codes_to_f64_fp8(c["dense_v"][b]) * c["v_scale"][b][None, :, None].astype(np.float64)
            for j in range(nq[b]):
                t = c["q_start"][b] + j
                p = lens[b] - nq[b] + j
                ref = dn.dense_attention(q[t], ks[:p + 1], vs[:p + 1], scale)
                err = np.abs(got[t] - ref).max()
                if not err <= 1e-12:
                    return f"prefill fp8 dense case {i} b={b} j={j}: {err}"
    return None


def pin_prefill_torch_causal(lib):
    # whole prompts only (is_causal aligns the query with the keys' start)
    B, H_q, H_kv, D, lens, nq = CASES[0]
    c = _case(400, B, H_q, H_kv, D, lens, nq)
    scale = float(np.float32(1.0 / np.sqrt(D)))
    got = _prefill(lib, c, scale)
    q = torch.from_numpy(dn.bits_to_f64_bf16(c["pq_bits"]))
    for b in range(B):
        t0, t1 = c["q_start"][b], c["q_start"][b + 1]
        kt = torch.from_numpy(dn.bits_to_f64_bf16(c["dense_k"][b])).permute(1, 0, 2)[None]
        vt = torch.from_numpy(dn.bits_to_f64_bf16(c["dense_v"][b])).permute(1, 0, 2)[None]
        qt = q[t0:t1].permute(1, 0, 2)[None]
        ref = F.scaled_dot_product_attention(qt, kt, vt, scale=scale, is_causal=True, enable_gqa=True)
        err = (torch.from_numpy(got[t0:t1]) - ref[0].permute(1, 0, 2)).abs().max().item()
        if not err <= 1e-12:
            return f"sdpa causal b={b}: {err}"
    return None


def pin_first_token_is_its_value(lib):
    # position 0 attends only itself: the output is V row 0 exactly
    B, H_q, H_kv, D, lens, nq = CASES[0]
    c = _case(500, B, H_q, H_kv, D, lens, nq)
    got = _prefill(lib, c, 0.125)
    G = H_q // H_kv
    for b in range(B):
        v0 = dn.bits_to_f64_bf16(c["dense_v"][b][0])      # [H_kv, D]
        if not np.array_equal(got[c["q_start"][b]], np.repeat(v0, G, axis=0)):
            return f"first token b={b}"
    return None


def pin_future_tokens_ignored(lib):
    # changing the keys/values after a query's position leaves its output unchanged
    B, H_q, H_kv, D, lens, nq = CASES[2]
    c = _case(600, B, H_q, H_kv, D, lens, nq)
    base = _prefill(lib, c, 0.1)
    c2 = dict(c)
    c2["k_pages"] = c["k_pages"].copy()
    c2["v_pages"] = c["v_pages"].copy()
    last = c["block_table"][0][(lens[0] - 1) // 16]
    c2["k_pages"][last] ^= np.uint16(0x0101)               # perturb the last page of the prompt
    c2["v_pages"][last] ^= np.uint16(0x0101)
    pert = _prefill(lib, c2, 0.1)
    first_on_last_page = ((lens[0] - 1) // 16) * 16
    keep = [j for j in range(nq[0]) if lens[0] - nq[0] + j < first_on_last_page]
    if not keep or not np.array_equal(base[keep], pert[keep]):
        return "causal independence"
    if np.array_equal(base[-1], pert[-1]):
        return "perturbation not seen by the last token"
    return None


def pin_kv_write_bytes(lib):
    # write prompts (after a cached prefix) into poisoned pools; compare with
    # pools laid out by reshapes, and the rest stays poison
    rng = np.random.default_rng(700)
    B, H_kv, D = 3, 2, 64
    pre, add = [0, 20, 7], [33, 5, 16]
    total = [a + b for a, b in zip(pre, add)]
    need = [(L + 15) // 16 for L in total]
    NP = sum(need) + 3
    perm = rng.permutation(NP).astype(np.int32)
    lists, pos = [], 0
    for n in need:
        lists.append(perm[pos:pos + n])
        pos += n
    bt = dn.block_table_from(lists, max(need) + 1)
    rows_k = [rng.integers(0, 1 << 16, size=(L, H_kv, D)).astype(np.uint16) for L in total]
    rows_v = [rng.integers(0, 1 << 16, size=(L, H_kv, D)).astype(np.uint16) for L in total]
    poison = np.uint16(0x7FC1)
    ref_k, ref_v = dn.write_pools(rows_k, rows_v, total, lists, NP, H_kv, D, 8, poison)
    # the cached prefix is already in place; the write adds the rest
    kp, vp = dn.write_pools([r[:p] for r, p in zip(rows_k, pre)], [r[:p] for r, p in zip(rows_v, pre)],
                            pre, lists, NP, H_kv, D, 8, poison)
    seq = np.asarray(pre, dtype=np.int32)
    k_new = np.concatenate([r[p:] for r, p in zip(rows_k, pre)])
    v_new = np.concatenate([r[p:] for r, p in zip(rows_v, pre)])
    q_start = np.concatenate([[0], np.cumsum(add)]).astype(np.int32)
    oracle.kv_write(k_new, v_new, kp, vp, bt, seq, q_start, lib=lib)
    if not (np.array_equal(kp, ref_k) and np.array_equal(vp, ref_v)):
        return "prompt write bytes"
    if seq.tolist() != total:
        return f"lengths {seq.tolist()}"
    return None


PREFILL_PINS = [pin_prefill_dense_numpy, pin_prefill_dense_fp8, pin_prefill_torch_causal, pin_first_token_is_its_value,
                pin_future_tokens_ignored, pin_kv_write_bytes]


@pytest.mark.parametrize("pin", PREFILL_PINS, ids=lambda f: f.__name__)
def test_prefill_pins(oracle_lib, pin):
    assert pin(oracle_lib) is None


# the prefill loop's scale lookup (the decode loop has the same two lines;
# the call after them tells the two apart)
_FP8_SCALES = ("                ks = (double)k_scale[(int64_t)b * H_kv + g];\n"
               "                vs = (double)v_scale[(int64_t)b * H_kv + g];\n            }\n")
_PREFILL_CALL = "            if (attend(q + (i * H_q + h) * D"

PREFILL_MUTANTS = {
    "position ignores cached prefix": ("const int p = seq_lens[b] - n + (int)(i - q_start[b]);",
                                       "const int p = (int)(i - q_start[b]);"),
    "attends one token less": ("attend(q + (i * H_q + h) * D, b, g, p + 1,", "attend(q + (i * H_q + h) * D, b, g, p,"),
    "write position from zero": ("int pos = L + (int)(i - q_start[b]);", "int pos = (int)(i - q_start[b]);"),
    "write keeps length": ("seq_lens[b] = L + (q_start[b + 1] - q_start[b]);", "seq_lens[b] = L;"),
    "fp8 scales swapped": (_FP8_SCALES + _PREFILL_CALL,
                           _FP8_SCALES.replace("k_scale[", "@").replace("v_scale[", "k_scale[").replace("@", "v_scale[")
                           + _PREFILL_CALL),
    "fp8 scales of request 0": (_FP8_SCALES + _PREFILL_CALL,
                                _FP8_SCALES.replace("(int64_t)b * H_kv + g", "g") + _PREFILL_CALL),
}


@pytest.mark.parametrize("name", sorted(PREFILL_MUTANTS))
def test_prefill_mutants_are_caught(name):
    src = open(ORACLE_C).read()
    old, new = PREFILL_MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name!r} not found exactly once"
    d = tempfile.mkdtemp()
    try:
        c = os.path.join(d, "oracle.c")
        so = os.path.join(d, "liboracle_mut.so")
        open(c, "w").write(src.replace(old, new))
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-std=c99", "-shared", "-fPIC", c, "-o", so, "-lm"])
        lib = oracle.load(so)
        fails = []
        for pin in PREFILL_PINS:
            try:
                r = pin(lib)
            except Exception as e:  # a crash counts as caught
                r = repr(e)
            if r is not None:
                fails.append(r)
        assert fails, f"mutant {name!r} passed every prefill pin"
    finally:
        shutil.rmtree(d, ignore_errors=True)
