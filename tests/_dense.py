"""Dense helpers for pinning the oracle: they write paged pools from dense
per-request K/V with reshapes and transposes (not with the oracle's offset
arithmetic) and compute attention densely with numpy in binary64."""
from __future__ import annotations

import numpy as np
import torch

PAGE = 16


def bits_to_f64_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).double().numpy()


def codes_to_f64_fp8(codes):
    return torch.from_numpy(np.ascontiguousarray(codes)).view(torch.float8_e4m3fn).double().numpy()


def write_pools(dense_k, dense_v, lens, page_lists, num_pages, H_kv, D, x, fill):
    """Scatter dense per-request rows into paged pools.

    dense_k[b], dense_v[b]: arrays [L_b, H_kv, D] of element codes.
    page_lists[b]: physical pages of request b in logical order.
    Layouts: K [NP, H_kv, D/x, 16, x], V [NP, H_kv, D, 16].
    """
    dt = dense_k[0].dtype
    kp = np.full((num_pages, H_kv, D // x, PAGE, x), fill, dtype=dt)
    vp = np.full((num_pages, H_kv, D, PAGE), fill, dtype=dt)
    for b, L in enumerate(lens):
        n = (L + PAGE - 1) // PAGE
        if n == 0:
            continue
        kk = np.full((n * PAGE, H_kv, D), fill, dtype=dt)
        vv = np.full((n * PAGE, H_kv, D), fill, dtype=dt)
        kk[:L] = dense_k[b]
        vv[:L] = dense_v[b]
        # [n, 16, H, D/x, x] -> [n, H, D/x, 16, x]
        kt = kk.reshape(n, PAGE, H_kv, D // x, x).transpose(0, 2, 3, 1, 4)
        # [n, 16, H, D] -> [n, H, D, 16]
        vt = vv.reshape(n, PAGE, H_kv, D).transpose(0, 2, 3, 1)
        pages = np.asarray(page_lists[b][:n])
        kp[pages] = kt
        vp[pages] = vt
    return kp, vp


def block_table_from(page_lists, max_pages):
    bt = np.full((len(page_lists), max_pages), -1, dtype=np.int32)
    for b, pl in enumerate(page_lists):
        bt[b, :len(pl)] = pl
    return bt


def dense_attention(q, ks, vs, scale):
    """q [H_q, D]; ks, vs [L, H_kv, D] (binary64) -> [H_q, D]; GQA h -> h // G."""
    H_q = q.shape[0]
    L, H_kv, D = ks.shape
    G = H_q // H_kv
    if L == 0:
        return np.zeros((H_q, D))
    kr = np.repeat(ks, G, axis=1)           # [L, H_q, D]
    vr = np.repeat(vs, G, axis=1)
    s = np.einsum("hd,lhd->hl", q, kr) * float(np.float32(scale))
    s = s - s.max(axis=1, keepdims=True)
    w = np.exp(s)
    w = w / w.sum(axis=1, keepdims=True)
    return np.einsum("hl,lhd->hd", w, vr)


def random_case(rng, B, H_q, H_kv, D, lens, kv="bf16", extra_pages=5):
    """Random dense rows + a scattered paged layout for them."""
    x = 8 if kv == "bf16" else 16
    need = [(L + PAGE - 1) // PAGE for L in lens]
    NP = sum(need) + extra_pages
    perm = rng.permutation(NP)
    page_lists, pos = [], 0
    for n in need:
        page_lists.append(perm[pos:pos + n].astype(np.int32))
        pos += n
    maxP = max(max(need), 1)
    if kv == "bf16":
        def draw(shape):
            f = torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(torch.bfloat16)
            return f.view(torch.int16).numpy().view(np.uint16)
        fill = np.uint16(0x7FC0)
        k_scale = v_scale = None
    else:
        def draw(shape):
            f = torch.from_numpy(rng.standard_normal(shape).astype(np.float32) * 40.0)
            return f.clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        fill = np.uint8(0x7F)
        k_scale = (rng.uniform(0.001, 0.1, size=(B, H_kv))).astype(np.float32)
        v_scale = (rng.uniform(0.001, 0.1, size=(B, H_kv))).astype(np.float32)
    dk = [draw((L, H_kv, D)) for L in lens]
    dv = [draw((L, H_kv, D)) for L in lens]
    q = torch.from_numpy(rng.standard_normal((B, H_q, D)).astype(np.float32)).to(torch.bfloat16)
    q_bits = q.view(torch.int16).numpy().view(np.uint16)
    kp, vp = write_pools(dk, dv, lens, page_lists, NP, H_kv, D, x, fill)
    bt = block_table_from(page_lists, maxP)
    return dict(q_bits=q_bits, dense_k=dk, dense_v=dv, k_pages=kp, v_pages=vp, block_table=bt,
                seq_lens=np.asarray(lens, dtype=np.int32), page_lists=page_lists, num_pages=NP,
                k_scale=k_scale, v_scale=v_scale, x=x)


def dense_reference(case, scale, kv="bf16"):
    """Binary64 dense attention for every request of a random_case."""
    q = bits_to_f64_bf16(case["q_bits"])
    out = []
    for b, L in enumerate(case["seq_lens"]):
        if kv == "bf16":
            ks = bits_to_f64_bf16(case["dense_k"][b])
            vs = bits_to_f64_bf16(case["dense_v"][b])
        else:
            ks = codes_to_f64_fp8(case["dense_k"][b]) * case["k_scale"][b][None, :, None].astype(np.float64)
            vs = codes_to_f64_fp8(case["dense_v"][b]) * case["v_scale"][b][None, :, None].astype(np.float64)
        out.append(dense_attention(q[b], ks, vs, scale))
    return np.stack(out)
