"""Checks of the seeded input generators (shapes, length laws, poison,
page ownership).  They hold none of the attention arithmetic."""
from __future__ import annotations

import numpy as np
import torch

from paper_2510_15330_amd import workloads as wl


def test_tiny_layout_and_poison():
    w = wl.build("tiny", seed=0)
    assert list(w.lens0) == [0, 16, 199]
    assert w.num_pages == 64
    bt = w.block_table.numpy()
    used = bt[bt >= 0]
    assert len(used) == 16 and len(set(used.tolist())) == 16
    assert w.k_pages.shape == (64, 2, 8, 16, 8) and w.v_pages.shape == (64, 2, 64, 16)
    kb = w.k_pages.view(torch.int16).numpy().view(np.uint16)
    vb = w.v_pages.view(torch.int16).numpy().view(np.uint16)
    # request 1 has 16 tokens: page 0 full, page 1 empty (NaN) before the append
    p0, p1 = bt[1, 0], bt[1, 1]
    assert not np.any(kb[p0] == wl.BF16_NAN_BITS)
    assert np.all(kb[p1] == wl.BF16_NAN_BITS) and np.all(vb[p1] == wl.BF16_NAN_BITS)
    # unowned pages are all NaN
    free = sorted(set(range(64)) - set(used.tolist()))
    assert np.all(kb[free] == wl.BF16_NAN_BITS)
    # request 2: 199 tokens -> last page has 7 live slots
    last = bt[2, 12]
    assert np.all(vb[last][:, :, 7:] == wl.BF16_NAN_BITS)
    assert not np.any(vb[last][:, :, :7] == wl.BF16_NAN_BITS)


def test_tiny_other_reading():
    lens, _ = wl.sample_lengths("tiny", tiny_reading="before")
    assert list(lens) == [1, 17, 200]


def test_length_laws():
    lens, _ = wl.sample_lengths("llama3_8b", 0)
    assert lens.min() >= 1024 and lens.max() <= 4096 and len(lens) == 64
    lens, info = wl.sample_lengths("summarization", 0)
    assert np.all(info["prompt"] >= 6000) and np.all(info["prompt"] <= 12000)
    assert np.all(info["generated"] >= 1) and np.all(info["generated"] <= 1500)
    lc, ic = wl.sample_lengths("summarization_capped", 0)
    assert np.array_equal(ic["prompt"], info["prompt"])
    assert np.all(ic["generated_capped"] <= ic["cap"])
    assert set(np.unique(ic["cap"]).tolist()) <= {100, 200, 400}
    assert np.all(lc <= lens)
    lz, _ = wl.sample_lengths("stress_fp8", 0)
    assert lz.min() >= 127 and lz.max() <= 32767 and len(lz) == 512


def test_lognormal_law_statistics():
    # E[floor(exp(N(ln 500, 0.5^2)))] clipped at 1500 is about 561
    z = np.random.default_rng(1).standard_normal(400000)
    g = np.clip(np.floor(np.exp(np.log(500.0) + 0.5 * z)), 1, 1500)
    assert 555 < g.mean() < 568
    assert abs(np.median(g) - 499.5) < 3


def test_fp8_workload_small_pool():
    # exercise the fp8 path of the generator on a shrunken copy of the config
    cfg = dict(wl.CONFIGS["stress_fp8"])
    wl.CONFIGS["_fp8_small"] = dict(cfg, B=4)
    try:
        orig = wl.sample_lengths

        def fake(name, seed=0, tiny_reading="after"):
            if name == "_fp8_small":
                return np.array([5, 16, 40, 127], dtype=np.int64), {}
            return orig(name, seed, tiny_reading)
        wl.sample_lengths = fake
        w = wl.build("_fp8_small", seed=3, steps=2)
    finally:
        wl.sample_lengths = orig
        del wl.CONFIGS["_fp8_small"]
    assert w.k_pages.dtype == torch.uint8 and w.k_pages.shape[2:] == (8, 16, 16)
    assert w.k_scale.shape == (4, 8) and torch.all(w.k_scale > 0)
    vals = w.k_pages.view(torch.float8_e4m3fn).float()
    finite = vals[torch.isfinite(vals)]
    assert finite.abs().max() <= 448.0
    assert w.k_new.dtype == torch.uint8


def test_fp8_prompt_batch():
    # fp8 prompt batches: code pools in the decode layout, per-(request, head)
    # scales set by the cached tokens (1 where none is cached), the new rows
    # quantised at those scales, and empty slots holding the NaN code
    cached, new = [0, 33, 200], [40, 17, 128]
    w = wl.build_prefill(cached=cached, new=new, H_q=8, H_kv=2, D=128, seed=3, kv="fp8")
    assert w.kv == "fp8"
    assert w.k_pages.dtype == torch.uint8 and w.k_pages.shape[1:] == (2, 8, 16, 16)
    assert w.v_pages.dtype == torch.uint8 and w.v_pages.shape[1:] == (2, 128, 16)
    assert w.k_new.dtype == torch.uint8 and w.k_new.shape == (sum(new), 2, 128)
    assert w.k_scale.shape == (3, 2) and w.v_scale.shape == (3, 2)
    assert torch.all(w.k_scale[0] == 1.0) and torch.all(w.v_scale[0] == 1.0)
    assert torch.all(w.k_scale[1:] > 0) and torch.all(w.k_scale[1:] < 1.0)
    # cached slots of request 1: every code finite, and the amax code of each
    # head is the largest finite e4m3fn value (scale = amax / 448)
    bt = w.block_table.cpu().numpy()
    kp = w.k_pages.view(torch.float8_e4m3fn).float()
    for g in range(2):
        vals = torch.cat([kp[bt[1, p], g].permute(1, 0, 2).reshape(16, -1) for p in range(3)])[:33]
        assert torch.isfinite(vals).all()
        assert vals.abs().max() == 448.0
    # slots past every request's cached length hold the NaN code
    filled = set()
    for b, c in enumerate(cached):
        for t in range(c):
            filled.add((int(bt[b, t // 16]), t % 16))
    kc = w.k_pages.cpu().numpy()
    for p in range(w.k_pages.shape[0]):
        for sl in range(16):
            if (p, sl) not in filled:
                assert np.all(kc[p, :, :, sl, :] == wl.FP8_NAN_CODE)
    # the new rows: codes of N(0,1) values at the request's scale, so the
    # dequantised rows have unit-order spread
    kn = w.k_new.view(torch.float8_e4m3fn).float()
    rows = torch.repeat_interleave(torch.arange(3), torch.tensor(new))
    deq = kn * w.k_scale[rows][:, :, None]
    assert torch.isfinite(deq).all() and 0.5 < float(deq.std()) < 2.0
