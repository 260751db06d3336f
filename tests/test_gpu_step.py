"""The fused decode step (bellman_decode_step) on the GPU: the append and the
attention over the grown cache in two launches.  Checked against the
oracle's two calls (append, then attention): pools byte for byte, lengths,
and attention element by element within the bf16 / fp8 bounds, on the tiny
and Llama-3-8B-shaped workloads (every step), the full-size summarization
and fp8 stress batches (whole output), and a seeded sweep of shapes, length
mixes at page edges (the new token opening a page, empty requests) and
launch knobs, with fp8 codes and bf16 rows quantised into fp8 pools; and
against the library's own two calls on malformed slots."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from tests import _dense as dn
from tests import _gpu as G

pytestmark = pytest.mark.gpu

bl = pytest.importorskip("paper_2510_15330_amd")
from paper_2510_15330_amd import workloads as wl  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bl.library()
    yield
    torch.cuda.synchronize()


def step_workload(w, s, out, **kw):
    bl.decode_step(w.q[s], w.k_new[s], w.v_new[s], w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.scale, out,
                   k_scale=w.k_scale, v_scale=w.v_scale, **kw)


@pytest.mark.parametrize("reading", ["after", "before"])
def test_step_tiny(reading):
    w = G.to_device(wl.build("tiny", seed=0, tiny_reading=reading))
    kp, vp = G.bits16(w.k_pages), G.bits16(w.v_pages)
    sl = w.seq_lens.cpu().numpy().astype(np.int32)
    bt = w.block_table.cpu().numpy()
    oracle.kv_append(G.bits16(w.k_new[0]), G.bits16(w.v_new[0]), kp, vp, bt, sl)
    ref = oracle.decode_attention(G.bits16(w.q[0]), kp, vp, bt, sl, w.scale)
    out = torch.full((w.B, w.H_q, w.D), float("nan"), dtype=torch.bfloat16, device="cuda")
    step_workload(w, 0, out)
    torch.cuda.synchronize()
    assert bl.device_errors() == 0
    assert np.array_equal(w.seq_lens.cpu().numpy(), sl)
    assert np.array_equal(G.bits16(w.k_pages), kp) and np.array_equal(G.bits16(w.v_pages), vp)
    G.assert_close(G.out_f64(out), ref, "bf16", f"step tiny/{reading}")


def test_step_llama3_8b_every_step():
    w = G.to_device(wl.build("llama3_8b", seed=0))
    kp, vp = G.bits16(w.k_pages), G.bits16(w.v_pages)
    sl = w.seq_lens.cpu().numpy().astype(np.int32)
    bt = w.block_table.cpu().numpy()
    out = torch.empty((w.B, w.H_q, w.D), dtype=torch.bfloat16, device="cuda")
    for s in range(w.steps):
        step_workload(w, s, out)
        oracle.kv_append(G.bits16(w.k_new[s]), G.bits16(w.v_new[s]), kp, vp, bt, sl)
        torch.cuda.synchronize()
        ref = oracle.decode_attention(G.bits16(w.q[s]), kp, vp, bt, sl, w.scale)
        G.assert_close(G.out_f64(out), ref, "bf16", f"step llama3_8b step {s}")
    assert bl.device_errors() == 0
    assert np.array_equal(w.seq_lens.cpu().numpy(), sl)
    assert np.array_equal(G.bits16(w.k_pages), kp), "K pool differs after 100 fused steps"
    assert np.array_equal(G.bits16(w.v_pages), vp), "V pool differs after 100 fused steps"


@pytest.mark.parametrize("name", ["summarization", "stress_fp8"])
def test_step_full_size_first_step(name):
    w = wl.build(name, seed=0, device="cuda", steps=1)
    out = torch.full((w.B, w.H_q, w.D), float("nan"), dtype=torch.bfloat16, device="cuda")
    L0 = w.seq_lens.cpu().numpy().copy()
    step_workload(w, 0, out)
    torch.cuda.synchronize()
    assert bl.device_errors() == 0
    assert np.array_equal(w.seq_lens.cpu().numpy(), L0 + 1)
    ref = G.oracle_full(w, 0)
    G.assert_close(G.out_f64(out), ref, w.kv, f"step {name} step 0, all {w.B} requests")


def _lens(rng, B):
    out = []
    for _ in range(B):
        kind = rng.integers(0, 5)
        k = int(rng.integers(1, 10))
        if kind == 0:
            out.append(0)                                  # the new token alone
        elif kind == 1:
            out.append(16 * k + int(rng.integers(-1, 1)))   # the new token opens a page, or fills one
        elif kind == 2:
            out.append(64 * k + int(rng.integers(-1, 2)))
        else:
            out.append(int(rng.integers(1, 900)))
    return out


def _new_rows(rng, B, H_kv, D, kv, quant):
    if kv == "bf16" or quant:
        x = torch.from_numpy(rng.standard_normal((B, H_kv, D)).astype(np.float32) * (0.05 if quant else 1.0))
        return x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    x = torch.from_numpy(rng.standard_normal((B, H_kv, D)).astype(np.float32) * 40.0)
    return x.clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _dev_rows(a):
    t = torch.from_numpy(np.ascontiguousarray(a.view(np.int16) if a.dtype == np.uint16 else a)).cuda()
    return t.view(torch.bfloat16) if a.dtype == np.uint16 else t


@pytest.mark.parametrize("seed", range(16))
def test_step_random_sweep(seed):
    rng = np.random.default_rng(6000 + seed)
    kv = ["bf16", "fp8", "fp8"][seed % 3]
    quant = kv == "fp8" and seed % 2 == 0
    D = 64 if seed % 4 == 1 else 128
    H_kv = int(rng.choice([1, 2, 4, 8]))
    Gq = int(rng.choice([1, 2, 4, 8, 16]))
    B = int(rng.integers(1, 20))
    lens = _lens(rng, B)
    case = dn.random_case(rng, B, Gq * H_kv, H_kv, D, [L + 1 for L in lens], kv)   # pages for the new token
    if kv == "fp8":
        case["k_scale"] = (rng.uniform(0.5, 1.5, size=(B, H_kv)) / 40.0).astype(np.float32)
        case["v_scale"] = (rng.uniform(0.5, 1.5, size=(B, H_kv)) / 40.0).astype(np.float32)
    sl0 = np.asarray(lens, dtype=np.int32)
    kn, vn = _new_rows(rng, B, H_kv, D, kv, quant), _new_rows(rng, B, H_kv, D, kv, quant)
    scale = float(np.float32(1.0 / np.sqrt(D)))
    kcode = G.kv_code(kv)
    kp, vp, sl = case["k_pages"].copy(), case["v_pages"].copy(), sl0.copy()
    oracle.kv_append(kn, vn, kp, vp, case["block_table"], sl, kcode, case["k_scale"], case["v_scale"])
    ref = oracle.decode_attention(case["q_bits"], kp, vp, case["block_table"], sl, scale, kcode,
                                  case["k_scale"], case["v_scale"])
    waves = int(rng.choice([0, 1, 3, 8, 33]))
    pps = int(rng.choice([1, 2, 4] if kv == "fp8" else [1, 2]))
    depth = int(rng.choice([1, 2]))
    what = (f"step sweep seed={seed} {kv}{' quant' if quant else ''} B={B} G={Gq} H_kv={H_kv} D={D} "
            f"lens={lens} waves={waves} pages/step={pps} depth={depth}")
    d = {k: torch.from_numpy(v).cuda() if isinstance(v, np.ndarray) else None
         for k, v in (("bt", case["block_table"]), ("sl", sl0), ("ks", case["k_scale"]), ("vs", case["v_scale"]))}
    if kv == "bf16":
        kpd = torch.from_numpy(case["k_pages"].view(np.int16)).view(torch.bfloat16).cuda()
        vpd = torch.from_numpy(case["v_pages"].view(np.int16)).view(torch.bfloat16).cuda()
    else:
        kpd, vpd = torch.from_numpy(case["k_pages"]).cuda(), torch.from_numpy(case["v_pages"]).cuda()
    q = torch.from_numpy(case["q_bits"].view(np.int16)).view(torch.bfloat16).cuda()
    out = torch.full((B, Gq * H_kv, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    bl.decode_step(q, _dev_rows(kn), _dev_rows(vn), kpd, vpd, d["bt"], d["sl"], scale, out, k_scale=d["ks"],
                   v_scale=d["vs"], max_waves=waves, pages_per_step=pps, pipeline_depth=depth)
    torch.cuda.synchronize()
    assert bl.device_errors() == 0, what
    assert np.array_equal(d["sl"].cpu().numpy(), sl), what
    host = (lambda t: G.bits16(t)) if kv == "bf16" else (lambda t: t.cpu().numpy())
    assert np.array_equal(host(kpd), kp) and np.array_equal(host(vpd), vp), f"pools: {what}"
    G.assert_close(G.out_f64(out), ref, kv, what)


def test_step_malformed_slots_match_two_calls():
    """A request whose table is full (no slot for the new token) and one whose
    new page's entry lies outside the pool: no append, length kept, flag 1,
    and the attention over the cached tokens, as the two calls give."""
    rng = np.random.default_rng(61)
    lens = [32, 47, 112]
    case = dn.random_case(rng, 3, 8, 2, 64, [33, 48, 112])
    bt = case["block_table"].copy()
    bt[0, 2] = case["num_pages"] + 7            # request 0's new token opens page 2: outside the pool
    maxL = bt.shape[1] * 16
    assert maxL == 112                          # request 2 fills its table: no slot left
    sl = np.asarray(lens, dtype=np.int32)
    q = torch.from_numpy(case["q_bits"].view(np.int16)).view(torch.bfloat16).cuda()
    kn = torch.from_numpy(rng.standard_normal((3, 2, 64)).astype(np.float32)).to(torch.bfloat16).cuda()
    vn = torch.from_numpy(rng.standard_normal((3, 2, 64)).astype(np.float32)).to(torch.bfloat16).cuda()
    mk = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    res = {}
    for mode in ("two_calls", "step"):
        kp, vp = mk(case["k_pages"]), mk(case["v_pages"])
        btd, sld = torch.from_numpy(bt).cuda(), torch.from_numpy(sl).cuda()
        out = torch.full((3, 8, 64), float("nan"), dtype=torch.bfloat16, device="cuda")
        bl.device_errors()
        if mode == "two_calls":
            bl.kv_append(kn, vn, kp, vp, btd, sld)
            bl.decode_attention(q, kp, vp, btd, sld, 0.125, out)
        else:
            bl.decode_step(q, kn, vn, kp, vp, btd, sld, 0.125, out)
        torch.cuda.synchronize()
        res[mode] = (bl.device_errors(), sld.cpu().numpy(), G.bits16(kp), G.bits16(vp), G.out_f64(out))
    a, b = res["two_calls"], res["step"]
    assert a[0] == b[0] and (b[0] & 1), (a[0], b[0])
    assert np.array_equal(a[1], b[1]) and b[1][0] == 32 and b[1][2] == maxL and b[1][1] == 48
    assert np.array_equal(a[2], b[2]) and np.array_equal(a[3], b[3])
    assert np.all(np.isfinite(b[4]))
    G.assert_close(b[4], a[4], "bf16", "step vs two calls on malformed slots")
