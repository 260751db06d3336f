"""The fused decode step (bellman_decode_step) against the two-call step
(bellman_kv_append, then bellman_decode_attention) on the same state: pools
byte for byte, lengths, error flags, and outputs bit for bit (the same
kernels read the same pools in the same work split), over bf16 rows, fp8
codes and bf16 rows quantised into fp8 pools, new positions on and next to
page edges, empty requests, a full table, many short requests, several work
splits, and HIP-graph replays; and the one documented difference, a new
position whose block-table entry lies outside the pool."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2510_15330_amd as bl
from tests import _dense as dn
from tests import _gpu as G

pytestmark = pytest.mark.gpu


def _state(seed, B, H_q, H_kv, D, lens, kind):
    """Pools with pages for every stored token and the new one; stored
    lengths `lens`; new rows (bf16, or fp8 codes, or bf16 for quantising)."""
    rng = np.random.default_rng(seed)
    pool = "bf16" if kind == "bf16" else "fp8"
    case = dn.random_case(rng, B, H_q, H_kv, D, [L + 1 for L in lens], pool)
    if pool == "bf16":
        kp = torch.from_numpy(case["k_pages"].view(np.int16)).view(torch.bfloat16)
        vp = torch.from_numpy(case["v_pages"].view(np.int16)).view(torch.bfloat16)
    else:
        kp, vp = torch.from_numpy(case["k_pages"]), torch.from_numpy(case["v_pages"])
    if kind == "fp8":
        kn = torch.from_numpy(rng.integers(0, 126, size=(B, H_kv, D), dtype=np.uint8) | (
            rng.integers(0, 2, size=(B, H_kv, D), dtype=np.uint8) << 7))
        vn = torch.from_numpy(rng.integers(0, 126, size=(B, H_kv, D), dtype=np.uint8))
    else:
        kn = torch.from_numpy(rng.standard_normal((B, H_kv, D)).astype(np.float32) * 3).to(torch.bfloat16)
        vn = torch.from_numpy(rng.standard_normal((B, H_kv, D)).astype(np.float32) * 3).to(torch.bfloat16)
    q = torch.from_numpy(case["q_bits"].view(np.int16)).view(torch.bfloat16)
    s = dict(q=q, k=kp, v=vp, bt=torch.from_numpy(case["block_table"]),
             sl=torch.tensor(lens, dtype=torch.int32), kn=kn, vn=vn,
             ks=None if case["k_scale"] is None else torch.from_numpy(case["k_scale"]),
             vs=None if case["v_scale"] is None else torch.from_numpy(case["v_scale"]))
    return {k: (None if v is None else v.cuda()) for k, v in s.items()}


def _clone(s):
    c = {k: (None if v is None else v.clone()) for k, v in s.items()}
    B, H_q, D = s["q"].shape
    c["out"] = torch.full((B, H_q, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    return c


def _two_calls(c, scale, **kw):
    bl.kv_append(c["kn"], c["vn"], c["k"], c["v"], c["bt"], c["sl"], k_scale=c["ks"], v_scale=c["vs"])
    bl.decode_attention(c["q"], c["k"], c["v"], c["bt"], c["sl"], scale, c["out"], k_scale=c["ks"],
                        v_scale=c["vs"], **kw)


def _step(c, scale, **kw):
    bl.decode_step(c["kn"], c["vn"], c["q"], c["k"], c["v"], c["bt"], c["sl"], scale, c["out"], k_scale=c["ks"],
                   v_scale=c["vs"], **kw)


def _bits(t):
    # pools compared bit for bit: unused slots hold a NaN pattern
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


def _same(a, b, what):
    for key in ("k", "v", "sl"):
        assert torch.equal(_bits(a[key]), _bits(b[key])), f"{what}: {key} differs"
    oa, ob = a["out"].view(torch.int16), b["out"].view(torch.int16)
    assert torch.equal(oa, ob), f"{what}: outputs differ in {(oa != ob).sum().item()} elements"


CASES = [
    # name, B, H_q, H_kv, D, stored lengths, rows
    ("bf16_page_edges", 6, 32, 8, 128, [0, 15, 16, 17, 1000, 63], "bf16"),
    ("bf16_d64_g4", 5, 8, 2, 64, [1, 31, 32, 64, 500], "bf16"),
    ("bf16_g1_long", 2, 4, 4, 128, [4095, 2048], "bf16"),
    ("fp8_codes", 4, 64, 8, 128, [0, 127, 128, 2000], "fp8"),
    ("fp8_quantising", 4, 64, 8, 128, [5, 16, 700, 31], "fp8q"),
    ("fp8_d64", 3, 16, 2, 64, [0, 47, 300], "fp8"),
]
SPLITS = [dict(), dict(max_waves=7), dict(max_waves=1)]
BF16_SPLITS = [dict(pages_per_step=1), dict(pages_per_step=2, max_waves=5)]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_step_matches_two_calls(case):
    name, B, H_q, H_kv, D, lens, kind = case
    base = _state(len(name), B, H_q, H_kv, D, lens, kind)
    scale = float(np.float32(1.0 / np.sqrt(D)))
    for kw in SPLITS + (BF16_SPLITS if kind == "bf16" else []):
        a, b = _clone(base), _clone(base)
        _two_calls(a, scale, **kw)
        torch.cuda.synchronize()
        assert bl.device_errors() == 0
        _step(b, scale, **kw)
        torch.cuda.synchronize()
        assert bl.device_errors() == 0
        _same(a, b, f"{name} {kw}")
        assert b["sl"].cpu().tolist() == [L + 1 for L in lens]


def test_step_many_short_requests():
    # 1500 requests (the planner's multi-batch path), lengths 0..40
    rng = np.random.default_rng(15)
    lens = [int(x) for x in rng.integers(0, 41, size=1500)]
    base = _state(16, 1500, 8, 2, 64, lens, "bf16")
    for kw in (dict(), dict(max_waves=37)):
        a, b = _clone(base), _clone(base)
        _two_calls(a, 0.125, **kw)
        _step(b, 0.125, **kw)
        torch.cuda.synchronize()
        assert bl.device_errors() == 0
        _same(a, b, f"1500 requests {kw}")


def test_step_against_oracle():
    # the step's output and pools against the oracle's append + attention
    lens = [0, 15, 16, 300]
    s = _state(99, 4, 16, 4, 128, lens, "bf16")
    # new rows of unit scale, like the stored ones, so that the outputs stay
    # near unit size, where the bf16 tolerance holds
    s["kn"], s["vn"] = (s["kn"].float() / 3).to(torch.bfloat16), (s["vn"].float() / 3).to(torch.bfloat16)
    kp, vp = G.bits16(s["k"]), G.bits16(s["v"])
    sl = s["sl"].cpu().numpy().astype(np.int32)
    bt = s["bt"].cpu().numpy()
    oracle.kv_append(G.bits16(s["kn"]), G.bits16(s["vn"]), kp, vp, bt, sl)
    ref = oracle.decode_attention(G.bits16(s["q"]), kp, vp, bt, sl, 0.0884)
    c = _clone(s)
    _step(c, 0.0884)
    torch.cuda.synchronize()
    assert bl.device_errors() == 0
    assert np.array_equal(G.bits16(c["k"]), kp) and np.array_equal(G.bits16(c["v"]), vp)
    assert np.array_equal(c["sl"].cpu().numpy(), sl)
    G.assert_close(G.out_f64(c["out"]), ref, "bf16", "decode step")


def test_step_full_table_and_page_outside_pool():
    lens = [20, 96, 47]   # request 1's new position opens page 6
    base = _state(7, 3, 8, 2, 128, lens, "bf16")
    maxP = base["bt"].shape[1]
    # request 0: its table is full (stored length = maxP * 16): neither path
    # appends, both flag 1, and both attend over the full table
    base["sl"][0] = maxP * 16
    row0 = base["bt"][0].clone()
    base["bt"][0, :] = base["bt"][2, 0]
    a, b = _clone(base), _clone(base)
    _two_calls(a, 0.1)
    torch.cuda.synchronize()
    assert bl.device_errors() == 1
    _step(b, 0.1)
    torch.cuda.synchronize()
    assert bl.device_errors() == 1
    _same(a, b, "full table")
    # request 1: the entry of its new position lies outside the pool: the two
    # calls skip the append and attend over the old tokens; the step attends
    # over the new position, finds the entry outside the pool and writes NaN
    # rows for that request (flags 1 and 4).  Every other request agrees: bit
    # for bit with one wave, and within the bf16 bound under the default split
    # (request 1's extra page moves the split points, so the rounding of the
    # requests cut at them changes)
    # (request 0 gets its own pages back: a new row must not land in a page
    # that another request of the call reads)
    base["sl"][0] = lens[0]
    base["bt"][0] = row0
    base["bt"][1, lens[1] // 16] = 1 << 30
    keep = [0, 2]
    for kw in (dict(max_waves=1), dict()):
        a, b = _clone(base), _clone(base)
        _two_calls(a, 0.1, **kw)
        torch.cuda.synchronize()
        assert bl.device_errors() == 1
        _step(b, 0.1, **kw)
        torch.cuda.synchronize()
        assert bl.device_errors() == 1 | 4
        for key in ("k", "v", "sl"):
            assert torch.equal(_bits(a[key]), _bits(b[key])), key
        assert torch.isnan(b["out"][1].float()).all()
        if kw:
            assert torch.equal(a["out"][keep].view(torch.int16), b["out"][keep].view(torch.int16))
        else:
            G.assert_close(G.out_f64(b["out"][keep]), G.out_f64(a["out"][keep]), "bf16", "outside pool")


def test_step_graph_replays():
    # three decode steps captured in one graph, replayed from the same start
    # state several times with eager work in between, against eager steps
    lens = [3, 16, 200, 0]
    base = _state(5, 4, 32, 8, 128, lens, "bf16")
    rows = [(torch.randn_like(base["kn"].float()).to(torch.bfloat16), torch.randn_like(base["vn"].float())
             .to(torch.bfloat16)) for _ in range(3)]
    eager = _clone(base)
    outs = []
    for kn, vn in rows:
        eager["kn"], eager["vn"] = kn, vn
        _step(eager, 0.09)
        outs.append(eager["out"].clone())
    torch.cuda.synchronize()
    g_state = _clone(base)
    bufs = [(kn.clone(), vn.clone()) for kn, vn in rows]
    gouts = [torch.empty_like(outs[0]) for _ in rows]
    # a first eager call sizes the workspace before the capture
    warm = _clone(base)
    _step(warm, 0.09)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    start = {k: g_state[k].clone() for k in ("k", "v", "sl")}
    with torch.cuda.graph(graph, stream=side):
        for i, (kn, vn) in enumerate(bufs):
            bl.decode_step(kn, vn, g_state["q"], g_state["k"], g_state["v"], g_state["bt"], g_state["sl"], 0.09,
                           gouts[i])
    for rep in range(3):
        for key in ("k", "v", "sl"):
            g_state[key].copy_(start[key])
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert bl.device_errors() == 0
        for i in range(3):
            assert torch.equal(gouts[i].view(torch.int16), outs[i].view(torch.int16)), f"replay {rep} step {i}"
        for key in ("k", "v", "sl"):
            assert torch.equal(_bits(g_state[key]), _bits(eager[key])), f"replay {rep}: {key}"
        _clone(base)   # eager work between replays


def test_step_rejects_unbuilt_shapes():
    # the step is built for the default steps only
    s = _state(3, 2, 16, 2, 128, [5, 40], "fp8")
    c = _clone(s)
    for kw in (dict(pages_per_step=1), dict(pages_per_step=4, pipeline_depth=2)):
        with pytest.raises(bl.BellmanError, match="default steps"):
            _step(c, 0.1, **kw)
    s = _state(3, 2, 16, 2, 128, [5, 40], "bf16")
    c = _clone(s)
    with pytest.raises(bl.BellmanError, match="default steps"):
        _step(c, 0.1, pipeline_depth=1)
    torch.cuda.synchronize()
    assert torch.equal(c["sl"].cpu(), torch.tensor([5, 40], dtype=torch.int32))


def test_step_empty_batch_is_noop():
    q = torch.empty((0, 8, 64), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((4, 2, 8, 16, 8), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros((4, 2, 64, 16), dtype=torch.bfloat16, device="cuda")
    rows = torch.empty((0, 2, 64), dtype=torch.bfloat16, device="cuda")
    bt = torch.empty((0, 1), dtype=torch.int32, device="cuda")
    sl = torch.empty((0,), dtype=torch.int32, device="cuda")
    out = torch.empty((0, 8, 64), dtype=torch.bfloat16, device="cuda")
    bl.decode_step(rows, rows.clone(), q, k, v, bt, sl, 0.125, out)
    torch.cuda.synchronize()
    assert bl.device_errors() == 0
    assert torch.equal(k, torch.zeros_like(k)) and torch.equal(v, torch.zeros_like(v))


def test_step_negative_length_matches_two_calls():
    # a negative stored length: both paths flag it (length 2, append 1), write
    # no row for it, leave its length alone and give it zero rows; the other
    # requests advance as usual
    lens = [5, 40, 17]
    base = _state(31, 3, 16, 4, 128, lens, "bf16")
    base["sl"][1] = -3
    for kw in (dict(), dict(max_waves=5)):
        a, b = _clone(base), _clone(base)
        _two_calls(a, 0.1, **kw)
        torch.cuda.synchronize()
        ea = bl.device_errors()
        _step(b, 0.1, **kw)
        torch.cuda.synchronize()
        eb = bl.device_errors()
        assert ea == eb == 1 | 2, (ea, eb)
        _same(a, b, f"negative length {kw}")
        assert b["sl"].cpu().tolist() == [6, -3, 18]
        assert torch.all(b["out"][1].float() == 0)
