"""The no-allocation decode entry point (bellman_decode_attention_noalloc):
through the C ABI, two calls in a row, the second with a smaller input, each
compared with bellman_decode_attention_opts on the same inputs (bit for bit:
same kernels and launch configuration) and with the oracle (within the
bf16 / fp8 bounds); and a call too large for the fixed array is rejected
before anything runs.  Collected last, after every other GPU test, and also
passes alone in a fresh process."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from tests import _dense as dn
from tests import _gpu as G

pytestmark = pytest.mark.gpu

bl = pytest.importorskip("paper_2510_15330_amd")


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bl.library()
    yield
    torch.cuda.synchronize()


def _dev(case, kv):
    if kv == "bf16":
        kp = torch.from_numpy(case["k_pages"].view(np.int16)).view(torch.bfloat16)
        vp = torch.from_numpy(case["v_pages"].view(np.int16)).view(torch.bfloat16)
    else:
        kp, vp = torch.from_numpy(case["k_pages"]), torch.from_numpy(case["v_pages"])
    sc = lambda a: None if a is None else torch.from_numpy(a).cuda()
    return dict(q=torch.from_numpy(case["q_bits"].view(np.int16)).view(torch.bfloat16).cuda(),
                k=kp.cuda(), v=vp.cuda(), bt=torch.from_numpy(case["block_table"]).cuda(),
                sl=torch.from_numpy(case["seq_lens"]).cuda(), ks=sc(case["k_scale"]), vs=sc(case["v_scale"]))


def _run(fn, d, scale, **kw):
    B, H_q, D = d["q"].shape
    out = torch.full((B, H_q, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    fn(d["q"], d["k"], d["v"], d["bt"], d["sl"], scale, out, k_scale=d["ks"], v_scale=d["vs"], **kw)
    torch.cuda.synchronize()
    return out


CALLS = [
    # B, H_q, H_kv, D, kv, lengths (cut by the work split into many partial pieces)
    (48, 32, 8, 128, "bf16", "mixed"),
    (5, 64, 8, 128, "fp8", [1, 200, 3000, 17, 640]),
]


def test_noalloc_matches_allocating_entry_point_twice():
    rng = np.random.default_rng(777)
    for i, (B, H_q, H_kv, D, kv, lens) in enumerate(CALLS):
        if lens == "mixed":
            lens = [int(x) for x in rng.integers(0, 5000, size=B)]
            lens[3] = 0
        case = dn.random_case(rng, B, H_q, H_kv, D, lens, kv)
        if kv == "fp8":
            case["k_scale"] = (rng.uniform(0.5, 1.5, size=(B, H_kv)) / 40.0).astype(np.float32)
            case["v_scale"] = (rng.uniform(0.5, 1.5, size=(B, H_kv)) / 40.0).astype(np.float32)
        scale = float(np.float32(1.0 / np.sqrt(D)))
        d = _dev(case, kv)
        print(f"call {i}: B={B} H_q={H_q} H_kv={H_kv} D={D} {kv}", flush=True)
        ref_out = _run(bl.decode_attention, d, scale, max_waves=0)
        for waves in (0, 37):
            got = _run(bl.decode_attention_noalloc, d, scale, max_waves=waves)
            want = ref_out if waves == 0 else _run(bl.decode_attention, d, scale, max_waves=waves)
            assert torch.equal(got.view(torch.int16), want.view(torch.int16)), f"call {i} waves={waves}"
            ref = oracle.decode_attention(case["q_bits"], case["k_pages"], case["v_pages"], case["block_table"],
                                          case["seq_lens"], scale, G.kv_code(kv), case["k_scale"], case["v_scale"])
            G.assert_close(G.out_f64(got), ref, kv, f"noalloc call {i} waves={waves}")
        assert bl.device_errors() == 0


def test_noalloc_rejects_calls_beyond_the_array():
    # fp8 pools with 16 query heads per KV head at head_dim 128: two partial
    # slots of 520 bytes per wave and head come to 34 MB over the 2048 waves
    # of a whole MI355X, more than the 32 MiB array; capping the waves fits
    rng = np.random.default_rng(778)
    B, H_kv, G_, D = 3, 8, 16, 128
    case = dn.random_case(rng, B, H_kv * G_, H_kv, D, [5000, 70, 1], "fp8")
    case["k_scale"] = (rng.uniform(0.5, 1.5, size=(B, H_kv)) / 40.0).astype(np.float32)
    case["v_scale"] = (rng.uniform(0.5, 1.5, size=(B, H_kv)) / 40.0).astype(np.float32)
    d = _dev(case, "fp8")
    scale = float(np.float32(1.0 / np.sqrt(D)))
    waves = torch.cuda.get_device_properties(0).multi_processor_count * 8
    need = 256 + 16 * waves + 2 * waves * G_ * 8 + 2 * waves * G_ * D * 4
    if need <= bl.FIXED_SCRATCH_BYTES:
        pytest.skip(f"{waves} waves fit the fixed array on this device")
    with pytest.raises(bl.BellmanError) as ei:
        _run(bl.decode_attention_noalloc, d, scale)
    assert ei.value.code == -2 and "fixed scratch array" in str(ei.value)
    got = _run(bl.decode_attention_noalloc, d, scale, max_waves=1900)
    want = _run(bl.decode_attention, d, scale, max_waves=1900)
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))
