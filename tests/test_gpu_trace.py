"""Per-wave timing records of the attention kernel (opts.wave_times): the
traced kernel computes the same bits as the untraced one, and every wave of
the call leaves a well-formed record (end not before start, an XCD id of the
device's eight)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

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


@pytest.mark.parametrize("name,pps", [("llama3_8b", 0), ("llama3_8b", 2), ("stress_fp8", 0)])
@pytest.mark.parametrize("waves", [0, 37])
def test_traced_kernel_same_bits_and_records(name, pps, waves):
    w = wl.build(name, seed=0, device="cuda", steps=1)
    plain = torch.empty((w.B, w.H_q, w.D), dtype=torch.bfloat16, device="cuda")
    traced = torch.empty_like(plain)
    rec = torch.full((3 * 16384,), -1, dtype=torch.int64, device="cuda")
    print(f"trace {name} pages/step={pps} waves={waves}", flush=True)
    kw = dict(k_scale=w.k_scale, v_scale=w.v_scale, max_waves=waves, pages_per_step=pps)
    bl.decode_attention(w.q[0], w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.scale, plain, **kw)
    bl.decode_attention(w.q[0], w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.scale, traced, wave_times=rec,
                        **kw)
    torch.cuda.synchronize()
    assert torch.equal(plain.view(torch.int16), traced.view(torch.int16))
    r = rec.view(-1, 3).cpu().numpy()
    n = int((r[:, 0] >= 0).sum())
    if waves:
        assert n == waves
    assert np.all(r[:n, 0] >= 0) and np.all(r[n:, 0] == -1), "records of a contiguous prefix of waves"
    assert np.all(r[:n, 1] >= r[:n, 0])
    xcc = (r[:n, 2] >> 32) & 15
    assert np.all(xcc < 8)
    assert bl.device_errors() == 0


def test_trace_rejects_untraced_shapes():
    w = G.to_device(wl.build("tiny", seed=0))          # head_dim 64: no traced twin
    out = torch.empty((w.B, w.H_q, w.D), dtype=torch.bfloat16, device="cuda")
    rec = torch.zeros(3 * 64, dtype=torch.int64, device="cuda")
    with pytest.raises(bl.BellmanError, match="wave_times"):
        bl.decode_attention(w.q[0], w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.scale, out, wave_times=rec)
