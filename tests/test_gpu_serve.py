"""Live mode of the serving model: every iteration runs the library's append
and decode-attention kernels on the decoding requests (rows that move as
requests finish, pages that grow one at a time, preemptions) and uses their
measured time.  The event order then depends on the GPU's timing, so these
tests check what holds for any timing: completion, ordering, the decode
count, clean device error flags (the run fails otherwise) and that the
measured kernels read a plausible number of bytes per second."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2510_15330_amd import serve, traces

MS = 1_000_000


def _live(tr, **kw):
    stream = torch.cuda.current_stream().cuda_stream
    cfg = dict(max_running=24, kv_capacity_pages=160, watermark_pages=2, fixed_ns=MS, prefill_ps_per_token=200_000,
               prefill_chunk_tokens=512, tick_ns=20 * MS, live=1, live_layers=4, live_q_heads=8,
               live_kv_heads=2, live_head_dim=128)
    cfg.update(kw)
    return serve.run(tr, stream=stream, max_iterations=1 << 20, **cfg)


@pytest.mark.gpu
def test_live_run_completes_in_order():
    tr = traces.small_trace(120, seed=3, mean_gap_ms=2, prompt=(64, 600), length=(1, 80))
    out = _live(tr)
    r = out.requests
    arr = tr.arrival_ns
    assert (r["finish_ns"] >= r["first_ns"]).all() and (r["first_ns"] > r["admit_ns"]).all()
    assert (r["admit_ns"] >= arr).all()
    assert list(np.argsort(r["admit_ns"], kind="stable")) == list(range(len(tr)))
    assert (r["target"] == tr.length).all()                      # no controller
    decoded = int(out.log["decoding"].sum())
    lo = int((r["target"] - 1 - r["preemptions"]).sum())
    assert lo <= decoded <= int((r["target"] - 1).sum())
    assert out.live_gpu_ms > 0 and out.live_kv_bytes > 0
    gbs = out.live_kv_bytes / (out.live_gpu_ms * 1e6)
    assert 1.0 < gbs < 8000.0, gbs
    assert out.preemptions > 0                                   # the small budget forces some


@pytest.mark.gpu
def test_live_controller_caps_under_load():
    # thresholds below every TBT: after the first tick every new request is capped
    tr = traces.small_trace(80, seed=4, mean_gap_ms=5, prompt=(64, 400), length=(20, 80))
    out = _live(tr, controller=serve.LINEAR, t1=0.0, t2=1.0)
    r = out.requests
    late = tr.arrival_ns > 100 * MS           # several 20 ms ticks with decoded tokens before
    assert late.any()
    assert (r["r_at_queue"][late] > 0).all()
    assert (r["target"][late] < tr.length[late]).all()
    assert (r["finish_ns"] > 0).all()
