"""HIP graph capture of the library's steps.

A decode step (append + attention) and a prompt step (prompt write + prompt
attention) enqueue only kernels on the caller's stream once the workspace
has grown to the step's size: no memset, copy or host wait.  Each test
captures the step on one copy of a workload, replays the graph several times
with fresh inputs copied in eagerly between replays (and a synchronisation
after each), and compares every replay bit for bit with the same step run
eagerly on an identical second copy."""
from __future__ import annotations

import numpy as np
import pytest
import torch

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


def _bits(t):
    return t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.uint8)


def _build(name, steps):
    if name != "fp8_mixed":
        return wl.build(name, seed=11, device="cuda", steps=steps)
    # a small fp8 batch with lengths on and next to page and step edges
    wl.CONFIGS["_graph_fp8"] = dict(wl.CONFIGS["stress_fp8"], B=24)
    orig = wl.sample_lengths
    lens = np.array([0, 1, 15, 16, 17, 63, 64, 65, 127, 128, 129, 200,
                     255, 256, 300, 511, 512, 513, 700, 1000, 1023, 1024, 1500, 2047], dtype=np.int64)

    def fake(n, seed=0, tiny_reading="after"):
        return (lens, {}) if n == "_graph_fp8" else orig(n, seed, tiny_reading)
    wl.sample_lengths = fake
    try:
        return wl.build("_graph_fp8", seed=11, device="cuda", steps=steps)
    finally:
        wl.sample_lengths = orig
        del wl.CONFIGS["_graph_fp8"]


@pytest.mark.parametrize("name", ["llama3_8b", "fp8_mixed"])
def test_decode_step_graph_matches_eager(name):
    steps = 5
    A, B = _build(name, steps), _build(name, steps)
    assert torch.equal(_bits(A.k_pages), _bits(B.k_pages))
    out_g = torch.empty((A.B, A.H_q, A.D), dtype=torch.bfloat16, device="cuda")
    out_e = torch.empty_like(out_g)
    kn, vn, q = A.k_new[0].clone(), A.v_new[0].clone(), A.q[0].clone()
    kw = dict(k_scale=A.k_scale, v_scale=A.v_scale)
    # grow the workspace outside the capture (attention alone leaves A unchanged)
    bl.decode_attention(q, A.k_pages, A.v_pages, A.block_table, A.seq_lens, A.scale, out_g, **kw)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        bl.kv_append(kn, vn, A.k_pages, A.v_pages, A.block_table, A.seq_lens)
        bl.decode_attention(q, A.k_pages, A.v_pages, A.block_table, A.seq_lens, A.scale, out_g, **kw)
    torch.cuda.synchronize()
    assert torch.equal(A.seq_lens, B.seq_lens)          # capture ran nothing
    for i in range(steps):
        kn.copy_(A.k_new[i])
        vn.copy_(A.v_new[i])
        q.copy_(A.q[i])
        g.replay()
        torch.cuda.synchronize()
        bl.kv_append(B.k_new[i], B.v_new[i], B.k_pages, B.v_pages, B.block_table, B.seq_lens)
        bl.decode_attention(B.q[i], B.k_pages, B.v_pages, B.block_table, B.seq_lens, B.scale, out_e,
                            k_scale=B.k_scale, v_scale=B.v_scale)
        torch.cuda.synchronize()
        assert torch.equal(A.seq_lens, B.seq_lens), f"{name} replay {i}: lengths"
        assert torch.equal(_bits(out_g), _bits(out_e)), f"{name} replay {i}: attention output"
    assert torch.equal(_bits(A.k_pages), _bits(B.k_pages)) and torch.equal(_bits(A.v_pages), _bits(B.v_pages))
    assert bl.device_errors() == 0


def test_prompt_step_graph_matches_eager():
    A = wl.build_prefill("prefill_tiny", seed=5, device="cuda")
    B = wl.build_prefill("prefill_tiny", seed=5, device="cuda")
    lens0 = A.seq_lens.clone()
    out_g = torch.empty((A.T, A.H_q, A.D), dtype=torch.bfloat16, device="cuda")
    out_e = torch.empty_like(out_g)
    kn, vn, q = A.k_new.clone(), A.v_new.clone(), A.q.clone()

    def step(w, k, v, qq, out):
        bl.kv_write(k, v, w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.q_start)
        bl.prefill_attention(qq, w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.q_start, w.scale, out)

    step(A, kn, vn, q, out_g)          # grows the workspace; the write is repeated on every replay
    torch.cuda.synchronize()
    A.seq_lens.copy_(lens0)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(A, kn, vn, q, out_g)
    torch.cuda.synchronize()
    gen = torch.Generator(device="cuda")
    for i in range(4):
        gen.manual_seed(100 + i)
        fresh_q = torch.randn(A.q.shape, generator=gen, device="cuda").to(torch.bfloat16)
        fresh_k = torch.randn(A.k_new.shape, generator=gen, device="cuda").to(torch.bfloat16)
        fresh_v = torch.randn(A.v_new.shape, generator=gen, device="cuda").to(torch.bfloat16)
        A.seq_lens.copy_(lens0)
        B.seq_lens.copy_(lens0)
        q.copy_(fresh_q)
        kn.copy_(fresh_k)
        vn.copy_(fresh_v)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        step(B, fresh_k, fresh_v, fresh_q, out_e)
        torch.cuda.synchronize()
        assert torch.equal(A.seq_lens, B.seq_lens), f"prompt replay {i}: lengths"
        assert torch.equal(_bits(out_g), _bits(out_e)), f"prompt replay {i}: attention output"
        assert torch.equal(_bits(A.k_pages), _bits(B.k_pages)) and torch.equal(_bits(A.v_pages), _bits(B.v_pages))
    assert bl.device_errors() == 0


def test_graph_survives_workspace_growth():
    """A graph captured while the workspace was small still replays correctly
    after a later call has grown the workspace (the old block is kept until
    bellman_shutdown), and a call that would have to grow the workspace during
    a capture is refused instead of allocating there."""
    bl.shutdown()                                  # start from no workspace at all
    A = wl.build("tiny", seed=12, device="cuda", steps=4)
    B = wl.build("tiny", seed=12, device="cuda", steps=4)
    out_g = torch.empty((A.B, A.H_q, A.D), dtype=torch.bfloat16, device="cuda")
    out_e = torch.empty_like(out_g)
    kn, vn, q = A.k_new[0].clone(), A.v_new[0].clone(), A.q[0].clone()
    bl.decode_attention(q, A.k_pages, A.v_pages, A.block_table, A.seq_lens, A.scale, out_g)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        bl.kv_append(kn, vn, A.k_pages, A.v_pages, A.block_table, A.seq_lens)
        bl.decode_attention(q, A.k_pages, A.v_pages, A.block_table, A.seq_lens, A.scale, out_g)
    torch.cuda.synchronize()
    bl.reserve_workspace(256 << 20)                # grows: the captured block is retired, not freed
    for i in range(4):
        kn.copy_(A.k_new[i])
        vn.copy_(A.v_new[i])
        q.copy_(A.q[i])
        g.replay()
        torch.cuda.synchronize()
        bl.kv_append(B.k_new[i], B.v_new[i], B.k_pages, B.v_pages, B.block_table, B.seq_lens)
        bl.decode_attention(B.q[i], B.k_pages, B.v_pages, B.block_table, B.seq_lens, B.scale, out_e)
        torch.cuda.synchronize()
        assert torch.equal(A.seq_lens, B.seq_lens), f"replay {i}: lengths"
        assert torch.equal(_bits(out_g), _bits(out_e)), f"replay {i}: attention output"
    assert bl.device_errors() == 0
    del g
    torch.cuda.synchronize()

    bl.shutdown()                                  # no workspace: the next attention must grow it
    g2 = torch.cuda.CUDAGraph()
    with pytest.raises(bl.BellmanError) as ei:
        with torch.cuda.graph(g2):
            out_g.zero_()
            bl.decode_attention(q, A.k_pages, A.v_pages, A.block_table, A.seq_lens, A.scale, out_g)
    assert ei.value.code == -2 and "graph capture" in str(ei.value)
    del g2
    torch.cuda.synchronize()
