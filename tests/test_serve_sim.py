"""Closed-loop serving model: the oracle against closed forms and hand-built
scenarios, then the library's simulator against the oracle, record by record.

The model's steps are those documented with bellman_sim_run (and in
oracle/serve_sim.py); the scenarios below fix what those steps imply for
small cases by reasoning, not by re-running the same loop."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import serve_sim as osim
from paper_2510_15330_amd import serve, traces

MS = 1_000_000


def _trace(arr, prompt, length):
    return traces.Trace(np.asarray(arr, np.int64), np.asarray(prompt, np.int32), np.asarray(length, np.int32))


def _osim(tr, **kw):
    if "controller" in kw:
        kw["controller"] = bool(kw["controller"])
    return osim.simulate(tr.arrival_ns, tr.prompt, tr.length, osim.SimConfig(**kw))


# ------------------------------------------------------------ oracle pins --

def test_single_request_closed_form():
    # one request: a prefill iteration, then L - 1 decode iterations whose KV
    # grows by one token each; the decode times form an arithmetic series
    P, L, a = 1000, 50, 7 * MS
    fixed, attn, pre = 2 * MS, 3000, 5000          # attn, pre: ps per token, multiples of 1000
    r = _osim(_trace([a], [P], [L]), fixed_ns=fixed, attn_ps_per_token=attn, prefill_ps_per_token=pre)
    first = a + fixed + pre * P // 1000
    n = L - 1
    decode_total = n * fixed + (attn // 1000) * (n * P + n * (n + 1) // 2)
    assert r.admit_ns == [a]
    assert r.first_ns == [first]
    assert r.finish_ns == [first + decode_total]
    assert r.iterations == L
    assert sum(d for (_, _, d, _, _, _) in r.log) == n        # one TBT sample per decoded token


def test_chunked_prefill_closed_form():
    # P = 1000 with 256-token chunks: three full chunks and one of 232
    P, a = 1000, 0
    fixed, pre = MS, 4000
    r = _osim(_trace([a], [P], [1]), fixed_ns=fixed, attn_ps_per_token=0, prefill_ps_per_token=pre,
              prefill_chunk_tokens=256)
    assert r.first_ns == [a + 3 * (fixed + 256 * 4) + (fixed + 232 * 4)]
    assert r.finish_ns == r.first_ns          # target 1: done with its first token
    assert [c for (_, _, _, c, _, _) in r.log] == [256, 256, 256, 232]


def test_fifo_one_slot():
    # max_running = 1: the second request starts when the first finishes
    tr = _trace([0, 0], [32, 32], [3, 2])
    fixed = MS
    r = _osim(tr, max_running=1, fixed_ns=fixed, attn_ps_per_token=0, prefill_ps_per_token=0)
    assert r.admit_ns == [0, 3 * fixed]
    assert r.finish_ns == [3 * fixed, 5 * fixed]


def test_page_budget_blocks_head():
    # each request needs ceil((16 + 8) / 16) = 2 pages at most, admission takes
    # ceil(16 / 16) = 1: a 2-page budget admits both (and must preempt when they
    # grow); with one page, a second 15-token request waits for the first
    tr = _trace([0, 0], [16, 16], [8, 8])
    r2 = _osim(tr, kv_capacity_pages=2, fixed_ns=MS, attn_ps_per_token=0, prefill_ps_per_token=0)
    assert r2.admit_ns == [0, 0]
    assert sum(r2.preemptions) >= 1          # both grow into a second page: one must yield
    r1 = _osim(_trace([0, 0], [15, 15], [1, 1]), kv_capacity_pages=1, fixed_ns=MS,
               attn_ps_per_token=0, prefill_ps_per_token=0)
    assert r1.admit_ns == [0, MS]             # the head waits for the first to finish


def test_preemption_recomputes_prompt_and_generated():
    # Two 16-token prompts, budget 3 pages.  Both prefill in iteration 1 (first
    # tokens).  Iteration 2 decodes both: request 0 appends position 16 (a new
    # page, the third); request 1 then needs a fourth page, none is free, and
    # the latest admitted (itself) is preempted.  Request 0 finishes at its
    # target; request 1 re-prefills prompt + 1 generated = 17 tokens.
    tr = _trace([0, 0], [16, 16], [3, 3])
    fixed, pre = MS, 1000
    r = _osim(tr, kv_capacity_pages=3, fixed_ns=fixed, attn_ps_per_token=0, prefill_ps_per_token=pre)
    assert r.preemptions == [0, 1]
    t1 = fixed + 32 * pre // 1000             # iteration 1: both prompts prefilled
    assert r.first_ns == [t1, t1]
    # iteration 2: only request 0 decodes; iteration 3: request 0 decodes its
    # last token while request 1 waits (request 0 holds 2 pages, 1 is free but
    # request 1 needs ceil(17 / 16) = 2)
    assert r.finish_ns[0] == t1 + 2 * fixed
    t_re = r.finish_ns[0] + fixed + 17 * pre // 1000   # re-prefill of 17 tokens
    assert r.log[3][3] == 17
    # after the re-prefill (its second token) one more decode reaches 3 tokens
    assert r.finish_ns[1] == t_re + fixed


def test_controller_caps_after_first_sample():
    # thresholds below every possible TBT: once the first tick pushes a sample
    # the rate is r_max, so requests queued later ask for round(0.8 L)
    arr = [0, int(0.5e9), int(2.5e9), int(3.5e9)]
    tr = _trace(arr, [64] * 4, [100] * 4)
    r = _osim(tr, controller=True, t1=0.0, t2=1.0, fixed_ns=10 * MS, attn_ps_per_token=0,
              prefill_ps_per_token=0)
    assert r.target[:2] == [100, 100]          # queued before the first tick
    assert r.target[2:] == [80, 80]
    assert r.r_at_queue[2:] == [0.2, 0.2]


def test_invariants_on_a_medium_trace():
    tr = traces.small_trace(400, seed=5, mean_gap_ms=8)
    cfg = dict(max_running=12, kv_capacity_pages=48, watermark_pages=1, fixed_ns=MS, attn_ps_per_token=20_000,
               prefill_ps_per_token=500_000, prefill_chunk_tokens=300, tick_ns=50 * MS)
    r = _osim(tr, **cfg)
    arr = tr.arrival_ns
    a, f, e = np.array(r.admit_ns), np.array(r.first_ns), np.array(r.finish_ns)
    assert (a >= arr).all() and (f > a).all() and (e >= f).all()
    assert list(np.argsort(a, kind="stable")) == list(range(len(tr)))   # first admissions in arrival order
    assert all(run <= cfg["max_running"] for (_, _, _, _, run, _) in r.log)
    # every decoded token is one TBT sample; a request's tokens come from its
    # completed prefills (the first, plus at most one per preemption) and decodes
    samples = sum(d for (_, _, d, _, _, _) in r.log)
    assert sum(t - 1 - p for t, p in zip(r.target, r.preemptions)) <= samples <= sum(t - 1 for t in r.target)
    # the ticks taken hold exactly the samples of the iterations that ended by then
    last = r.ticks[-1][0]
    assert sum(c for (_, c, _, _, _, _) in r.ticks) == sum(d for (end, _, d, _, _, _) in r.log if end <= last)


# ---------------------------------------------------- library vs oracle --

def _same(out, ref):
    rq = out.requests
    assert rq["admit_ns"].tolist() == ref.admit_ns
    assert rq["first_ns"].tolist() == ref.first_ns
    assert rq["finish_ns"].tolist() == ref.finish_ns
    assert rq["target"].tolist() == ref.target
    assert rq["preemptions"].tolist() == ref.preemptions
    assert rq["r_at_queue"].tolist() == ref.r_at_queue
    assert out.iterations == ref.iterations
    assert [tuple(x) for x in out.ticks.tolist()] == [tuple(t) for t in ref.ticks]
    if len(out.log):
        assert [tuple(x) for x in out.log.tolist()] == ref.log


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("chunk", [0, 64, 300])
@pytest.mark.parametrize("budget", [38, 60, 400])
def test_library_matches_oracle_small(seed, chunk, budget):
    tr = traces.small_trace(250, seed=seed, mean_gap_ms=15)
    cfg = dict(max_running=16, kv_capacity_pages=budget, watermark_pages=1, fixed_ns=MS,
               attn_ps_per_token=50_000, prefill_ps_per_token=2_000_000, prefill_chunk_tokens=chunk,
               tick_ns=100 * MS)
    ref = _osim(tr, **cfg)
    _same(serve.run(tr, max_iterations=1 << 20, **cfg), ref)
    t1, t2 = osim.thresholds_from(ref)
    out_u = serve.run(tr, **cfg)
    assert serve.thresholds(out_u) == (t1, t2)
    refc = _osim(tr, controller=1, t1=t1, t2=t2, **cfg)
    _same(serve.run(tr, max_iterations=1 << 20, controller=serve.LINEAR, t1=t1, t2=t2, **cfg), refc)


def test_library_matches_oracle_paper_trace():
    # the full 22-minute trace on the paper-shaped server, both runs
    cfg = {k: v for k, v in serve.PAPER_SERVER.items() if not k.startswith("live")}
    tr = traces.paper_trace(serve.PAPER_CAPACITY_RPS, seed=0)
    ref = _osim(tr, **cfg)
    out = serve.run(tr, **cfg)
    _same(out, ref)
    t1, t2 = osim.thresholds_from(ref)
    assert serve.thresholds(out) == (t1, t2)
    _same(serve.run(tr, controller=serve.LINEAR, t1=t1, t2=t2, **cfg), _osim(tr, controller=1, t1=t1, t2=t2, **cfg))


def test_library_rejects_bad_inputs():
    tr = _trace([5, 1], [10, 10], [1, 1])
    with pytest.raises(serve._binding.BellmanError):
        serve.run(tr)                                     # unsorted arrivals
    with pytest.raises(serve._binding.BellmanError):
        serve.run(_trace([0], [10_000], [10]), kv_capacity_pages=10)   # larger than the budget
    with pytest.raises(serve._binding.BellmanError):
        serve.run(_trace([0], [10], [1]), max_running=0)
    with pytest.raises(serve._binding.BellmanError):
        serve.run(_trace([0], [10], [1]), controller=7)
    with pytest.raises(TypeError):
        serve.run(_trace([0], [10], [1]), no_such_option=1)
