"""The library's controller variants and class policies against the oracle:
identical rates on random tick sequences (same binary64 operations in the
same order), identical caps, the serving model with each variant and with
classes record for record, and rejected parameters."""
from __future__ import annotations

import random

import numpy as np
import pytest

from oracle import controller as oc
from oracle import serve_sim as osim
from paper_2510_15330_amd import _binding as B
from paper_2510_15330_amd import serve, traces

MS = 1_000_000

PARAM_SETS = {
    B.CTL_MPC: [dict(), dict(horizon=3, tau=2.5, w_delta=0.0, window=3, floor_window=7),
                dict(w_quality=0.0, w_energy=0.3, step=0.03, r_min=0.0, r_max=0.3)],
    B.CTL_BBR: [dict(), dict(bw_window=3, rt_window=5, cycle=3, margin=0.1, bbr_step=0.05, probe=0.0),
                dict(r_max=0.5, cycle=1)],
    B.CTL_PCC: [dict(), dict(interval=1, epsilon=0.05, gain=0.1), dict(interval=3, pcc_w_quality=0.0, r_max=0.4)],
    B.CTL_LINEAR: [dict(), dict(window=2, r_min=0.1, r_max=0.3)],
}

ORACLE_NAMES = {"bbr_step": "step", "pcc_w_lat": "w_lat", "pcc_w_quality": "w_quality"}


def _oracle(kind, t1, t2, params):
    p = {ORACLE_NAMES.get(k, k): v for k, v in params.items()}
    if kind == B.CTL_MPC:
        return oc.OracleMPC(t1, t2, **p)
    if kind == B.CTL_BBR:
        return oc.OracleBBR(**p)
    if kind == B.CTL_PCC:
        return oc.OraclePCC(t1, t2, **p)
    return oc.OracleLinear(t1, t2, **p)


@pytest.mark.parametrize("kind", sorted(PARAM_SETS))
def test_rates_match_the_oracle(kind):
    rnd = random.Random(kind)
    for params in PARAM_SETS[kind]:
        t1, t2 = 0.08, 0.2
        lib = B.VariantController(kind, t1, t2, **params)
        ora = _oracle(kind, t1, t2, params)
        level = 0.05
        for step in range(400):
            level = min(max(level + rnd.uniform(-0.02, 0.025), 0.01), 0.5)
            has = rnd.random() < 0.9
            y = level * rnd.uniform(0.9, 1.1)
            n = rnd.uniform(0, 800)
            tick = rnd.choice([1.0, 0.5, 2.0])
            r_l = lib.observe(has, y, n, tick)
            r_o = ora.observe(has, y, n, tick)
            assert r_l == r_o, (kind, params, step, r_l, r_o)
            for L in (0, 1, 15, 16, 17, 100, 999):
                for w, byp in ((1.0, 0), (0.0, 0), (0.5, 16), (2.0, 0)):
                    want = oc.cap_for_class(L, r_o, w, byp, lib.params.r_max)
                    assert lib.cap(L, w, byp) == want


def test_length_cap_on_a_variant_pushes_a_tick():
    # bellman_length_cap's sample reaches a variant as a tick with no tokens
    lib = B.VariantController(B.CTL_MPC, 0.1, 0.2)
    ora = oc.OracleMPC(0.1, 0.2)
    for y in (0.05, 0.3, 0.4, 0.5, 0.6, 0.2):
        sig = B.LoadSignal(lib._h, 1, y, 100)
        n = B.library().bellman_length_cap(sig)
        ora.observe(True, y, 0.0, 1.0)
        assert n == ora_cap(ora.r, 100)


def ora_cap(r, L):
    return oc.cap_for_class(L, r)


@pytest.mark.parametrize("kind,bad", [
    (B.CTL_MPC, dict(t2=0.05)), (B.CTL_MPC, dict(horizon=0)), (B.CTL_MPC, dict(tau=0.0)),
    (B.CTL_MPC, dict(step=0.0)), (B.CTL_MPC, dict(w_delta=-1.0)), (B.CTL_PCC, dict(t2=0.1)),
    (B.CTL_PCC, dict(interval=0)), (B.CTL_BBR, dict(margin=1.0)), (B.CTL_BBR, dict(cycle=0)),
    (B.CTL_BBR, dict(rt_window=0)), (B.CTL_LINEAR, dict(window=0)), (B.CTL_MPC, dict(r_max=1.0)),
])
def test_rejected_parameters(kind, bad):
    args = dict(t1=0.1, t2=0.2)
    args.update(bad)
    with pytest.raises(B.BellmanError):
        B.VariantController(kind, **args)


def test_rejected_observations():
    c = B.VariantController(B.CTL_BBR, 0.1, 0.2)
    for args in ((True, float("nan"), 1.0, 1.0), (True, 0.1, -1.0, 1.0), (True, 0.1, 1.0, 0.0)):
        with pytest.raises(B.BellmanError):
            c.observe(*args)
    with pytest.raises(B.BellmanError):
        c.cap(-1)
    with pytest.raises(B.BellmanError):
        c.cap(10, weight=-0.5)
    assert B.library().bellman_ctl_params_default(9, 0.0, 0.0, None) < 0


# ----------------------------------------------------------- serving model --

def _osim(tr, cls=None, **kw):
    return osim.simulate(tr.arrival_ns, tr.prompt, tr.length, osim.SimConfig(**kw), cls=cls)


def _same(out, ref):
    rq = out.requests
    assert rq["target"].tolist() == ref.target
    assert rq["r_at_queue"].tolist() == ref.r_at_queue
    assert rq["admit_ns"].tolist() == ref.admit_ns
    assert rq["finish_ns"].tolist() == ref.finish_ns
    assert [tuple(x) for x in out.ticks.tolist()] == [tuple(t) for t in ref.ticks]


SMALL = dict(max_running=16, kv_capacity_pages=60, watermark_pages=1, fixed_ns=MS, attn_ps_per_token=50_000,
             prefill_ps_per_token=2_000_000, prefill_chunk_tokens=64, tick_ns=100 * MS)


@pytest.mark.parametrize("kind", [serve.MPC, serve.BBR, serve.PCC])
@pytest.mark.parametrize("seed", [1, 2])
def test_library_matches_oracle_with_variants(kind, seed):
    tr = traces.small_trace(250, seed=seed, mean_gap_ms=15)
    ref0 = _osim(tr, **SMALL)
    t1, t2 = osim.thresholds_from(ref0)
    _same(serve.run(tr, controller=kind, t1=t1, t2=t2, **SMALL), _osim(tr, controller=kind, t1=t1, t2=t2, **SMALL))
    # non-default parameters go through the same path
    over = {serve.MPC: dict(horizon=4, tau=3.0), serve.BBR: dict(cycle=4, margin=0.1),
            serve.PCC: dict(interval=2, gain=0.05)}[kind]
    ora = {ORACLE_NAMES.get(k, k): v for k, v in over.items()}
    _same(serve.run(tr, controller=kind, t1=t1, t2=t2, ctl_params=over, **SMALL),
          _osim(tr, controller=kind, t1=t1, t2=t2, ctl_params=ora, **SMALL))


def test_library_matches_oracle_with_classes():
    tr = traces.small_trace(300, seed=7, mean_gap_ms=12)
    t1, t2 = osim.thresholds_from(_osim(tr, **SMALL))
    cls = np.random.default_rng(3).integers(0, 3, size=len(tr))
    classes = [(1.0, 0), (0.0, 0), (0.5, 40)]
    for kind in (serve.LINEAR, serve.MPC):
        out = serve.run(tr, controller=kind, t1=t1, t2=t2, cls=cls, classes=classes, **SMALL)
        ref = _osim(tr, controller=kind, t1=t1, t2=t2, cls=cls, class_weight=(1.0, 0.0, 0.5),
                    class_bypass=(0, 0, 40), **SMALL)
        _same(out, ref)
        t = out.requests["target"]
        assert (t[cls == 1] == tr.length[cls == 1]).all()              # exempt class
        short = (cls == 2) & (tr.length <= 40)
        assert (t[short] == tr.length[short]).all()                    # bypass


def test_library_matches_oracle_paper_trace_variants():
    cfg = {k: v for k, v in serve.PAPER_SERVER.items() if not k.startswith("live")}
    tr = traces.paper_trace(serve.PAPER_CAPACITY_RPS, seed=0)
    ref0 = _osim(tr, **cfg)
    t1, t2 = osim.thresholds_from(ref0)
    for kind in (serve.MPC, serve.BBR, serve.PCC):
        _same(serve.run(tr, controller=kind, t1=t1, t2=t2, **cfg), _osim(tr, controller=kind, t1=t1, t2=t2, **cfg))


def test_simulator_rejects_bad_classes():
    tr = traces.small_trace(20, seed=1, mean_gap_ms=15)
    with pytest.raises(B.BellmanError):
        serve.run(tr, controller=serve.LINEAR, t1=1.0, t2=2.0, cls=np.full(len(tr), 3), classes=[(1.0, 0)], **SMALL)
    with pytest.raises(B.BellmanError):
        serve.run(tr, controller=serve.LINEAR, t1=1.0, t2=2.0, classes=[(-1.0, 0)], **SMALL)
    with pytest.raises(B.BellmanError):
        serve.run(tr, controller=9, **SMALL)
    with pytest.raises(B.BellmanError):
        serve.run(tr, controller=serve.MPC, t1=2.0, t2=1.0, **SMALL)     # MPC needs t2 > t1
