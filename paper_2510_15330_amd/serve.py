"""The closed-loop serving model (bellman_sim_run) from Python.

``run`` is the binding: it marshals a ``traces.Trace`` and configuration
keywords (the fields of bellman_sim_config_t) into the library, where the
model runs, and returns the per-request and per-tick records as numpy
structured arrays plus the run's totals.  The rest of the module is the
experiment driver on top of those records, computed on the host:
calibrating the controller's thresholds from an unbounded run
(``thresholds``), the paper's bounded-versus-unbounded experiment
(``paper_experiment``, ``summarize``), per-run latency and throughput
metrics (``run_metrics``) and the comparison of controller variants
(``compare_controllers``).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np

from . import _binding

NO_CONTROL, LINEAR, MPC, BBR, PCC = 0, 1, 2, 3, 4


class SimConfig(ctypes.Structure):
    _fields_ = [
        ("max_running", ctypes.c_int32), ("controller", ctypes.c_int32),
        ("kv_capacity_pages", ctypes.c_int64), ("watermark_pages", ctypes.c_int64),
        ("fixed_ns", ctypes.c_int64), ("attn_ps_per_token", ctypes.c_int64),
        ("prefill_ps_per_token", ctypes.c_int64), ("tick_ns", ctypes.c_int64),
        ("t1", ctypes.c_double), ("t2", ctypes.c_double),
        ("window", ctypes.c_int32), ("prefill_chunk_tokens", ctypes.c_int32),
        ("r_min", ctypes.c_double), ("r_max", ctypes.c_double),
        ("live", ctypes.c_int32), ("live_layers", ctypes.c_int32), ("live_q_heads", ctypes.c_int32),
        ("live_kv_heads", ctypes.c_int32), ("live_head_dim", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("stream", ctypes.c_void_p),
        ("ctl_params", ctypes.POINTER(_binding.CtlParams)), ("req_class", ctypes.c_void_p),
        ("classes", ctypes.POINTER(_binding.ClassPolicy)), ("n_classes", ctypes.c_int32),
        ("reserved2", ctypes.c_int32),
    ]


class SimRequest(ctypes.Structure):
    _fields_ = [("admit_ns", ctypes.c_int64), ("first_ns", ctypes.c_int64), ("finish_ns", ctypes.c_int64),
                ("target", ctypes.c_int32), ("preemptions", ctypes.c_int32), ("r_at_queue", ctypes.c_double)]


class SimTick(ctypes.Structure):
    _fields_ = [("t_ns", ctypes.c_int64), ("tokens", ctypes.c_int64), ("tbt_sum_ns", ctypes.c_int64),
                ("r", ctypes.c_double), ("queued", ctypes.c_int32), ("running", ctypes.c_int32)]


class SimIteration(ctypes.Structure):
    _fields_ = [("end_ns", ctypes.c_int64), ("dt_ns", ctypes.c_int64), ("decoding", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("running", ctypes.c_int32), ("queued", ctypes.c_int32)]


class SimStats(ctypes.Structure):
    _fields_ = [("iterations", ctypes.c_int64), ("ticks", ctypes.c_int64), ("end_ns", ctypes.c_int64),
                ("preemptions", ctypes.c_int64), ("live_gpu_ms", ctypes.c_double),
                ("live_kv_bytes", ctypes.c_int64)]


REQUEST_DTYPE = np.dtype([("admit_ns", "<i8"), ("first_ns", "<i8"), ("finish_ns", "<i8"),
                          ("target", "<i4"), ("preemptions", "<i4"), ("r_at_queue", "<f8")])
TICK_DTYPE = np.dtype([("t_ns", "<i8"), ("tokens", "<i8"), ("tbt_sum_ns", "<i8"), ("r", "<f8"),
                       ("queued", "<i4"), ("running", "<i4")])
ITERATION_DTYPE = np.dtype([("end_ns", "<i8"), ("dt_ns", "<i8"), ("decoding", "<i4"), ("chunk", "<i4"),
                            ("running", "<i4"), ("queued", "<i4")])
assert REQUEST_DTYPE.itemsize == ctypes.sizeof(SimRequest)
assert ITERATION_DTYPE.itemsize == ctypes.sizeof(SimIteration)
assert TICK_DTYPE.itemsize == ctypes.sizeof(SimTick)

DEFAULTS = dict(max_running=256, controller=NO_CONTROL, kv_capacity_pages=65536, watermark_pages=0,
                fixed_ns=1_000_000, attn_ps_per_token=10_000, prefill_ps_per_token=9_000_000,
                tick_ns=1_000_000_000, t1=0.0, t2=0.0, window=5, prefill_chunk_tokens=0,
                r_min=0.05, r_max=0.20, live=0, live_layers=62, live_q_heads=4, live_kv_heads=2,
                live_head_dim=128, reserved=0)


@dataclass
class SimOutput:
    requests: np.ndarray   # REQUEST_DTYPE [R]
    ticks: np.ndarray      # TICK_DTYPE [T]
    log: np.ndarray        # ITERATION_DTYPE [I] (first max_iterations iterations)
    iterations: int
    end_ns: int
    preemptions: int
    live_gpu_ms: float
    live_kv_bytes: int


def _lib():
    lib = _binding.library()
    if not getattr(lib, "_sim_bound", False):
        lib.bellman_sim_run.argtypes = [ctypes.POINTER(SimConfig), ctypes.c_int64, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.POINTER(SimStats)]
        lib.bellman_sim_run.restype = ctypes.c_int
        lib._sim_bound = True
    return lib


def make_config(stream=None, **kw) -> SimConfig:
    vals = dict(DEFAULTS)
    for k, v in kw.items():
        if k not in vals:
            raise TypeError(f"unknown simulator option {k!r}")
        vals[k] = v
    c = SimConfig()
    for k, v in vals.items():
        setattr(c, k, v)
    c.stream = stream
    return c


def run(trace, stream=None, max_ticks=None, max_iterations=0, ctl_params=None, cls=None, classes=None,
        **kw) -> SimOutput:
    """``ctl_params``: parameter overrides of the controller variant (names of
    bellman_ctl_params_t; defaults otherwise, with t1, t2, window, r_min,
    r_max taken from the keywords); ``cls``: per-request class; ``classes``:
    a (weight, bypass_len) policy per class."""
    arr = np.ascontiguousarray(trace.arrival_ns, dtype=np.int64)
    prompt = np.ascontiguousarray(trace.prompt, dtype=np.int32)
    length = np.ascontiguousarray(trace.length, dtype=np.int32)
    n = len(arr)
    cfg = make_config(stream=stream, **kw)
    keep = []
    if ctl_params is not None:
        base = {k: kw[k] for k in ("window", "r_min", "r_max") if k in kw}
        base.update(ctl_params)
        p = _binding.ctl_params(cfg.controller, cfg.t1, cfg.t2, **{k: v for k, v in base.items()})
        keep.append(p)
        cfg.ctl_params = ctypes.pointer(p)
    if cls is not None:
        c = np.ascontiguousarray(cls, dtype=np.int32)
        if c.shape != (n,):
            raise ValueError("cls must give one class per request")
        keep.append(c)
        cfg.req_class = c.ctypes.data
    if classes is not None:
        arrp = (_binding.ClassPolicy * len(classes))(*[_binding.ClassPolicy(float(w), int(b), 0) for w, b in classes])
        keep.append(arrp)
        cfg.classes = arrp
        cfg.n_classes = len(classes)
    elif cls is not None:
        cfg.n_classes = int(np.max(cls)) + 1 if n else 1
    if max_ticks is None:
        max_ticks = 1 << 16
    req = np.zeros(n, dtype=REQUEST_DTYPE)
    ticks = np.zeros(max_ticks, dtype=TICK_DTYPE)
    its = np.zeros(max(max_iterations, 1), dtype=ITERATION_DTYPE)
    st = SimStats()
    rc = _lib().bellman_sim_run(ctypes.byref(cfg), n, arr.ctypes.data, prompt.ctypes.data, length.ctypes.data,
                                req.ctypes.data, ticks.ctypes.data, max_ticks, its.ctypes.data, max_iterations,
                                ctypes.byref(st))
    _binding._check(rc)
    if st.ticks > max_ticks:
        raise RuntimeError(f"{st.ticks} ticks, only {max_ticks} stored; pass a larger max_ticks")
    return SimOutput(req, ticks[:st.ticks].copy(), its[:min(st.iterations, max_iterations)].copy(),
                     int(st.iterations), int(st.end_ns), int(st.preemptions),
                     float(st.live_gpu_ms), int(st.live_kv_bytes))


def thresholds(out: SimOutput):
    """(T1, T2): median and 75th percentile of the per-second TBT averages of
    an uncontrolled run, computed by the library's calibration routine."""
    t = out.ticks[out.ticks["tokens"] > 0]
    samples = np.ascontiguousarray(t["tbt_sum_ns"] / t["tokens"], dtype=np.float64)
    t1, t2 = ctypes.c_double(), ctypes.c_double()
    lib = _binding.library()
    _binding._check(lib.bellman_calibrate_thresholds(samples.ctypes.data, len(samples),
                                                     ctypes.byref(t1), ctypes.byref(t2)))
    return t1.value, t2.value


# ----------------------------------------------------------- experiment --
# The paper's evaluation (Sec. 4): an uncontrolled run over the trace, then a
# controlled run whose thresholds are the median and 75th percentile of the
# uncontrolled run's per-second TBT.  Server model: a Gemma-3-27B-sized model
# at tensor parallelism 8 on MI355X, per GPU 4 query heads and 2 KV heads of
# dim 128 in each of 62 layers.  Per iteration: 2.5 ms for the dense layers
# and collectives; attention 62 layers x 1 KiB per KV token at ~5.7 TB/s
# (11.1 ns per KV token); prefill ~7.3 GFLOP per prompt token per GPU at
# ~1 PFLOP/s (7.3 us per token); a 256-request running limit (the usual
# serving default) and a KV budget of 65,536 pages (~1M tokens, the KV room an
# 80 GB GPU leaves next to its weight shard, so that admission is KV-bound as
# on the paper's testbed).  Under this model the queue starts to grow at ~7.4
# requests/s; the trace's rates are scaled so that this point plays the role
# of the paper's 2.4 requests/s.
PAPER_SERVER = dict(max_running=256, kv_capacity_pages=65536, watermark_pages=655, fixed_ns=2_500_000,
                    attn_ps_per_token=11_100, prefill_ps_per_token=7_300_000, prefill_chunk_tokens=2048,
                    live_layers=62, live_q_heads=4, live_kv_heads=2, live_head_dim=128)
PAPER_CAPACITY_RPS = 7.4


def summarize(trace, unbounded: SimOutput, bounded: SimOutput, t1, t2, window=(130.0, 500.0)):
    """Numbers the paper reports for its trace (Sec. 4, "beLLMan in action",
    "beLLMan energy savings"), measured on the two runs."""
    arr = trace.arrival_ns.astype(np.float64) / 1e9

    def lat(o):
        r = o.requests
        return dict(queue=(r["admit_ns"] / 1e9 - arr), ttft=(r["first_ns"] / 1e9 - arr),
                    e2e=(r["finish_ns"] / 1e9 - arr))

    lu, lb = lat(unbounded), lat(bounded)
    tk = bounded.ticks
    on = tk["t_ns"][tk["r"] > 0] / 1e9
    active = bounded.requests["r_at_queue"] > 0
    w0, w1 = window

    def in_window(o):
        f = o.requests["finish_ns"] / 1e9
        return int(((f >= w0) & (f < w1)).sum())

    def tokens_in_window(o):
        t = o.ticks
        sel = (t["t_ns"] / 1e9 > w0) & (t["t_ns"] / 1e9 <= w1)
        return int(t["tokens"][sel].sum())

    def tbt_ms(o):
        t = o.ticks[o.ticks["tokens"] > 0]
        return t["tbt_sum_ns"] / t["tokens"] / 1e6

    ratio = lu["e2e"] / lb["e2e"]
    # periods with r > 0, from tick to tick
    onf = (tk["r"] > 0).astype(np.int8)
    edges = np.flatnonzero(np.diff(np.concatenate([[0], onf, [0]])))
    periods = sorted(((float(tk["t_ns"][a] / 1e9), float(tk["t_ns"][b - 1] / 1e9)) for a, b in
                      zip(edges[::2], edges[1::2])), key=lambda p: p[0] - p[1])
    return {
        "requests": int(len(trace)),
        "t1_ms": t1 / 1e6, "t2_ms": t2 / 1e6,
        "control_on_s": float(on.min()) if len(on) else None,
        "control_off_s": float(on.max()) if len(on) else None,
        "control_active_fraction": float(onf.mean()) if len(onf) else 0.0,
        "control_longest_periods_s": periods[:3],
        "median_r_when_active": float(np.median(bounded.requests["r_at_queue"][active])) if active.any() else 0.0,
        "requests_capped": int(active.sum()),
        "e2e_p50_s": [float(np.median(lu["e2e"])), float(np.median(lb["e2e"]))],
        "e2e_p99_s": [float(np.percentile(lu["e2e"], 99)), float(np.percentile(lb["e2e"], 99))],
        "e2e_max_s": [float(lu["e2e"].max()), float(lb["e2e"].max())],
        "e2e_max_reduction": float(ratio.max()),
        "queue_max_s": [float(lu["queue"].max()), float(lb["queue"].max())],
        "ttft_p99_s": [float(np.percentile(lu["ttft"], 99)), float(np.percentile(lb["ttft"], 99))],
        "tbt_max_ms": [float(tbt_ms(unbounded).max()), float(tbt_ms(bounded).max())],
        "completed_in_window": [in_window(unbounded), in_window(bounded)],
        "decode_tokens_in_window": [tokens_in_window(unbounded), tokens_in_window(bounded)],
        "window_s": [w0, w1],
        "end_s": [unbounded.end_ns / 1e9, bounded.end_ns / 1e9],
    }


def paper_experiment(seed=0, live=False, stream=None, capacity_rps=PAPER_CAPACITY_RPS, duration_s=None,
                     log=None, **server):
    """Uncontrolled run, thresholds, controlled run; returns (summary, runs)."""
    import time

    from . import traces
    cfg = dict(PAPER_SERVER)
    cfg.update(server)
    tr = traces.paper_trace(capacity_rps, seed=seed, duration_s=duration_s)
    t0 = time.perf_counter()
    unb = run(tr, stream=stream, live=int(live), controller=NO_CONTROL, **cfg)
    if log:
        log(f"[serve] uncontrolled run: {len(tr)} requests, {unb.iterations} iterations, "
            f"{time.perf_counter() - t0:.1f} s")
    t1, t2 = thresholds(unb)
    t0 = time.perf_counter()
    bnd = run(tr, stream=stream, live=int(live), controller=LINEAR, t1=t1, t2=t2, **cfg)
    if log:
        log(f"[serve] controlled run: {bnd.iterations} iterations, {time.perf_counter() - t0:.1f} s")
    s = summarize(tr, unb, bnd, t1, t2)
    s["mode"] = "live" if live else "model"
    if live:
        s["live_attention"] = {
            "gpu_ms": [unb.live_gpu_ms, bnd.live_gpu_ms],
            "kv_bytes": [unb.live_kv_bytes, bnd.live_kv_bytes],
            "gb_per_s": [unb.live_kv_bytes / max(unb.live_gpu_ms, 1e-9) / 1e6,
                         bnd.live_kv_bytes / max(bnd.live_gpu_ms, 1e-9) / 1e6],
        }
    return s, (tr, unb, bnd)


CONTROLLER_NAMES = {NO_CONTROL: "none", LINEAR: "linear", MPC: "mpc", BBR: "bbr", PCC: "pcc"}


def run_metrics(trace, out: SimOutput, base: SimOutput | None = None):
    """Latency, control activity, output kept and busy time of one run."""
    arr = trace.arrival_ns.astype(np.float64) / 1e9
    r = out.requests
    e2e = r["finish_ns"] / 1e9 - arr
    ttft = r["first_ns"] / 1e9 - arr
    rs = out.ticks["r"]
    busy_s = float(out.log["dt_ns"].sum()) / 1e9 if len(out.log) else float("nan")
    m = {
        "e2e_p50_s": float(np.median(e2e)), "e2e_p99_s": float(np.percentile(e2e, 99)),
        "e2e_max_s": float(e2e.max()), "ttft_p99_s": float(np.percentile(ttft, 99)),
        "queue_max_s": float((r["admit_ns"] / 1e9 - arr).max()),
        "control_active_fraction": float((rs > 0).mean()) if len(rs) else 0.0,
        "rate_switches": int(np.count_nonzero(np.diff((rs > 0).astype(np.int8)))) if len(rs) else 0,
        "mean_abs_rate_change": float(np.abs(np.diff(rs)).mean()) if len(rs) > 1 else 0.0,
        "mean_r": float(r["r_at_queue"].mean()),
        "output_kept": float(r["target"].sum() / trace.length.sum()),
        "busy_s": busy_s,
        "end_s": out.end_ns / 1e9,
        "preemptions": out.preemptions,
    }
    if base is not None and len(base.log) and len(out.log):
        m["busy_vs_uncontrolled"] = busy_s / (float(base.log["dt_ns"].sum()) / 1e9)
    return m


def compare_controllers(seed=0, duration_s=None, capacity_rps=PAPER_CAPACITY_RPS, kinds=(LINEAR, MPC, BBR, PCC),
                        cls=None, classes=None, log=None, **server):
    """Uncontrolled run, thresholds from it, then one run per controller kind
    on the same trace (model mode); returns {name: metrics}."""
    from . import traces
    cfg = dict(PAPER_SERVER)
    cfg.update(server)
    cfg = {k: v for k, v in cfg.items() if not k.startswith("live")}
    tr = traces.paper_trace(capacity_rps, seed=seed, duration_s=duration_s)
    big = 1 << 23
    unb = run(tr, controller=NO_CONTROL, max_iterations=big, **cfg)
    t1, t2 = thresholds(unb)
    res = {"none": run_metrics(tr, unb), "t1_ms": t1 / 1e6, "t2_ms": t2 / 1e6, "requests": len(tr)}
    for k in kinds:
        out = run(tr, controller=k, t1=t1, t2=t2, max_iterations=big, cls=cls, classes=classes, **cfg)
        res[CONTROLLER_NAMES[k]] = run_metrics(tr, out, unb)
        if cls is not None:
            per = {}
            for c in np.unique(cls):
                sel = np.asarray(cls) == c
                e2e = out.requests["finish_ns"][sel] / 1e9 - tr.arrival_ns[sel] / 1e9
                per[int(c)] = {"requests": int(sel.sum()),
                               "output_kept": float(out.requests["target"][sel].sum() / tr.length[sel].sum()),
                               "e2e_p50_s": float(np.median(e2e))}
            res[CONTROLLER_NAMES[k]]["classes"] = per
        if log:
            log(f"[serve] {CONTROLLER_NAMES[k]}: done")
    return res


def main():
    import argparse
    import json
    ap = argparse.ArgumentParser(description="beLLMan closed-loop serving model over the paper's trace")
    ap.add_argument("--live", action="store_true", help="time the real kernels on the GPU for the attention term")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--duration", type=float, default=None, help="trace length in seconds (default: all 1320 s)")
    ap.add_argument("--compare", action="store_true",
                    help="model mode: the linear, MPC, BBR-style and PCC controllers on the same trace")
    args = ap.parse_args()
    import sys
    if args.compare:
        print(json.dumps(compare_controllers(seed=args.seed, duration_s=args.duration,
                                             log=lambda m: print(m, file=sys.stderr, flush=True))), flush=True)
        return
    stream = None
    if args.live:
        import torch
        stream = torch.cuda.current_stream().cuda_stream
    s, _ = paper_experiment(seed=args.seed, live=args.live, stream=stream, duration_s=args.duration,
                            log=lambda m: print(m, file=sys.stderr, flush=True))
    print(json.dumps(s), flush=True)


if __name__ == "__main__":
    main()
