"""Reference closed-loop serving simulator (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper evaluates its controller on a served model under a Poisson trace
(Sec. 4, "Setup and trace", "Default unbounded run", "beLLMan in action"): the
scheduler admits queued requests into continuous batches, reports the
per-second average time between tokens (TBT), and the controller turns the
5-second moving average of that signal into a reduction rate r applied to the
requests as they are queued (Sec. 3, "Our key proposal").  The paper gives the
behaviour, not an algorithm, and serves with vLLM; this is the reading both
simulators implement, step by step in the same order (the server side follows
vLLM's paged KV allocation, chunked prefill and preemption by recomputation):

1. Events up to the current time ``now`` are taken in time order, a tick
   before an arrival at the same instant.  A tick at k*tick_ns averages the TBT
   samples of tokens decoded in ((k-1)*tick_ns, k*tick_ns] and pushes that
   average to the controller (no push for a second without samples).  An
   arrival is queued with target N = cap(L) under the controller's current r
   (N = L without a controller).
2. Admission, first come first served (the head blocks the rest): while fewer
   than ``max_running`` requests run, the head, which must prefill
   P = prompt + generated tokens (generated > 0 after a preemption), is
   admitted if ceil(P / 16) pages can be taken with ``watermark_pages`` left
   free; it takes them and starts prefilling.
3. With nothing running, time jumps to the next arrival.
4. Pages for this iteration's decodes, in running order: a decoding request
   whose next KV position (prompt + generated - 1) falls past its pages needs
   one more; when none is free the most recently admitted running request is
   preempted (pages returned, progress of its prefill dropped, put back at the
   queue head ahead of requests preempted before it in this pass) until the
   page is found or the request itself was preempted.
5. Prefill chunks, in running order: each prefilling request takes up to the
   iteration's remaining budget of ``prefill_chunk_tokens`` prompt tokens
   (no limit when 0).
6. Iteration time, integer nanoseconds:
   fixed_ns + (attn_ps_per_token * KV + prefill_ps_per_token * chunk) // 1000,
   KV = sum over decoding requests of prompt + generated (their KV length
   after this step's append), chunk = prefill tokens taken in step 5.
7. At the end: every decoding request gains a token and contributes one TBT
   sample equal to the iteration time; a request finishing its prefill gains
   a token (its first token, which fixes TTFT, unless it was preempted before)
   and starts decoding; a request whose generated count reaches N finishes and
   returns its pages.  Running order is kept.

Thresholds for a controlled run come from an uncontrolled run: T1 and T2 are
the median and 75th percentile of its per-second TBT averages (Sec. 4,
"Default unbounded run").

Controller variants (Sec. 5, "Toward novel LLM congestion control"): with
``controller`` 2, 3 or 4 the MPC, BBR-style or PCC controller of
``oracle.controller`` takes the tick instead, observing (samples > 0, their
mean TBT in ns, the tokens they decoded, the tick in seconds); a tick
without samples is still an observation for them.  Per-class policies
("Nuanced fairness issues"): request j of class c gets
``cap_for_class(L, r, weight[c], bypass_len[c], r_max)``.
"""
from __future__ import annotations

from collections import deque
from dataclasses import dataclass, field

from .controller import (OracleBBR, OracleController, OracleLinear, OracleMPC, OraclePCC, calibrate_thresholds,
                         cap_for_class)

PAGE = 16
QUEUED, PREFILL, DECODE, DONE = 1, 2, 3, 4


@dataclass
class SimConfig:
    max_running: int = 256
    kv_capacity_pages: int = 65536
    fixed_ns: int = 1_000_000
    attn_ps_per_token: int = 10_000
    prefill_ps_per_token: int = 9_000_000
    tick_ns: int = 1_000_000_000
    prefill_chunk_tokens: int = 0
    watermark_pages: int = 0
    controller: int = 0          # 0 none, 1 linear, 2 MPC, 3 BBR-style, 4 PCC
    t1: float = 0.0
    t2: float = 0.0
    window: int = 5
    r_min: float = 0.05
    r_max: float = 0.20
    ctl_params: dict = field(default_factory=dict)   # variant parameters (oracle.controller names)
    class_weight: tuple = (1.0,)                      # per class: r multiplier
    class_bypass: tuple = (0,)                        # per class: lengths at or below are not reduced


@dataclass
class SimResult:
    target: list
    r_at_queue: list
    admit_ns: list       # first admission
    first_ns: list
    finish_ns: list
    preemptions: list    # per request
    ticks: list = field(default_factory=list)  # (t_ns, samples, tbt_sum_ns, r_after, queued, running)
    iterations: int = 0
    log: list = field(default_factory=list)    # per iteration: (end_ns, dt_ns, decoding, chunk,
    #                                            running and queued at the start of step 4)


def ceil_pages(tokens):
    return -(-int(tokens) // PAGE)


def make_controller(cfg: SimConfig):
    k = int(cfg.controller)
    if k == 0:
        return None
    if k == 1:
        return OracleLinear(cfg.t1, cfg.t2, cfg.window, cfg.r_min, cfg.r_max)
    if k == 2:
        return OracleMPC(cfg.t1, cfg.t2, window=cfg.window, r_min=cfg.r_min, r_max=cfg.r_max, **cfg.ctl_params)
    if k == 3:
        return OracleBBR(r_max=cfg.r_max, **cfg.ctl_params)
    if k == 4:
        return OraclePCC(cfg.t1, cfg.t2, r_max=cfg.r_max, **cfg.ctl_params)
    raise ValueError(f"controller {k}")


def simulate(arrival_ns, prompt, length, cfg: SimConfig, cls=None) -> SimResult:
    n = len(arrival_ns)
    arrival_ns = [int(v) for v in arrival_ns]
    prompt = [int(v) for v in prompt]
    length = [int(v) for v in length]
    cls = [0] * n if cls is None else [int(v) for v in cls]
    for j in range(n):
        if ceil_pages(prompt[j] + length[j]) + cfg.watermark_pages > cfg.kv_capacity_pages:
            raise ValueError(f"request {j} does not fit the page budget")
    ctl = make_controller(cfg)
    res = SimResult([0] * n, [0.0] * n, [-1] * n, [-1] * n, [-1] * n, [0] * n)
    state = [0] * n
    gen = [0] * n
    held = [0] * n        # pages held
    todo = [0] * n        # prefill tokens of the current admission
    filled = [0] * n      # prefill tokens done
    queue = deque()
    running = []
    pages_free = cfg.kv_capacity_pages
    windows = {}
    now = 0
    next_tick = cfg.tick_ns
    i = 0
    done = 0
    while done < n:
        # 1. ticks and arrivals up to now, in time order
        while True:
            ta = arrival_ns[i] if i < n else None
            if next_tick <= now and (ta is None or next_tick <= ta):
                s, c = windows.pop(next_tick // cfg.tick_ns, (0, 0))
                if ctl is not None:
                    # mean TBT in ns (the thresholds' unit), tokens, tick in seconds
                    ctl.observe(c > 0, s / c if c > 0 else 0.0, float(c), cfg.tick_ns / 1e9)
                res.ticks.append((next_tick, c, s, ctl.r if ctl else 0.0, len(queue), len(running)))
                next_tick += cfg.tick_ns
                continue
            if ta is not None and ta <= now:
                k = cls[i]
                res.target[i] = (cap_for_class(length[i], ctl.r, cfg.class_weight[k], cfg.class_bypass[k], cfg.r_max)
                                 if ctl else length[i])
                res.r_at_queue[i] = ctl.r if ctl else 0.0
                state[i] = QUEUED
                queue.append(i)
                i += 1
                continue
            break
        # 2. admission
        while queue and len(running) < cfg.max_running:
            j = queue[0]
            P = prompt[j] + gen[j]
            need = ceil_pages(P)
            if pages_free - need < cfg.watermark_pages:
                break
            queue.popleft()
            pages_free -= need
            held[j] = need
            todo[j] = P
            filled[j] = 0
            state[j] = PREFILL
            running.append(j)
            if res.admit_ns[j] < 0:
                res.admit_ns[j] = now
        # 3. idle
        if not running:
            now = arrival_ns[i]
            continue
        run0, queued0 = len(running), len(queue)
        # 4. pages for the decodes
        k = 0
        while k < len(running):
            j = running[k]
            if state[j] == DECODE and (prompt[j] + gen[j] - 1) // PAGE >= held[j]:
                victim_of_self = False
                back = []
                while pages_free == 0:
                    v = running.pop()
                    pages_free += held[v]
                    held[v] = 0
                    state[v] = QUEUED
                    res.preemptions[v] += 1
                    back.append(v)
                    if v == j:
                        victim_of_self = True
                        break
                for v in back:
                    queue.appendleft(v)
                if victim_of_self:
                    continue          # j is gone; running[k] is now past the end
                pages_free -= 1
                held[j] += 1
            k += 1
        # 5. prefill chunks
        budget = cfg.prefill_chunk_tokens if cfg.prefill_chunk_tokens > 0 else None
        chunk = 0
        completing = []
        for j in running:
            if state[j] != PREFILL:
                continue
            t = todo[j] - filled[j]
            if budget is not None:
                t = min(t, budget)
                budget -= t
            filled[j] += t
            chunk += t
            if filled[j] == todo[j]:
                completing.append(j)
            if budget == 0:
                break
        # 6. iteration time
        kv = 0
        decoding = 0
        for j in running:
            if state[j] == DECODE:
                kv += prompt[j] + gen[j]
                decoding += 1
        dt = cfg.fixed_ns + (cfg.attn_ps_per_token * kv + cfg.prefill_ps_per_token * chunk) // 1000
        end = now + dt
        # 7. tokens, finishes
        if decoding:
            w = -(-end // cfg.tick_ns)
            s, c = windows.get(w, (0, 0))
            windows[w] = (s + dt * decoding, c + decoding)
        completing = set(completing)
        still = []
        for j in running:
            if state[j] == DECODE:
                gen[j] += 1
            elif j in completing:
                gen[j] += 1
                if res.first_ns[j] < 0:
                    res.first_ns[j] = end
                state[j] = DECODE
            if state[j] == DECODE and gen[j] >= res.target[j]:
                res.finish_ns[j] = end
                pages_free += held[j]
                held[j] = 0
                state[j] = DONE
                done += 1
            else:
                still.append(j)
        res.log.append((end, dt, decoding, chunk, run0, queued0))
        running = still
        now = end
        res.iterations += 1
    return res


def thresholds_from(result: SimResult):
    """(T1, T2) from the per-second TBT averages of an uncontrolled run."""
    samples = [s / c for (_, c, s, _, _, _) in result.ticks if c > 0]
    return calibrate_thresholds(samples)

