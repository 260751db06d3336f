"""Seeded synthetic request traces for the serving simulator.

Input generation only: this module draws arrival times and request sizes and
holds none of the simulator's or the controller's arithmetic.  Both the
library's simulator and the oracle's take the arrays it returns.

The paper's trace (Sec. 4, "Setup and trace"): Poisson arrivals whose rate
ramps up, holds and ramps down through two peaks over 22 minutes, the first
at an overload rate (2.5 requests/s where the testbed saturated near 2.4),
the second at a moderate one (1.5 requests/s).  The profile's exact knots are
not given in the text; ``PAPER_PROFILE`` is a reading of them, with rates
expressed as fractions of the simulated server's saturation rate so the same
shape applies to any server model.  Request sizes follow the summarization
workload: prompt tokens uniform in [6000, 12000], unbounded output length
floor(lognormal(median 500, sigma 0.5)) clipped to [1, 1500].
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

NS = 1_000_000_000

# (time s, rate as a fraction of the saturation rate), linear in between.
# 1.0 / 2.4, 2.5 / 2.4 and 1.5 / 2.4 are the paper's base, first-peak and
# second-peak rates over its saturation point; the first peak holds ~90 s.
PAPER_PROFILE = (
    (0.0, 1.0 / 2.4), (60.0, 1.0 / 2.4), (120.0, 2.5 / 2.4), (210.0, 2.5 / 2.4),
    (270.0, 1.0 / 2.4), (600.0, 1.0 / 2.4), (660.0, 1.5 / 2.4), (750.0, 1.5 / 2.4),
    (810.0, 1.0 / 2.4), (1320.0, 1.0 / 2.4),
)


@dataclass
class Trace:
    arrival_ns: np.ndarray   # int64 [R], non-decreasing
    prompt: np.ndarray       # int32 [R], prompt tokens
    length: np.ndarray       # int32 [R], unbounded output tokens (the predicted length L)

    def __len__(self):
        return len(self.arrival_ns)


def rate_at(profile, t):
    """Piecewise-linear rate of ``profile`` at time ``t`` (seconds)."""
    ts = [p[0] for p in profile]
    vs = [p[1] for p in profile]
    return float(np.interp(t, ts, vs))


def poisson_arrivals(profile, capacity_rps, seed, duration_s=None):
    """Arrival times (ns) of a Poisson process with rate
    capacity_rps * profile(t), drawn by thinning a homogeneous process."""
    duration_s = profile[-1][0] if duration_s is None else duration_s
    peak = capacity_rps * max(p[1] for p in profile)
    rng = np.random.default_rng(np.random.SeedSequence([seed, 1]))
    out = []
    t = 0.0
    while True:
        t += rng.exponential(1.0 / peak)
        if t >= duration_s:
            break
        if rng.random() * peak < capacity_rps * rate_at(profile, t):
            out.append(int(t * NS))
    return np.asarray(out, dtype=np.int64)


def request_sizes(n, seed):
    """Prompt tokens U[6000, 12000] and unbounded output lengths
    floor(exp(N(ln 500, 0.5^2))) clipped to [1, 1500]."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 2]))
    prompt = rng.integers(6000, 12000, size=n, endpoint=True).astype(np.int32)
    z = rng.standard_normal(n)
    length = np.clip(np.floor(np.exp(math.log(500.0) + 0.5 * z)), 1, 1500).astype(np.int32)
    return prompt, length


def paper_trace(capacity_rps, seed=0, profile=PAPER_PROFILE, duration_s=None):
    arr = poisson_arrivals(profile, capacity_rps, seed, duration_s)
    prompt, length = request_sizes(len(arr), seed)
    return Trace(arr, prompt, length)


def constant_trace(rps, duration_s, seed=0):
    """Poisson arrivals at a constant rate (used to find the saturation point)."""
    return paper_trace(rps, seed, profile=((0.0, 1.0), (duration_s, 1.0)), duration_s=duration_s)


def small_trace(n, seed=0, mean_gap_ms=50.0, prompt=(64, 512), length=(1, 64)):
    """A short trace with small requests, for quick exact comparisons."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 3]))
    gaps = rng.exponential(mean_gap_ms * 1e6, size=n)
    arr = np.cumsum(gaps).astype(np.int64)
    p = rng.integers(prompt[0], prompt[1], size=n, endpoint=True).astype(np.int32)
    L = rng.integers(length[0], length[1], size=n, endpoint=True).astype(np.int32)
    return Trace(arr, p, L)
