"""Reference oracle for beLLMan's length controller.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the paper states (Sec. 3):
* "Our key proposal": under congestion the controller picks a word-reduction
  rate r between 5% and 20%, predicts the unbounded length L of a queued
  request and asks for N = L * (1 - r); no reduction is enforced without
  congestion.
* "Placeholder for congestion control": congestion is sensed from TBT; the
  trigger sets r = 5%, r rises linearly to 20% at the maximum latency
  threshold, and r is reset when TBT is low.
* "Default unbounded run": T1 is the median TBT of an unbounded run (the
  trigger, r = 5%) and T2 its 75th percentile (r = 20%).
* "beLLMan in action": the scheduler's per-second average TBT is smoothed by a
  moving average over the last 5 seconds; congestion control triggers when the
  average exceeds T1.

Readings where the text is silent (each listed in the design notes):
* r is linear in the moving average between (T1, 5%) and (T2, 20%) and is
  clamped to [5%, 20%]; the trigger is strict (MA > T1); r = 0 when MA <= T1.
* If T2 <= T1 the ramp has no width and r jumps to 20% on trigger.
* The moving average is the mean of the last min(n, 5) samples, summed from
  the oldest to the newest.
* N = floor(L * (1 - r) + 0.5) (round half up), at least 1, and N = L when
  r = 0 or L = 0.  All arithmetic is binary64.
* Thresholds use linear interpolation between order statistics: the p-th
  percentile of n sorted samples sits at fractional index p/100 * (n - 1).
"""
from __future__ import annotations

import math


def percentile_linear(samples, p):
    """p-th percentile by linear interpolation between order statistics."""
    xs = sorted(float(v) for v in samples)
    if not xs:
        raise ValueError("no samples")
    pos = (p / 100.0) * (len(xs) - 1)
    lo = math.floor(pos)
    hi = min(lo + 1, len(xs) - 1)
    frac = pos - lo
    return xs[lo] + (xs[hi] - xs[lo]) * frac


def calibrate_thresholds(tbt_samples):
    """(T1, T2) = (median, 75th percentile) of an unbounded run's TBTs."""
    return percentile_linear(tbt_samples, 50.0), percentile_linear(tbt_samples, 75.0)


class OracleController:
    def __init__(self, t1, t2, window=5, r_min=0.05, r_max=0.20):
        self.t1, self.t2 = float(t1), float(t2)
        self.window = int(window)
        self.r_min, self.r_max = float(r_min), float(r_max)
        self.samples = []
        self.r = 0.0

    def moving_average(self):
        last = self.samples[-self.window:]
        total = 0.0
        for v in last:
            total += v
        return total / len(last)

    def push(self, tbt_avg_1s):
        """Take one per-second TBT average and return the new rate r."""
        self.samples.append(float(tbt_avg_1s))
        ma = self.moving_average()
        if not ma > self.t1:
            self.r = 0.0
        elif self.t2 <= self.t1:
            self.r = self.r_max
        else:
            r = self.r_min + (self.r_max - self.r_min) * (ma - self.t1) / (self.t2 - self.t1)
            self.r = min(max(r, self.r_min), self.r_max)
        return self.r

    def cap(self, predicted_len):
        """Target length N for a request whose unbounded length is L."""
        L = int(predicted_len)
        if L < 0:
            raise ValueError("predicted length must be >= 0")
        if self.r == 0.0 or L == 0:
            return L
        return max(1, math.floor(L * (1.0 - self.r) + 0.5))
