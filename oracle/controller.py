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


# ------------------------------------------------------------------ variants
#
# The paper's future-work section (Sec. 5, "Toward novel LLM congestion
# control", "Nuanced fairness issues") names three other controllers and
# per-class policies without giving algorithms.  What it states:
# * MPC: predict the load and set r ahead of it, minimising a cost over a
#   moving horizon that includes latency, output quality and energy, and
#   avoid oscillations in r.
# * BBR-style: run at the equivalent of Kleinrock's point, keeping TBT low
#   while the served tokens/s are at their maximum.
# * PCC: run micro-experiments with different r and move r along a measured
#   utility that combines latency and response quality.
# * Classes: r may differ per class (e.g. r = 0 for coding); very short
#   outputs may bypass the reduction; one r per batch within a class.
# The readings below are this library's; every step is written out so that
# the C++ controllers can follow it operation for operation.  A controller
# sees one observation per tick: whether TBT samples arrived, their mean
# TBT, the tokens they decoded, and the tick length.

def _clamp(x, lo, hi):
    return min(max(x, lo), hi)


class OracleMPC:
    """Receding-horizon choice of r over a grid.

    Per tick with samples: once `window` samples exist, the last `window` get a
    least squares line (slope s per tick, value v at the newest sample);
    before that s = 0 and v is the newest sample.  The floor b is the minimum
    of the last floor_window samples.
    For a candidate rc the prediction h ticks ahead is
        u_h  = max(v + s h, b)                     (load trend, not below b)
        f_h  = 1 - exp(-h / tau)                   (share of decode work from
                                                    requests capped at rc)
        y_h  = b + (u_h - b) ((1 - f_h) + f_h (1 - rc) / (1 - r))
    and the cost
        J = sum_h w_lat (max(0, y_h - t1) / (t2 - t1))^2
            + horizon (w_quality - w_energy) rc + w_delta ((rc - r) / r_max)^2.
    Candidates: 0, then r_min, r_min + step, ... (while below r_max), r_max;
    the first candidate with the least J wins.  Ticks without samples keep r.
    """

    def __init__(self, t1, t2, window=5, r_min=0.05, r_max=0.20, horizon=10, tau=20.0, floor_window=60,
                 w_lat=1.0, w_quality=0.25, w_energy=0.1, w_delta=0.2, step=0.01):
        if not t2 > t1:
            raise ValueError("MPC needs t2 > t1")
        self.t1, self.t2 = float(t1), float(t2)
        self.window, self.horizon, self.floor_window = int(window), int(horizon), int(floor_window)
        self.r_min, self.r_max, self.tau, self.step = float(r_min), float(r_max), float(tau), float(step)
        self.w_lat, self.w_quality, self.w_energy, self.w_delta = float(w_lat), float(w_quality), float(w_energy), float(w_delta)
        self.samples = []
        self.r = 0.0

    def candidates(self):
        out = [0.0]
        i = 0
        while True:
            rc = self.r_min + i * self.step
            if not rc < self.r_max:
                break
            out.append(rc)
            i += 1
        out.append(self.r_max)
        return out

    def trend(self):
        m = self.window
        if len(self.samples) < m or m < 2:
            return 0.0, self.samples[-1]
        ys = self.samples[-m:]
        tm = (m - 1) / 2.0
        total = 0.0
        for y in ys:
            total += y
        ym = total / m
        sxy = 0.0
        sxx = 0.0
        for t, y in enumerate(ys):
            sxy += (t - tm) * (y - ym)
            sxx += (t - tm) * (t - tm)
        s = sxy / sxx
        return s, ym + s * ((m - 1) - tm)

    def cost(self, rc, s, v, b):
        J = 0.0
        for h in range(1, self.horizon + 1):
            u = max(v + s * h, b)
            f = 1.0 - math.exp(-h / self.tau)
            y = b + (u - b) * ((1.0 - f) + f * (1.0 - rc) / (1.0 - self.r))
            e = max(0.0, y - self.t1) / (self.t2 - self.t1)
            J += self.w_lat * e * e
        d = (rc - self.r) / self.r_max
        return J + self.horizon * (self.w_quality - self.w_energy) * rc + self.w_delta * d * d

    def observe(self, has_sample, tbt=0.0, tokens=0.0, tick_s=1.0):
        if not has_sample:
            return self.r
        self.samples.append(float(tbt))
        s, v = self.trend()
        b = min(self.samples[-self.floor_window:])
        best, best_J = 0.0, math.inf
        for rc in self.candidates():
            J = self.cost(rc, s, v, b)
            if J < best_J:
                best, best_J = rc, J
        self.r = best
        return self.r


class OracleBBR:
    """Two estimators and a gain cycle, after BBR.

    x = tokens / tick_s is the delivery rate of a tick; BtlBw is the largest x
    of the last bw_window ticks and RTprop the smallest TBT of the last
    rt_window ticks with samples.  On a tick with samples:
      * past the knee (TBT > RTprop (1 + margin) while x >= (1 - margin) BtlBw):
        r_base += step (capped at r_max);
      * near the floor (TBT <= RTprop (1 + margin / 2)): r_base -= step (at least 0);
      * otherwise r_base holds.
    The applied rate cycles like BBR's pacing gain over `cycle` ticks: the
    first tick of a cycle probes at r_base - probe, the second drains at
    r_base + probe, the rest cruise at r_base; clamped to [0, r_max].
    """

    def __init__(self, r_max=0.20, bw_window=10, rt_window=30, margin=0.25, step=0.02, probe=0.02, cycle=8):
        self.r_max, self.margin, self.step, self.probe = float(r_max), float(margin), float(step), float(probe)
        self.bw_window, self.rt_window, self.cycle = int(bw_window), int(rt_window), int(cycle)
        self.xs, self.ys = [], []
        self.ticks = 0
        self.r_base = 0.0
        self.r = 0.0

    def observe(self, has_sample, tbt=0.0, tokens=0.0, tick_s=1.0):
        x = float(tokens) / float(tick_s)
        self.xs.append(x)
        self.ticks += 1
        if has_sample:
            self.ys.append(float(tbt))
            btlbw = max(self.xs[-self.bw_window:])
            rtprop = min(self.ys[-self.rt_window:])
            if tbt > rtprop * (1.0 + self.margin) and x >= (1.0 - self.margin) * btlbw:
                self.r_base = min(self.r_base + self.step, self.r_max)
            elif tbt <= rtprop * (1.0 + self.margin / 2.0):
                self.r_base = max(self.r_base - self.step, 0.0)
        phase = (self.ticks - 1) % self.cycle
        off = -self.probe if phase == 0 else (self.probe if phase == 1 else 0.0)
        self.r = _clamp(self.r_base + off, 0.0, self.r_max)
        return self.r


class OraclePCC:
    """Paired micro-experiments and a gradient step, after PCC Vivace.

    Rounds of two monitor intervals of `interval` ticks each run at
    r_center + epsilon and r_center - epsilon (clamped to [0, r_max]); the
    order alternates between rounds, the first round going up first.  An
    interval's utility is
        U = -w_lat max(0, ybar - t1) / (t2 - t1) - w_quality r_mi / r_max,
    ybar the mean of the TBT samples it saw (no latency term without
    samples).  After a round, with the two intervals' (r, U) pairs,
    g = (U_a - U_b) / (r_a - r_b) (0 when the rates coincide) and
    r_center = clamp(r_center + gain g, 0, r_max).  The applied rate is the
    running interval's.
    """

    def __init__(self, t1, t2, r_max=0.20, interval=10, epsilon=0.02, gain=0.02, w_lat=1.0, w_quality=0.5):
        if not t2 > t1:
            raise ValueError("PCC needs t2 > t1")
        self.t1, self.t2, self.r_max = float(t1), float(t2), float(r_max)
        self.interval, self.epsilon, self.gain = int(interval), float(epsilon), float(gain)
        self.w_lat, self.w_quality = float(w_lat), float(w_quality)
        self.center = 0.0
        self.round = 0          # rounds completed
        self.second = False     # running the round's second interval
        self.acc, self.n, self.ticks = 0.0, 0, 0
        self.first = None       # (r, U) of the round's first interval
        self.r = self._rate()

    def _rate(self):
        up = (self.round % 2 == 0) != self.second
        d = self.epsilon if up else -self.epsilon
        return _clamp(self.center + d, 0.0, self.r_max)

    def observe(self, has_sample, tbt=0.0, tokens=0.0, tick_s=1.0):
        if has_sample:
            self.acc += float(tbt)
            self.n += 1
        self.ticks += 1
        if self.ticks == self.interval:
            lat = 0.0
            if self.n:
                lat = max(0.0, self.acc / self.n - self.t1) / (self.t2 - self.t1)
            U = -self.w_lat * lat - self.w_quality * self.r / self.r_max
            if not self.second:
                self.first = (self.r, U)
                self.second = True
            else:
                ra, Ua = self.first
                g = 0.0 if ra == self.r else (Ua - U) / (ra - self.r)
                self.center = _clamp(self.center + self.gain * g, 0.0, self.r_max)
                self.second = False
                self.round += 1
            self.acc, self.n, self.ticks = 0.0, 0, 0
            self.r = self._rate()
        return self.r


class OracleLinear(OracleController):
    """The paper's controller behind the tick interface."""

    def observe(self, has_sample, tbt=0.0, tokens=0.0, tick_s=1.0):
        if has_sample:
            self.push(tbt)
        return self.r


def cap_for_class(predicted_len, r, weight=1.0, bypass_len=0, r_max=0.20):
    """Target length under a class policy: outputs predicted at or below
    bypass_len are not reduced; otherwise the class applies
    rc = min(weight r, r_max) (weight 0 exempts the class)."""
    L = int(predicted_len)
    if L < 0:
        raise ValueError("predicted length must be >= 0")
    if L <= bypass_len:
        return L
    rc = min(weight * r, r_max)
    if rc == 0.0 or L == 0:
        return L
    return max(1, math.floor(L * (1.0 - rc) + 0.5))
