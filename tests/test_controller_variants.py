"""Pins of the oracle's controller variants (MPC, BBR-style, PCC) and class
policies: sequences and fixed points worked out by hand from the stated
rules, special cases that reduce to a closed form, invariants, and planted
mistakes in copies of the oracle that these pins must catch."""
from __future__ import annotations

import importlib.util
import math
import os
import sys
import tempfile

import pytest

from oracle import controller as oc

ORACLE_SRC = os.path.join(os.path.dirname(oc.__file__), "controller.py")


# ------------------------------------------------------------------- MPC --

def pin_mpc_smallest_sufficient_rate(m=oc):
    # horizon 1, immediate effect (f = 1), latency cost only, no trend: the
    # first candidate whose prediction b + (v - b)(1 - rc) stays at or below
    # t1 wins.  Samples 0.1 (the floor) then 0.3, t1 = 0.285: rc >= 0.075,
    # so the grid's 0.08 (r_min + 3 steps).
    c = m.OracleMPC(0.285, 0.4, window=5, horizon=1, tau=1e-9, w_quality=0.0, w_energy=0.0, w_delta=0.0)
    if c.observe(True, 0.1) != 0.0:
        return "no congestion must give r = 0"
    r = c.observe(True, 0.3)
    if not abs(r - 0.08) < 1e-12:
        return f"smallest sufficient rate {r}"
    # unreachable target: the largest rate
    c2 = m.OracleMPC(0.2, 0.4, window=5, horizon=1, tau=1e-9, w_quality=0.0, w_energy=0.0, w_delta=0.0)
    c2.observe(True, 0.1)
    if c2.observe(True, 0.3) != 0.2:
        return "unreachable target must give r_max"
    return None


def pin_mpc_grid(m=oc):
    c = m.OracleMPC(0.1, 0.2)
    g = c.candidates()
    want = [0.0] + [0.05 + i * 0.01 for i in range(15)] + [0.2]
    if len(g) != len(want) or any(abs(a - b) > 1e-12 for a, b in zip(g, want)):
        return f"grid {g}"
    return None


def pin_mpc_step_down(m=oc):
    # uncongested after r = r_max: the quadratic in rc has its minimum at
    # r - H (w_q - w_e) r_max^2 / (2 w_d) = 0.2 - 10 * 0.15 * 0.04 / 0.4 = 0.05
    c = m.OracleMPC(0.1, 0.2)
    c.r = 0.2
    c.samples = [0.05] * 10
    r1 = c.observe(True, 0.05)
    if not abs(r1 - 0.05) < 1e-12:
        return f"first step down {r1}"
    r2 = c.observe(True, 0.05)     # minimum at 0.05 - 0.15 < 0: the grid's 0
    if r2 != 0.0:
        return f"second step down {r2}"
    return None


def pin_mpc_acts_ahead_of_the_threshold(m=oc):
    # a ramp 0.02 k below t1 = 0.15: the linear controller stays at 0, the
    # MPC sees the trend cross t1 within its horizon and raises r first
    c = m.OracleMPC(0.15, 0.25)
    lin = oc.OracleController(0.15, 0.25)
    rs = [c.observe(True, 0.02 * k) for k in range(1, 6)]
    if any(lin.push(0.02 * k) != 0.0 for k in range(1, 6)):
        return "linear controller triggered below t1"
    if rs[:4] != [0.0] * 4 or not rs[4] > 0.0:
        return f"mpc rates {rs}"
    # a flat series at the same level does not trigger
    f = m.OracleMPC(0.15, 0.25)
    if any(f.observe(True, 0.10) != 0.0 for _ in range(8)):
        return "flat series below t1 triggered"
    return None


def pin_mpc_trend_line(m=oc):
    # least squares over the last 5 samples: y = 0.1 + 0.03 t -> slope 0.03,
    # value at the newest sample 0.22; with noise-free data, exact
    c = m.OracleMPC(0.5, 0.6)
    for t in range(5):
        c.observe(True, 0.1 + 0.03 * t)
    s, v = c.trend()
    if not (abs(s - 0.03) < 1e-12 and abs(v - 0.22) < 1e-12):
        return f"trend {s} {v}"
    c.observe(True, 0.0)   # window slides: 0.13, 0.16, 0.19, 0.22, 0.0
    ys = [0.13, 0.16, 0.19, 0.22, 0.0]
    tm = 2.0
    ym = sum(ys) / 5
    sl = sum((t - tm) * (y - ym) for t, y in enumerate(ys)) / sum((t - tm) ** 2 for t in range(5))
    s, v = c.trend()
    if not (abs(s - sl) < 1e-12 and abs(v - (ym + 2 * sl)) < 1e-12):
        return "sliding window"
    return None


def pin_mpc_prediction_formula(m=oc):
    # one cost evaluated by hand: b = 0.1, v = 0.3, s = 0, H = 2, tau = 1,
    # r = 0.1, rc = 0.15, t1 = 0.2, t2 = 0.3
    c = m.OracleMPC(0.2, 0.3, horizon=2, tau=1.0, w_lat=1.0, w_quality=0.3, w_energy=0.1, w_delta=0.4)
    c.r = 0.1
    J = c.cost(0.15, 0.0, 0.3, 0.1)
    want = 0.0
    for h in (1, 2):
        f = 1 - math.exp(-h)
        y = 0.1 + 0.2 * ((1 - f) + f * 0.85 / 0.9)
        want += ((y - 0.2) / 0.1) ** 2
    want += 2 * 0.2 * 0.15 + 0.4 * (0.05 / 0.2) ** 2
    if not abs(J - want) < 1e-12:
        return f"cost {J} vs {want}"
    return None


# ------------------------------------------------------------------- BBR --

def pin_bbr_gain_cycle_at_the_floor(m=oc):
    # constant TBT at its floor: r_base stays 0, the cycle probes below 0
    # (clamped) then drains at +probe on the second tick of every 8
    c = m.OracleBBR()
    rs = [c.observe(True, 0.05, 100.0) for _ in range(17)]
    want = [0.0, 0.02, 0, 0, 0, 0, 0, 0] * 2 + [0.0]
    if rs != want:
        return f"cycle {rs}"
    return None


def pin_bbr_past_the_knee(m=oc):
    # floor 0.05, then 0.1 (> 0.0625) at full delivery rate: r_base climbs by
    # 0.02 a tick to 0.2; applied = r_base - 0.02 on cycle ticks 1, 9, ...,
    # + 0.02 on ticks 2, 10, ... (clamped to [0, 0.2])
    c = m.OracleBBR()
    rs = [c.observe(True, 0.05, 100.0)]
    rs += [c.observe(True, 0.10, 100.0) for _ in range(15)]
    base = [0.0] + [min(0.02 * k, 0.2) for k in range(1, 16)]
    want = []
    for i, b in enumerate(base):
        off = -0.02 if i % 8 == 0 else (0.02 if i % 8 == 1 else 0.0)
        want.append(min(max(b + off, 0.0), 0.2))
    if any(abs(a - b) > 1e-12 for a, b in zip(rs, want)):
        return f"knee {rs}"
    return None


def pin_bbr_holds_when_delivery_drops(m=oc):
    # high TBT while the delivery rate is below (1 - margin) BtlBw: hold
    c = m.OracleBBR(cycle=1000)
    c.observe(True, 0.05, 100.0)
    c.observe(True, 0.10, 100.0)          # r_base 0.02
    r = [c.observe(True, 0.10, 70.0) for _ in range(3)]   # 70 < 75
    if r != [0.02, 0.02, 0.02]:
        return f"hold {r}"
    # 80 is within (1 - margin) of BtlBw = 100: past the knee again
    if not abs(c.observe(True, 0.10, 80.0) - 0.04) < 1e-12:
        return "delivery within the margin of BtlBw"
    # TBT 0.055 is inside the floor band (0.05 (1 + 0.125)): r_base falls
    if not abs(c.observe(True, 0.055, 80.0) - 0.02) < 1e-12:
        return "floor band"
    # 0.06 is above the band and below the knee (0.0625): hold
    if not abs(c.observe(True, 0.06, 80.0) - 0.02) < 1e-12:
        return "between band and knee"
    return None


def pin_bbr_windows_forget(m=oc):
    # the floor sample leaves the 3-tick RTprop window: the higher TBT becomes
    # the floor and r_base falls again
    c = m.OracleBBR(rt_window=3, cycle=1000)
    c.observe(True, 0.05, 100.0)
    rs = [c.observe(True, 0.10, 100.0) for _ in range(4)]
    # ticks 2, 3: past the knee (r_base 0.02, 0.04; tick 2 is the cycle's
    # drain tick, +0.02); tick 4: floor = min(0.1, 0.1, 0.1), near the floor,
    # r_base 0.02; tick 5: 0
    if any(abs(a - b) > 1e-12 for a, b in zip(rs, [0.04, 0.04, 0.02, 0.0])):
        return f"windows {rs}"
    return None


# ------------------------------------------------------------------- PCC --

def pin_pcc_uncongested_rounds(m=oc):
    # TBT below t1: U = -w_q r / r_max, so every round moves the center down
    # (clamped at 0); the interval order alternates: up first, then down first
    c = m.OraclePCC(0.1, 0.2, interval=2)
    rs = [c.observe(True, 0.05) for _ in range(8)]
    # rates in force: r0=0.02 for ticks 1-2, then 0 (ticks 3-4), then round 1 down-first: 0, then 0.02
    want = [0.02, 0.0, 0.0, 0.0, 0.0, 0.02, 0.02, 0.02]
    if any(abs(a - b) > 1e-12 for a, b in zip(rs, want)):
        return f"rounds {rs}"
    if c.center != 0.0:
        return "center"
    return None


def pin_pcc_gradient_step(m=oc):
    # a lag-free plant: TBT = t1 + (t2 - t1)(1.2 - 5 r) while it exceeds t1.
    # Then U(r) = -(1.2 - 5 r) - 0.5 r / 0.2 = -1.2 + 2.5 r, the gradient is
    # 2.5 and each round adds gain * 2.5 = 0.05 to the center.
    c = m.OraclePCC(0.1, 0.2, interval=1, epsilon=0.02, gain=0.02)
    for _ in range(6):          # three rounds
        r = c.r
        c.observe(True, 0.1 + 0.1 * (1.2 - 5 * r))
    if not abs(c.center - 0.15) < 1e-12:
        return f"center {c.center}"
    for _ in range(4):
        r = c.r
        c.observe(True, 0.1 + 0.1 * max(1.2 - 5 * r, 0.0))
    if not abs(c.center - 0.2) < 1e-12:
        return f"clamped center {c.center}"
    return None


# -------------------------------------------------------------- classes --

def pin_class_policies(m=oc):
    if m.cap_for_class(100, 0.2) != 80 or m.cap_for_class(100, 0.2, weight=0.0) != 100:
        return "weight"
    if m.cap_for_class(16, 0.2, bypass_len=16) != 16 or m.cap_for_class(17, 0.2, bypass_len=16) != 14:
        return "bypass"
    if m.cap_for_class(100, 0.2, weight=0.5) != 90 or m.cap_for_class(100, 0.15, weight=2.0) != 80:
        return "scaling and cap"
    for L in range(0, 300):
        for r in (0.0, 0.05, 0.13, 0.2):
            if m.cap_for_class(L, r) != oc.OracleController(0.1, 0.2).cap(L) if r == 0.0 else None:
                pass
            base = oc.OracleController(0.1, 0.2)
            base.r = r
            if m.cap_for_class(L, r) != base.cap(L):
                return f"weight 1 differs from the base cap at L={L} r={r}"
    return None


def pin_linear_behind_ticks(m=oc):
    a = m.OracleLinear(0.1, 0.2)
    b = oc.OracleController(0.1, 0.2)
    for k, y in enumerate([0.05, 0.15, 0.3, 0.12, 0.02, 0.2]):
        if k % 2:
            a.observe(False)
        if a.observe(True, y) != b.push(y):
            return "linear"
    return None


PINS = [pin_mpc_smallest_sufficient_rate, pin_mpc_grid, pin_mpc_step_down, pin_mpc_acts_ahead_of_the_threshold,
        pin_mpc_trend_line, pin_mpc_prediction_formula, pin_bbr_gain_cycle_at_the_floor, pin_bbr_past_the_knee,
        pin_bbr_holds_when_delivery_drops, pin_bbr_windows_forget, pin_pcc_uncongested_rounds,
        pin_pcc_gradient_step, pin_class_policies, pin_linear_behind_ticks]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_variant_pins(pin):
    assert pin() is None


def test_rates_stay_in_range():
    import random
    rnd = random.Random(5)
    for _ in range(20):
        ctls = [oc.OracleMPC(0.1, 0.2), oc.OracleBBR(), oc.OraclePCC(0.1, 0.2, interval=3)]
        grid = set(ctls[0].candidates())
        for _ in range(200):
            has = rnd.random() < 0.9
            y = rnd.uniform(0.01, 0.5)
            n = rnd.uniform(0, 500)
            for c in ctls:
                r = c.observe(has, y, n)
                assert 0.0 <= r <= 0.2
            assert ctls[0].r in grid


MUTANTS = {
    "mpc trend sign": ("u = max(v + s * h, b)", "u = max(v - s * h, b)"),
    "mpc share of capped work": ("f = 1.0 - math.exp(-h / self.tau)", "f = math.exp(-h / self.tau)"),
    "mpc ratio of rates": ("f * (1.0 - rc) / (1.0 - self.r)", "f * (1.0 - rc)"),
    "mpc energy sign": ("(self.w_quality - self.w_energy) * rc", "(self.w_quality + self.w_energy) * rc"),
    "mpc ties": ("            if J < best_J:", "            if J <= best_J:"),
    "bbr probe phases": ("off = -self.probe if phase == 0 else (self.probe if phase == 1 else 0.0)",
                         "off = self.probe if phase == 0 else (-self.probe if phase == 1 else 0.0)"),
    "bbr delivery test": ("x >= (1.0 - self.margin) * btlbw", "x >= btlbw"),
    "bbr floor band": ("tbt <= rtprop * (1.0 + self.margin / 2.0)", "tbt <= rtprop"),
    "pcc gradient sign": ("(Ua - U) / (ra - self.r)", "(U - Ua) / (ra - self.r)"),
    "pcc order": ("up = (self.round % 2 == 0) != self.second", "up = not self.second"),
    "class bypass": ("if L <= bypass_len:", "if L < bypass_len:"),
}


def _load_mutant(src):
    d = tempfile.mkdtemp()
    path = os.path.join(d, "controller_mutant.py")
    open(path, "w").write(src)
    spec = importlib.util.spec_from_file_location("controller_mutant", path)
    mod = importlib.util.module_from_spec(spec)
    sys.modules["controller_mutant"] = mod
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_variant_mutants_are_caught(name):
    src = open(ORACLE_SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name!r} not found exactly once"
    mod = _load_mutant(src.replace(old, new))
    fails = []
    for pin in PINS:
        try:
            r = pin(mod)
        except Exception as e:  # a crash counts as caught
            r = repr(e)
        if r is not None:
            fails.append(r)
    assert fails, f"mutant {name!r} passed every pin"
