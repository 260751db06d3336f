"""The library's C++ controller against the controller oracle: identical rates
and caps on seeded TBT series (both binary64, same formula order), and the
threshold calibration against the oracle's percentiles."""
from __future__ import annotations

import numpy as np
import pytest

from oracle.controller import OracleController, calibrate_thresholds as oracle_calibrate


@pytest.fixture(scope="module")
def P():
    import paper_2510_15330_amd as p
    return p


@pytest.mark.parametrize("seed", range(6))
def test_matches_oracle_on_random_series(P, seed):
    rng = np.random.default_rng(seed)
    t1 = float(rng.uniform(0.02, 0.05))
    t2 = t1 + float(rng.uniform(0.0, 0.05)) if seed != 5 else t1 - 0.01
    window = int(rng.integers(1, 8))
    lib_c = P.Controller(t1, t2, window=window)
    ora = OracleController(t1, t2, window=window)
    # a ramp up into congestion, a plateau and a recovery, with noise
    base = np.concatenate([np.linspace(0.5 * t1, 2.0 * max(t1, t2), 120), np.full(60, 1.5 * t1),
                           np.linspace(1.5 * t1, 0.3 * t1, 60)])
    tbt = base * rng.lognormal(0.0, 0.1, size=base.size)
    lengths = rng.integers(0, 3000, size=base.size)
    for v, L in zip(tbt, lengths):
        n_lib = lib_c.length_cap(int(L), float(v))
        r_or = ora.push(float(v))
        assert lib_c.rate == r_or
        assert n_lib == ora.cap(int(L))
        # a request between two samples uses the current rate
        assert lib_c.length_cap(int(L) + 7) == ora.cap(int(L) + 7)


def test_calibration_matches_oracle(P):
    rng = np.random.default_rng(9)
    for n in (1, 2, 5, 64, 1321):
        xs = rng.lognormal(-3.0, 0.4, size=n)
        assert P.calibrate_thresholds(xs) == oracle_calibrate(xs)


def test_paper_golden_through_library(P):
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "controller_paper_rules.json")))
    for case in g["cases"]:
        c = P.Controller(g["t1"], g["t2"], window=g["window"])
        for v in case["tbt"]:
            c.length_cap(0, v)
        assert abs(c.rate - case["r"]) <= case.get("r_tol", 1e-12), case["name"]
        assert c.length_cap(case["L"]) == case["N"], case["name"]
