"""Pins of the controller oracle: the paper's stated points (golden fixture)
and numpy's percentile routine for the threshold calibration."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

from oracle.controller import OracleController, calibrate_thresholds, percentile_linear

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "controller_paper_rules.json")


def _cases():
    return json.load(open(GOLDEN))


@pytest.mark.parametrize("case", _cases()["cases"], ids=lambda c: c["name"])
def test_paper_rules(case):
    g = _cases()
    c = OracleController(g["t1"], g["t2"], window=g["window"])
    for v in case["tbt"]:
        r = c.push(v)
    assert abs(r - case["r"]) <= case.get("r_tol", 1e-12)
    assert c.cap(case["L"]) == case["N"]


def test_percentile_matches_numpy():
    rng = np.random.default_rng(0)
    for n in (1, 2, 3, 10, 101, 1000):
        xs = rng.lognormal(size=n)
        for p in (0, 25, 50, 75, 90, 100):
            assert abs(percentile_linear(xs, p) - np.percentile(xs, p)) <= 1e-12 * max(1.0, abs(np.percentile(xs, p)))


def test_calibration_is_median_and_p75():
    xs = [5.0, 1.0, 4.0, 2.0, 3.0]
    assert calibrate_thresholds(xs) == (3.0, 4.0)


def test_cap_rounding_and_minimum():
    c = OracleController(1.0, 2.0)
    c.push(2.0)                      # r = 20%
    assert c.cap(1) == 1             # 0.8 rounds to 1
    assert c.cap(3) == 2             # 2.4 -> 2
    assert c.cap(0) == 0
    with pytest.raises(ValueError):
        c.cap(-1)
