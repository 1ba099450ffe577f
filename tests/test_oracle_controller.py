"""Pins for the oracle's controller (Eq. 5-8, Section 4.2 EMA, Algorithm 1 decision)."""
import json
import math
import os

import pytest

from oracle import controller as C

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_threshold_golden_values():
    p = C.LaserParams()
    for case in load("threshold_eq5_defaults.json")["cases"]:
        assert C.raw_threshold(case["L_bar"], p) == pytest.approx(case["raw"], abs=1e-12)
        assert C.adaptive_threshold(case["L_bar"], p) == pytest.approx(case["lambda"], abs=1e-12)


def test_threshold_at_target_is_exactly_base():
    # tanh(0) = 0: at L_bar == L_target the threshold is lambda_base for any beta, gamma
    for beta in (0.0, 0.04, 0.3):
        for gamma in (0.5, 1.0, 3.0):
            p = C.LaserParams(beta=beta, gamma=gamma, lambda_min=0.0, lambda_max=1.0)
            assert C.adaptive_threshold(p.L_target, p) == 0.95


def test_threshold_odd_symmetry_about_target():
    # tanh is odd, so unclamped thresholds at L_target +/- x average to lambda_base
    p = C.LaserParams(lambda_min=0.0, lambda_max=1.0)
    for x in (0.5, 1.0, 3.7, 9.9, 25.0):
        hi = C.adaptive_threshold(p.L_target + x, p)
        lo = C.adaptive_threshold(p.L_target - x, p)
        assert hi < 0.95 < lo  # more load lowers the bar
        assert (hi + lo) / 2 == pytest.approx(0.95, abs=1e-15)


def test_threshold_monotone_and_bounded():
    p = C.LaserParams()
    prev = None
    for i in range(0, 2001):
        lam = C.adaptive_threshold(i * 0.05, p)
        assert p.lambda_min <= lam <= p.lambda_max
        if prev is not None:
            assert lam <= prev
        prev = lam


def test_threshold_clamp_min_reachable_with_large_beta():
    # at the defaults raw >= 0.91 so lambda_min=0.88 never binds; with beta=0.1 it does
    p = C.LaserParams(beta=0.1)
    assert C.raw_threshold(1e9, p) == pytest.approx(0.85)
    assert C.adaptive_threshold(1e9, p) == 0.88
    assert C.adaptive_threshold(0.0, p) == 0.97


def test_fixed_threshold_special_case():
    # Section 4.1: with both mechanisms disabled LASER is fixed-threshold early exit
    p = C.LaserParams(beta=0.0, f_min=1.0, f_max=1.0, L_target=1e9)
    for L_bar in (0.0, 3.0, 1e6):
        assert C.adaptive_threshold(L_bar, p) == 0.95
    for plen in (1, 50, 300, 5000):
        for L in (0, 1, 50, 10**6):
            assert C.allocate_budget(plen, L, p) == p.B_base


def test_ema_closed_form():
    g = load("ema_constant_load.json")
    L_bar = 0.0
    for n, expect in enumerate(g["sequence"], start=1):
        L_bar = C.ema_update(L_bar, g["L"], g["alpha"])
        assert L_bar == pytest.approx(expect, abs=1e-12)
        assert L_bar == pytest.approx(g["L"] * (1 - (1 - g["alpha"]) ** n), abs=1e-12)


def test_budget_golden_values():
    p = C.LaserParams()
    for case in load("budget_eq6_defaults.json")["cases"]:
        assert C.allocate_budget(case["prompt_len"], case["L"], p) == case["B"], case


def _budget_integer(plen, L):
    # independent integer-only evaluation of Eq. 6-8 at the defaults:
    # f_diff = (60*225 + (plen-50)*90) / (100*225) clipped to [60/100, 150/100]
    # f_load = min(1, 10 / max(1, L))
    num_diff = 60 * 225 + (plen - 50) * 90
    num_diff = min(max(num_diff, 60 * 225), 150 * 225)
    den_diff = 100 * 225
    Lm = max(1, L)
    if Lm <= 10:
        num, den = 10 * num_diff, den_diff
    else:
        num, den = 10 * num_diff * 10, den_diff * Lm
    return max(2, num // den)


def test_budget_brute_force_integer_arithmetic():
    p = C.LaserParams()
    for plen in range(0, 400):
        for L in range(0, 60):
            assert C.allocate_budget(plen, L, p) == _budget_integer(plen, L), (plen, L)


def test_budget_monotonicity():
    p = C.LaserParams()
    for plen in range(0, 400, 7):
        prev = None
        for L in range(0, 80):
            b = C.allocate_budget(plen, L, p)
            assert p.B_min <= b <= 15
            if prev is not None:
                assert b <= prev  # more load -> smaller or equal budget
            prev = b
    for L in (1, 12, 40):
        prev = None
        for plen in range(0, 400):
            b = C.allocate_budget(plen, L, p)
            if prev is not None:
                assert b >= prev  # longer prompt (harder) -> larger or equal budget
            prev = b


def test_exit_decision_strict_and_monotone():
    p = C.LaserParams()
    lam = C.adaptive_threshold(C.ema_update(0.0, 4, p.alpha), p)
    d, lam_out, _ = C.exit_decision(0.0, lam, 4, 0, 10, p)
    assert lam_out == lam and d == C.CONTINUE  # C == lambda continues (strict >)
    d, _, _ = C.exit_decision(0.0, math.nextafter(lam, 2.0), 4, 0, 10, p)
    assert d == C.EARLY_EXIT
    # monotone in the threshold: a request exits at threshold lam iff it exits at every lower threshold
    for conf in (0.5, 0.9, 0.93, 0.95, 0.96, 0.99):
        prev_exit = False
        for beta in (0.0, 0.02, 0.04, 0.08, 0.16):  # larger beta at high load -> lower lambda
            q = C.LaserParams(beta=beta, lambda_min=0.0)
            d, _, _ = C.exit_decision(50.0, conf, 50, 0, 10, q)
            ex = d == C.EARLY_EXIT
            assert ex or not prev_exit
            prev_exit = ex


def test_exit_decision_budget():
    p = C.LaserParams()
    assert C.exit_decision(0.0, 0.1, 1, 0, 2, p)[0] == C.CONTINUE
    assert C.exit_decision(0.0, 0.1, 1, 1, 2, p)[0] == C.BUDGET_EXHAUSTED
    assert C.exit_decision(0.0, 0.999, 1, 1, 2, p)[0] == C.EARLY_EXIT  # exit wins over exhaustion


def test_algorithm1_loop():
    p = C.LaserParams()
    # never confident: runs exactly B probes then forces the conclusion
    k, early, exhausted, lams, _ = C.run_request([0.1] * 20, [1] * 20, 5, p)
    assert (k, early, exhausted, len(lams)) == (5, False, True, 5)
    # confident at the third ATP
    k, early, exhausted, lams, _ = C.run_request([0.1, 0.2, 0.999, 0.1], [1] * 4, 5, p)
    assert (k, early, exhausted, len(lams)) == (2, True, False, 3)
    # under heavy load the threshold drops below a confidence that fails at light load
    conf = 0.93
    k_l, early_l, *_ = C.run_request([conf] * 10, [1] * 10, 10, p)
    k_h, early_h, *_ = C.run_request([conf] * 10, [40] * 10, 10, p)
    assert not early_l and early_h and k_h < k_l
