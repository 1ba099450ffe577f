"""LASER's host-side controller: load-aware exit threshold, EMA load, reasoning budget.

Oracle (test infrastructure).  Written from Section 4 of the paper:
  * EMA load signal (Section 4.2): L_bar(t) = alpha * L(t) + (1 - alpha) * L_bar(t-1),
    starting from L_bar = 0 (Algorithm 1, initialisation).  L(t) is the active
    request count, supplied by the caller.
  * Adaptive threshold (Eq. 5): lambda = lambda_base - beta * tanh(gamma * (L_bar - L_target) / L_target),
    clamped to [lambda_min, lambda_max] (the constraint of Eq. 4).
  * Budget pre-allocation (Eq. 6): B = max(B_min, floor(B_base * f_diff(|p|) * f_load(L))), with
    f_diff (Eq. 7) = clip(f_min + (|p| - p_min) / (p_max - p_min) * (f_max - f_min), f_min, f_max) and
    f_load (Eq. 8) = min(1, L_target / max(1, L)).
  * Decision at an ATP (Algorithm 1 loop body): update L_bar, recompute lambda, exit if
    C > lambda (strict, Section 3.1), otherwise k <- k + 1; when k reaches B the
    conclusion is forced (budget exhausted).

Defaults are the paper's (Section 5.1 for lambda/L_target/beta/gamma/alpha/B_base/
lambda_min/lambda_max/B_min; Section 4.3 for f_min/f_max/p_min/p_max).

Readings (the design doc lists them): the floor in Eq. 6 is taken of the exact
rational value of the product, with the decimal parameters read as the
decimals printed in the paper; one global L_bar is updated once per ATP
decision in call order.

Pinned by: closed forms at L_bar = L_target and in the tanh limits, the odd
symmetry of tanh about L_target, monotonicity, the fixed-threshold special
case (beta = 0, Section 4.1), exact budget values derived by hand from
Eq. 6-8, and brute force over rational arithmetic.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from fractions import Fraction
from typing import List, Sequence, Tuple

CONTINUE = 0
EARLY_EXIT = 1
BUDGET_EXHAUSTED = 2


@dataclass
class LaserParams:
    lambda_base: float = 0.95
    beta: float = 0.04
    gamma: float = 1.0
    alpha: float = 0.3
    L_target: float = 10.0
    lambda_min: float = 0.88
    lambda_max: float = 0.97
    B_base: int = 10
    B_min: int = 2
    f_min: float = 0.6
    f_max: float = 1.5
    p_min: int = 50
    p_max: int = 275


def ema_update(L_bar: float, L: float, alpha: float) -> float:
    """One EMA step of the load signal (Section 4.2)."""
    return alpha * L + (1.0 - alpha) * L_bar


def raw_threshold(L_bar: float, p: LaserParams) -> float:
    """Eq. 5 before clamping."""
    return p.lambda_base - p.beta * math.tanh(p.gamma * (L_bar - p.L_target) / p.L_target)


def adaptive_threshold(L_bar: float, p: LaserParams) -> float:
    """Eq. 5 clamped to [lambda_min, lambda_max]."""
    return min(max(raw_threshold(L_bar, p), p.lambda_min), p.lambda_max)


def _q(x) -> Fraction:
    """Exact rational value of a parameter as printed (decimal reading)."""
    return Fraction(str(x)) if isinstance(x, float) else Fraction(x)


def difficulty_factor(prompt_len: int, p: LaserParams) -> Fraction:
    """Eq. 7, exact."""
    fmin, fmax = _q(p.f_min), _q(p.f_max)
    lin = fmin + Fraction(prompt_len - p.p_min, p.p_max - p.p_min) * (fmax - fmin)
    return min(max(lin, fmin), fmax)


def load_factor(L: int, p: LaserParams) -> Fraction:
    """Eq. 8, exact."""
    return min(Fraction(1), _q(p.L_target) / max(1, L))


def allocate_budget(prompt_len: int, L: int, p: LaserParams) -> int:
    """Eq. 6: floor of the exact product, at least B_min."""
    val = p.B_base * difficulty_factor(prompt_len, p) * load_factor(L, p)
    return max(p.B_min, math.floor(val))


def exit_decision(L_bar: float, confidence: float, L: int, k_done: int, B_i: int, p: LaserParams) -> Tuple[int, float, float]:
    """Decision after the probe at ATP_{k_done+1} of a request with budget B_i.

    Returns (decision, lambda, new L_bar).  EARLY_EXIT if C > lambda; otherwise the
    failed-probe count becomes k_done + 1 and the decision is BUDGET_EXHAUSTED when it
    reaches B_i, else CONTINUE.
    """
    L_bar = ema_update(L_bar, L, p.alpha)
    lam = adaptive_threshold(L_bar, p)
    if confidence > lam:
        return EARLY_EXIT, lam, L_bar
    if k_done + 1 >= B_i:
        return BUDGET_EXHAUSTED, lam, L_bar
    return CONTINUE, lam, L_bar


def run_request(confidences: Sequence[float], loads: Sequence[int], B_i: int, p: LaserParams, L_bar: float = 0.0):
    """Algorithm 1 for one request given the confidence at each successive ATP and the load seen there.

    Returns (k, early_exited, budget_exhausted, thresholds, final L_bar): k counts failed probes.
    """
    k = 0
    lams: List[float] = []
    early = False
    i = 0
    while k < B_i and not early:
        if i >= len(confidences):
            break
        L_bar = ema_update(L_bar, loads[i], p.alpha)
        lam = adaptive_threshold(L_bar, p)
        lams.append(lam)
        if confidences[i] > lam:
            early = True
        else:
            k += 1
        i += 1
    exhausted = (k == B_i) and not early
    return k, early, exhausted, lams, L_bar
