"""The native serving simulation (laser_simulate) against the oracle, request by request.

Runs on the CPU.  Integer results (outcome, chunks, probes, reasoning tokens, budget,
correctness) must be equal; times agree to 1e-9 relative (the two sum the same costs in a
different order); the summaries agree likewise.  Every method, several loads (including
overload, where Eq. 8 shrinks budgets and Eq. 5 lowers the threshold), the probe cap, the
reasoning-token cap and the phased (burst) arrival pattern are covered.
"""
import math

import numpy as np
import pytest

from oracle import controller as OC
from oracle import sim as S
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth

COSTS = dict(prefill_ms=25.0, prefill_ms_per_token=0.2, decode_ms=2.5, decode_ms_per_ctx=2e-5, probe_ms=11.0,
             probe_ms_per_ctx=3e-4)


def _oracle_reqs(tr, arrivals):
    out, c0 = [], 0
    for i, a in enumerate(arrivals):
        K = int(tr["n_chunks"][i])
        out.append(S.Request(float(a), int(tr["prompt_len"][i]), [int(x) for x in tr["chunk_tokens"][c0:c0 + K]],
                             [float(x) for x in tr["confidence"][c0:c0 + K]], [bool(x) for x in tr["correct"][c0:c0 + K]],
                             int(tr["conclusion_tokens"][i]), bool(tr["nothink_correct"][i])))
        c0 += K
    return out


def _compare(arrivals, tr, method, fixed_lambda=0.95, max_probes=0, max_think=0, slo=30.0):
    p = L.laser_params_default()
    cfg = L.sim_config(method, COSTS, fixed_lambda=fixed_lambda, max_probes=max_probes, max_think_tokens=max_think,
                       slo_s=slo)
    got, gs = L.laser_simulate(p, cfg, arrivals, tr)
    reqs = _oracle_reqs(tr, arrivals)
    ref = S.simulate(reqs, method, S.Costs(**COSTS), OC.LaserParams(), fixed_lambda=fixed_lambda,
                     max_probes=max_probes, max_think_tokens=max_think)
    for i, (g, r) in enumerate(zip(got, ref)):
        tag = f"method {method} request {i}"
        assert (g.outcome, g.chunks, g.probes, g.think_tokens, g.budget, bool(g.correct)) == \
            (r.outcome, r.chunks, r.probes, r.think_tokens, r.budget, r.correct), tag
        for f in ("start_s", "finish_s", "latency_s"):
            assert getattr(g, f) == pytest.approx(getattr(r, f), rel=1e-9, abs=1e-9), (tag, f)
        if r.probes:
            assert g.lambda_last == pytest.approx(r.lambda_last, rel=1e-12), tag
        else:
            assert math.isnan(g.lambda_last), tag
    rs = S.summarize(reqs, ref, slo)
    assert gs.n == rs.n
    for f in ("mean_latency_s", "p95_latency_s", "throughput_qps", "slo_rate", "accuracy", "mean_tokens",
              "early_exit_rate"):
        assert getattr(gs, f) == pytest.approx(getattr(rs, f), rel=1e-9, abs=1e-12), f
    return got, gs


@pytest.mark.parametrize("method", range(6))
@pytest.mark.parametrize("qps", [0.01, 0.08, 0.5])
def test_native_matches_oracle(method, qps):
    n = 70
    tr = synth.make_sim_traces(n, seed=100 + int(qps * 100))
    arr = synth.make_poisson_arrivals(n, qps, seed=200 + method)
    _compare(arr, tr, method)


@pytest.mark.parametrize("method", [L.SIM_VANILLA, L.SIM_FIXED, L.SIM_THRESHOLD_ONLY, L.SIM_LASER])
def test_caps_match_oracle(method):
    n = 50
    tr = synth.make_sim_traces(n, seed=300)
    arr = synth.make_poisson_arrivals(n, 0.1, seed=301)
    got, _ = _compare(arr, tr, method, fixed_lambda=0.97, max_probes=3, max_think=5000)
    outcomes = {g.outcome for g in got}
    assert L.SIM_CAPPED in outcomes  # the token cap is exercised
    if method in (L.SIM_FIXED, L.SIM_THRESHOLD_ONLY):
        assert L.SIM_EXHAUSTED in outcomes  # the probe cap is exercised


def test_burst_pattern_matches_oracle():
    arr = synth.make_phased_arrivals([0.02, 0.1, 0.02], [1500.0, 1500.0, 1500.0], seed=400)
    tr = synth.make_sim_traces(len(arr), seed=401)
    got, gs = _compare(arr, tr, L.SIM_LASER)
    assert max(g.budget for g in got) > min(g.budget for g in got)


def test_laser_lowers_latency_under_load():
    # the structure of the paper's comparison: in overload (the queue grows past L_target)
    # LASER finishes requests sooner than the fixed threshold and far sooner than no early
    # exit.  (Under light load Eq. 5 raises the threshold to lambda_max instead.)
    n = 125
    tr = synth.make_sim_traces(n, seed=500)
    arr = synth.make_poisson_arrivals(n, 0.5, seed=501)
    p = L.laser_params_default()
    out = {}
    for m in (L.SIM_VANILLA, L.SIM_FIXED, L.SIM_LASER):
        out[m] = L.laser_simulate(p, L.sim_config(m, COSTS), arr, tr)[1]
    assert out[L.SIM_LASER].mean_latency_s < out[L.SIM_FIXED].mean_latency_s < out[L.SIM_VANILLA].mean_latency_s


def test_errors_leave_nothing_half_done():
    p = L.laser_params_default()
    tr = synth.make_sim_traces(3, seed=600)
    cfg = L.sim_config(L.SIM_LASER, COSTS)
    with pytest.raises(L.LaserError):
        L.laser_simulate(p, cfg, [1.0, 0.5, 2.0], tr)  # decreasing arrivals
    bad = dict(tr)
    bad["confidence"] = tr["confidence"].copy()
    bad["confidence"][0] = np.nan
    with pytest.raises(L.LaserError):
        L.laser_simulate(p, cfg, [0.0, 1.0, 2.0], bad)
    bad = dict(tr)
    bad["n_chunks"] = tr["n_chunks"].copy()
    bad["n_chunks"][1] = 0
    with pytest.raises(L.LaserError):
        L.laser_simulate(p, cfg, [0.0, 1.0, 2.0], bad)
    with pytest.raises(L.LaserError):
        L.laser_simulate(p, L.sim_config(9, COSTS), [0.0, 1.0, 2.0], tr)
    with pytest.raises(L.LaserError):
        L.laser_simulate(p, L.sim_config(L.SIM_FIXED, dict(COSTS, decode_ms=-1.0)), [0.0, 1.0, 2.0], tr)
    res, s = L.laser_simulate(p, cfg, [], {k: v[:0] for k, v in tr.items()})
    assert res == [] and s.n == 0
