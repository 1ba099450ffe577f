"""Pins of the serving-simulation oracle (oracle/sim.py) to queueing theory and closed forms.

Each check comes from outside the oracle: Lindley's recursion for the waiting times of a
FIFO single server, the Pollaczek-Khinchine mean wait of an M/D/1 queue, the number in
system recounted from the (arrival, finish) records, closed-form exit points of a fixed
threshold and of LASER when requests never overlap (EMA of a constant load 1:
L_bar_n = 1 - (1 - alpha)^n), and hand-computed small cases.
"""
import math

import numpy as np
import pytest

from oracle import controller as OC
from oracle import sim as S
from paper_2606_31580_amd import synth

P = OC.LaserParams()


def _reqs(tr, arrivals):
    out, c0 = [], 0
    for i, a in enumerate(arrivals):
        K = int(tr["n_chunks"][i])
        out.append(S.Request(float(a), int(tr["prompt_len"][i]), [int(x) for x in tr["chunk_tokens"][c0:c0 + K]],
                             [float(x) for x in tr["confidence"][c0:c0 + K]], [bool(x) for x in tr["correct"][c0:c0 + K]],
                             int(tr["conclusion_tokens"][i]), bool(tr["nothink_correct"][i])))
        c0 += K
    return out


COSTS = S.Costs(prefill_ms=25.0, prefill_ms_per_token=0.2, decode_ms=2.5, decode_ms_per_ctx=2e-5, probe_ms=11.0,
                probe_ms_per_ctx=3e-4)


def _series_ms(ctx, n):
    # sum_{j<n} (a + b (ctx + j)) by the arithmetic-series formula
    return n * COSTS.decode_ms + COSTS.decode_ms_per_ctx * (n * ctx + n * (n - 1) / 2)


def _vanilla_service_s(r):
    ctx = r.prompt_len
    ms = COSTS.prefill_ms + COSTS.prefill_ms_per_token * r.prompt_len
    for n in r.chunk_tokens:
        ms += _series_ms(ctx, n)
        ctx += n
    ms += _series_ms(ctx, r.conclusion_tokens)
    return ms / 1000.0


def test_decode_time_is_the_arithmetic_series():
    for ctx, n in ((0, 0), (0, 1), (100, 7), (14000, 913)):
        assert S.decode_time_ms(COSTS, ctx, n) == pytest.approx(_series_ms(ctx, n), rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("qps", [0.02, 0.1, 1.0])
def test_vanilla_waits_follow_lindley(qps):
    n = 60
    tr = synth.make_sim_traces(n, seed=11)
    reqs = _reqs(tr, synth.make_poisson_arrivals(n, qps, seed=12))
    res = S.simulate(reqs, S.VANILLA, COSTS, P)
    svc = [_vanilla_service_s(r) for r in reqs]
    w = 0.0
    for i, r in enumerate(reqs):
        if i > 0:  # Lindley: W_i = max(0, W_{i-1} + S_{i-1} - (A_i - A_{i-1}))
            w = max(0.0, w + svc[i - 1] - (r.arrival_s - reqs[i - 1].arrival_s))
        assert res[i].start_s - r.arrival_s == pytest.approx(w, rel=1e-9, abs=1e-9)
        assert res[i].finish_s - res[i].start_s == pytest.approx(svc[i], rel=1e-9)
        assert res[i].outcome == S.FINISHED and res[i].probes == 0 and res[i].chunks == len(r.chunk_tokens)
        assert res[i].correct == r.correct[-1]


def test_md1_mean_wait_matches_pollaczek_khinchine():
    # deterministic 1 s service, Poisson arrivals at rate 0.5: E[W] = rho / (2 mu (1 - rho)) = 0.5 s
    n = 40000
    arr = synth.make_poisson_arrivals(n, 0.5, seed=13)
    reqs = [S.Request(float(a), 0, [1], [0.0], [True], 0) for a in arr]
    costs = S.Costs(decode_ms=1000.0)
    res = S.simulate(reqs, S.VANILLA, costs, P)
    wait = np.mean([r.start_s - q.arrival_s for r, q in zip(res, reqs)])
    assert abs(wait - 0.5) < 0.03


def test_fixed_threshold_exit_points_closed_form():
    n = 40
    tr = synth.make_sim_traces(n, seed=21)
    reqs = _reqs(tr, synth.make_poisson_arrivals(n, 0.2, seed=22))
    for lam, cap in ((0.95, 0), (0.9, 0), (0.97, 3)):
        res = S.simulate(reqs, S.FIXED, COSTS, P, fixed_lambda=lam, max_probes=cap)
        for r, q in zip(res, reqs):
            K = len(q.chunk_tokens)
            first = next((c for c in range(K - 1) if q.confidence[c] > lam), None)
            limit = K - 1 if cap == 0 else min(cap, K - 1)
            if first is not None and first < limit:
                assert (r.outcome, r.probes, r.chunks) == (S.EXITED, first + 1, first + 1)
                assert r.correct == q.correct[first]
            elif cap and cap <= K - 1:  # Algorithm 1 stops at k = B: the last chunk is never reached
                assert (r.outcome, r.probes, r.chunks) == (S.EXHAUSTED, cap, cap)
            else:
                assert (r.outcome, r.probes, r.chunks) == (S.FINISHED, K - 1, K)


def test_laser_without_overlap_uses_load_one():
    # arrivals far apart: every request runs alone, so L = 1 at every ATP and at every start
    n = 12
    tr = synth.make_sim_traces(n, seed=31)
    arr = np.arange(n) * 1e6
    reqs = _reqs(tr, arr)
    res = S.simulate(reqs, S.LASER, COSTS, P)
    probes_so_far = 0
    for r, q in zip(res, reqs):
        B = OC.allocate_budget(q.prompt_len, 1, P)
        assert r.budget == B
        K = len(q.chunk_tokens)
        expect = None
        for c in range(min(K - 1, B)):
            m = probes_so_far + c + 1  # global probe index: L_bar_m = 1 - (1 - alpha)^m
            lam = OC.adaptive_threshold(1.0 - (1.0 - P.alpha) ** m, P)
            if q.confidence[c] > lam:
                expect = (S.EXITED, c + 1)
                break
        if expect is None:
            expect = (S.EXHAUSTED, B) if B < K - 1 else (S.FINISHED, K - 1)
        assert (r.outcome, r.probes) == expect
        probes_so_far += r.probes
        assert r.start_s == q.arrival_s


def test_load_at_each_probe_is_the_number_in_system():
    n = 80
    tr = synth.make_sim_traces(n, seed=41)
    reqs = _reqs(tr, synth.make_poisson_arrivals(n, 0.4, seed=42))
    seen = []
    orig = OC.exit_decision

    def spy(L_bar, conf, L, k, B, p):
        seen.append(L)
        return orig(L_bar, conf, L, k, B, p)

    S.C.exit_decision = spy
    try:
        res = S.simulate(reqs, S.THRESHOLD_ONLY, COSTS, P)
    finally:
        S.C.exit_decision = orig
    # recount: probe times of each request from its start, and who is in the system then
    k = 0
    for i, (r, q) in enumerate(zip(res, reqs)):
        t = r.start_s + (COSTS.prefill_ms + COSTS.prefill_ms_per_token * q.prompt_len) / 1000.0
        ctx = q.prompt_len
        for c in range(r.probes):
            t += _series_ms(ctx, q.chunk_tokens[c]) / 1000.0
            ctx += q.chunk_tokens[c]
            t += (COSTS.probe_ms + COSTS.probe_ms_per_ctx * ctx) / 1000.0
            count = sum(1 for qq, rr in zip(reqs, res) if qq.arrival_s <= t < rr.finish_s)
            assert seen[k] == count
            k += 1
    assert k == len(seen) and max(seen) > 1


def test_hand_computed_two_requests():
    # unit costs: 1 ms per token, 10 ms per probe, no prefill cost
    costs = S.Costs(decode_ms=1.0, probe_ms=10.0)
    a = S.Request(0.0, 0, [100, 200, 300], [0.5, 0.99, 0.0], [False, True, True], 50)
    b = S.Request(0.05, 0, [400], [0.0], [True], 10)
    res = S.simulate([a, b], S.FIXED, costs, P, fixed_lambda=0.95)
    # a: chunk 100, probe (0.5 fails), chunk 200, probe (0.99 exits), conclusion 50:
    # 100 + 10 + 200 + 10 + 50 ms
    assert res[0].finish_s == pytest.approx(0.37) and res[0].outcome == S.EXITED and res[0].correct
    assert res[0].probes == 2 and res[0].chunks == 2
    # b waits for a, then 400 + 10 tokens (a single chunk: no ATP, no probe)
    assert res[1].start_s == pytest.approx(0.37) and res[1].finish_s == pytest.approx(0.78)
    assert res[1].latency_s == pytest.approx(0.73) and res[1].outcome == S.FINISHED and res[1].probes == 0
    s = S.summarize([a, b], res, slo_s=0.5)
    assert s.mean_latency_s == pytest.approx((0.37 + 0.73) / 2)
    assert s.p95_latency_s == pytest.approx(0.73) and s.slo_rate == 0.5
    assert s.throughput_qps == pytest.approx(2 / 0.78) and s.accuracy == 1.0
    assert s.mean_tokens == pytest.approx((300 + 50 + 400 + 10) / 2) and s.early_exit_rate == 0.5


def test_nothinking_and_token_cap():
    costs = S.Costs(decode_ms=1.0, probe_ms=10.0, prefill_ms=5.0)
    a = S.Request(0.0, 0, [100, 200, 300], [0.0, 0.0, 0.0], [False, True, True], 50, nothink_correct=True)
    r = S.simulate([a], S.NOTHINKING, costs, P)[0]
    assert (r.outcome, r.chunks, r.probes, r.correct) == (S.SKIPPED, 0, 0, True)
    assert r.finish_s == pytest.approx(0.055)
    # the cap cuts the second chunk at 250 reasoning tokens: no probe after it
    r = S.simulate([a], S.FIXED, costs, P, fixed_lambda=0.95, max_think_tokens=250)[0]
    assert (r.outcome, r.chunks, r.probes, r.think_tokens, r.correct) == (S.CAPPED, 2, 1, 250, True)
    assert r.finish_s == pytest.approx((5 + 100 + 10 + 150 + 50) / 1000)
    # a cap that coincides with the natural end is no cut
    r = S.simulate([a], S.VANILLA, costs, P, max_think_tokens=600)[0]
    assert (r.outcome, r.think_tokens) == (S.FINISHED, 600)


def test_nearest_rank_p95():
    reqs = [S.Request(0.0, 0, [1], [0.0], [True], 0) for _ in range(20)]
    res = [S.Result(latency_s=float(i + 1), finish_s=float(i + 1)) for i in range(20)]
    assert S.summarize(reqs, res, 10.0).p95_latency_s == 19.0  # ceil(0.95 * 20) = 19th smallest
    res = res[:21] + [S.Result(latency_s=21.0, finish_s=21.0)]
    assert S.summarize(reqs + reqs[:1], res, 10.0).p95_latency_s == 20.0  # ceil(19.95) = 20


def test_laser_budget_uses_the_load_at_start_of_service():
    n = 80
    tr = synth.make_sim_traces(n, seed=51)
    reqs = _reqs(tr, synth.make_poisson_arrivals(n, 0.5, seed=52))
    res = S.simulate(reqs, S.LASER, COSTS, P)
    loads = []
    for r, q in zip(res, reqs):
        L = sum(1 for qq, rr in zip(reqs, res) if qq.arrival_s <= r.start_s < rr.finish_s)
        loads.append(L)
        assert r.budget == OC.allocate_budget(q.prompt_len, L, P)
        assert r.probes <= r.budget
    assert max(loads) > P.L_target  # the run reaches overload, where Eq. 8 shrinks budgets
