"""Serving simulation of the paper's evaluation (Section 5.1), as a plain event-driven program.

Oracle (test infrastructure).  Written from the paper:
  * Latency of request i (Eq. 1): l_i = w_i + t_inf_i, queueing delay plus inference time.
  * Inference time (Eq. 2): prefill + the reasoning chunks generated, each with the probe
    (trial answer and confidence) at the ATP that follows it, + the conclusion.
  * Requests arrive (Poisson, or a three-phase rate pattern) and one server takes them
    first come, first served (Section 5.1).
  * LASER (Algorithm 1): the budget B_i is set when the request starts (Eq. 6-8, load at
    that moment); at every ATP the EMA load and the Eq. 5 threshold are updated and the
    request exits if C > lambda, otherwise counts a failed probe and stops at B_i.
  * Baselines (Section 5.1) and ablation variants (Section 5.4): Vanilla (no early exit),
    Fixed (a fixed threshold), NoThinking (no reasoning chunks), LASER, threshold only,
    budget only.

Readings (the design doc lists them): L(t) is the number of requests in the system (waiting or
in service) at time t, arrivals at exactly t included; the EMA runs over every probe in
time order from L_bar = 0; an ATP follows every chunk but the last; probe tokens do not
stay in the context; a request that stops after chunk c is scored with that chunk's
correctness flag; a cap on reasoning tokens cuts the chunk in progress and forces the
conclusion; P95 is the nearest-rank percentile; throughput is n over the span from the
first arrival to the last completion.

Cost model: decoding one token at context c costs decode_ms + decode_ms_per_ctx * c; a
probe at context c costs probe_ms + probe_ms_per_ctx * c; a prefill of p tokens costs
prefill_ms + prefill_ms_per_token * p (milliseconds).

Structure: an event heap (arrivals before service events at equal times), an explicit
waiting queue, and a server that runs each request as a list of timed steps.  Pinned in
tests/test_oracle_sim.py by Lindley's recursion, the sample-path form of Little's law,
the Pollaczek-Khinchine mean wait of an M/D/1 queue, closed-form exit points of the fixed
threshold, and hand-computed small cases.
"""
from __future__ import annotations

import heapq
import math
from collections import deque
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

from . import controller as C

VANILLA, FIXED, LASER, THRESHOLD_ONLY, BUDGET_ONLY, NOTHINKING = range(6)
FINISHED, EXITED, EXHAUSTED, CAPPED, SKIPPED = range(5)


@dataclass
class Costs:
    prefill_ms: float = 0.0
    prefill_ms_per_token: float = 0.0
    decode_ms: float = 0.0
    decode_ms_per_ctx: float = 0.0
    probe_ms: float = 0.0
    probe_ms_per_ctx: float = 0.0


@dataclass
class Request:
    arrival_s: float
    prompt_len: int
    chunk_tokens: List[int]
    confidence: List[float]  # at the ATP after each chunk (the last entry is not used)
    correct: List[bool]      # answer after each chunk is right
    conclusion_tokens: int
    nothink_correct: bool = False


@dataclass
class Result:
    start_s: float = 0.0
    finish_s: float = 0.0
    latency_s: float = 0.0
    budget: int = 0
    chunks: int = 0
    probes: int = 0
    think_tokens: int = 0
    outcome: int = FINISHED
    correct: bool = False
    lambda_last: float = math.nan


def decode_time_ms(costs: Costs, ctx: int, n: int) -> float:
    """n tokens generated one by one from context ctx."""
    total = 0.0
    for j in range(n):
        total += costs.decode_ms + costs.decode_ms_per_ctx * (ctx + j)
    return total


def simulate(reqs: Sequence[Request], method: int, costs: Costs, p: C.LaserParams, fixed_lambda: float = 0.95,
             max_probes: int = 0, max_think_tokens: int = 0) -> List[Result]:
    n = len(reqs)
    res = [Result() for _ in range(n)]
    events = []  # (time, kind, order, request): kind 0 = arrival, 1 = end of a service step
    order = 0
    for i, r in enumerate(reqs):
        heapq.heappush(events, (r.arrival_s, 0, order, i))
        order += 1
    waiting: deque = deque()
    serving: Optional[int] = None
    L_bar = 0.0
    # state of the request in service
    st = {}

    def in_system() -> int:
        return len(waiting) + (1 if serving is not None else 0)

    def schedule(t: float, i: int):
        nonlocal order
        heapq.heappush(events, (t, 1, order, i))
        order += 1

    def start(i: int, t: float):
        nonlocal serving
        serving = i
        r = reqs[i]
        res[i].start_s = t
        budget = None
        if method in (LASER, BUDGET_ONLY):
            budget = C.allocate_budget(r.prompt_len, in_system(), p)
            res[i].budget = budget
        elif max_probes > 0:
            budget = max_probes
        st.clear()
        st.update(i=i, budget=budget, k=0, ctx=r.prompt_len, phase="prefill", answer=None)
        schedule(t + (costs.prefill_ms + costs.prefill_ms_per_token * r.prompt_len) / 1000.0, i)

    def next_step(t: float):
        """The step that just ended decides what runs next; returns the next end time or None when done."""
        nonlocal L_bar
        i = st["i"]
        r = reqs[i]
        R = res[i]
        phase = st["phase"]
        if phase == "prefill":
            if method == NOTHINKING:
                R.outcome = SKIPPED
                return conclude(t)
            return run_chunk(t, 0)
        if phase == "chunk":
            k = st["chunk"]
            if st["cut"]:
                R.outcome = CAPPED
                return conclude(t)
            if k == len(r.chunk_tokens) - 1:
                R.outcome = FINISHED
                return conclude(t)
            if method == VANILLA:
                return run_chunk(t, k + 1)
            st["phase"] = "probe"
            return t + (costs.probe_ms + costs.probe_ms_per_ctx * st["ctx"]) / 1000.0
        if phase == "probe":
            k = st["chunk"]
            R.probes += 1
            L = in_system()
            conf = r.confidence[k]
            budget = st["budget"]
            if method in (LASER, THRESHOLD_ONLY):
                dec, lam, L_bar = C.exit_decision(L_bar, conf, L, R.probes - 1, budget if budget else 1 << 62, p)
            else:
                L_bar = C.ema_update(L_bar, L, p.alpha)
                lam = fixed_lambda
                if conf > lam:
                    dec = C.EARLY_EXIT
                elif budget and R.probes >= budget:
                    dec = C.BUDGET_EXHAUSTED
                else:
                    dec = C.CONTINUE
            R.lambda_last = lam
            if dec == C.EARLY_EXIT:
                R.outcome = EXITED
                return conclude(t)
            if dec == C.BUDGET_EXHAUSTED:
                R.outcome = EXHAUSTED
                return conclude(t)
            return run_chunk(t, k + 1)
        if phase == "conclusion":
            return None
        raise AssertionError(phase)

    def run_chunk(t: float, k: int) -> float:
        r = reqs[st["i"]]
        R = res[st["i"]]
        ntok = r.chunk_tokens[k]
        cut = False
        if max_think_tokens > 0 and R.think_tokens + ntok >= max_think_tokens:
            cut = R.think_tokens + ntok > max_think_tokens or k < len(r.chunk_tokens) - 1
            ntok = max_think_tokens - R.think_tokens
        end = t + decode_time_ms(costs, st["ctx"], ntok) / 1000.0
        st["ctx"] += ntok
        R.think_tokens += ntok
        R.chunks += 1
        st.update(phase="chunk", chunk=k, cut=cut, answer=k)
        return end

    def conclude(t: float) -> float:
        r = reqs[st["i"]]
        R = res[st["i"]]
        R.correct = bool(r.nothink_correct) if st["answer"] is None else bool(r.correct[st["answer"]])
        st["phase"] = "conclusion"
        return t + decode_time_ms(costs, st["ctx"], r.conclusion_tokens) / 1000.0

    start_pending = False
    while events:
        t, kind, _, i = heapq.heappop(events)
        if kind == 0:
            waiting.append(i)
            if serving is None and not start_pending:  # start after every arrival at t is queued
                schedule(t, -1)
                start_pending = True
            continue
        if i == -1:
            start_pending = False
            start(waiting.popleft(), t)
            continue
        nxt = next_step(t)
        if nxt is not None:
            schedule(nxt, i)
            continue
        res[i].finish_s = t
        res[i].latency_s = t - reqs[i].arrival_s
        serving = None
        if waiting:
            start(waiting.popleft(), t)
    return res


@dataclass
class Summary:
    n: int
    mean_latency_s: float
    p95_latency_s: float
    throughput_qps: float
    slo_rate: float
    accuracy: float
    mean_tokens: float
    early_exit_rate: float


def summarize(reqs: Sequence[Request], res: Sequence[Result], slo_s: float) -> Summary:
    n = len(res)
    if n == 0:
        return Summary(0, 0, 0, 0, 0, 0, 0, 0)
    lat = sorted(r.latency_s for r in res)
    rank = max(1, math.ceil(0.95 * n))
    span = max(r.finish_s for r in res) - min(q.arrival_s for q in reqs)
    return Summary(
        n=n,
        mean_latency_s=sum(r.latency_s for r in res) / n,
        p95_latency_s=lat[rank - 1],
        throughput_qps=n / span if span > 0 else 0.0,
        slo_rate=sum(r.latency_s <= slo_s for r in res) / n,
        accuracy=sum(r.correct for r in res) / n,
        mean_tokens=sum(r.think_tokens + q.conclusion_tokens for r, q in zip(res, reqs)) / n,
        early_exit_rate=sum(r.outcome == EXITED for r in res) / n,
    )


def number_in_system_area(reqs: Sequence[Request], res: Sequence[Result]) -> float:
    """Integral over time of the number of requests in the system, from the event times."""
    pts = [(q.arrival_s, 1) for q in reqs] + [(r.finish_s, -1) for r in res]
    pts.sort(key=lambda x: (x[0], -x[1]))
    area, count, last = 0.0, 0, None
    for t, d in pts:
        if last is not None:
            area += count * (t - last)
        count += d
        last = t
    return area
