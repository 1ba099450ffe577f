"""The paper's serving experiments (Section 5.2-5.4) on this engine's measured costs.

    python -m paper_2606_31580_amd.serving [--costs profiles/bench_7b_b1_kv14336.json] [--n 125] [--json]

Runs the native simulation (laser_simulate: one FIFO server, per-request inference time from
Eq. 2) on synthetic reasoning traces (synth.make_sim_traces) with the cost model that
bench.py measures on the GPU (decode and probe time against context, prompt prefill).
Prints the layout of Table 1 (latency, P95, throughput, SLO rate per method at QPS 0.5, 2
and 8), Table 2 (the 1 -> 5 -> 1 QPS burst, 10 minutes per phase) and the ablation of
Section 5.4 (QPS 2).  The traces stand in for per-sample profiles of trained models, so
the tables show the structure of the paper's comparison, not its values.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

from . import laser as L
from . import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEFAULT_COSTS = os.path.join(ROOT, "profiles", "bench_7b_b1_kv14336.json")

METHODS = [("Vanilla", L.SIM_VANILLA, 0.95), ("NoThinking", L.SIM_NOTHINKING, 0.95),
           ("Fixed-High", L.SIM_FIXED, 0.95), ("Fixed-Low", L.SIM_FIXED, 0.90), ("LASER", L.SIM_LASER, 0.95)]
ABLATION = [("Fixed threshold", L.SIM_FIXED, 0.95), ("Threshold only", L.SIM_THRESHOLD_ONLY, 0.95),
            ("Budget only", L.SIM_BUDGET_ONLY, 0.95), ("LASER", L.SIM_LASER, 0.95)]
KEYS = ("prefill_ms", "prefill_ms_per_token", "decode_ms", "decode_ms_per_ctx", "probe_ms", "probe_ms_per_ctx")


def load_costs(path: str) -> dict:
    rec = json.load(open(path))
    costs = rec.get("sim_costs") if isinstance(rec, dict) else None
    if not costs:
        raise SystemExit(f"{path} has no sim_costs (run bench.py on a one-request workload)")
    return {k: float(costs[k]) for k in KEYS}


def run(costs: dict, n: int = 125, seed: int = 6000, slo_s: float = 30.0) -> dict:
    p = L.laser_params_default()
    out = {"qps": {}, "burst": {}, "ablation": {}}

    def summary(method, lam, arrivals, tr):
        _, s = L.laser_simulate(p, L.sim_config(method, costs, fixed_lambda=lam, slo_s=slo_s), arrivals, tr)
        return {"mean_latency_s": s.mean_latency_s, "p95_latency_s": s.p95_latency_s, "throughput_qps": s.throughput_qps,
                "slo_pct": 100 * s.slo_rate, "accuracy_pct": 100 * s.accuracy, "mean_tokens": s.mean_tokens,
                "early_exit_pct": 100 * s.early_exit_rate, "n": s.n}

    tr = synth.make_sim_traces(n, seed=seed)
    for qps in (0.5, 2.0, 8.0):
        arr = synth.make_poisson_arrivals(n, qps, seed=7000)
        out["qps"][qps] = {name: summary(m, lam, arr, tr) for name, m, lam in METHODS}
        if qps == 2.0:
            out["ablation"] = {name: summary(m, lam, arr, tr) for name, m, lam in ABLATION}
    arr = synth.make_phased_arrivals([1.0, 5.0, 1.0], [600.0, 600.0, 600.0], seed=7001)
    trb = synth.make_sim_traces(len(arr), seed=seed + 1)
    out["burst"] = {name: summary(m, lam, arr, trb) for name, m, lam in METHODS}
    out["burst_requests"] = len(arr)
    return out


def format_tables(res: dict) -> str:
    lines = ["Table 1 layout: mean latency (s), P95 (s), throughput (QPS), SLO (%), accuracy (%)"]
    for qps, rows in res["qps"].items():
        lines.append(f"  QPS={qps}")
        for name, r in rows.items():
            lines.append(f"    {name:<11s} {r['mean_latency_s']:9.1f} {r['p95_latency_s']:9.1f} {r['throughput_qps']:7.3f} "
                         f"{r['slo_pct']:6.1f} {r['accuracy_pct']:6.1f}")
    lines.append(f"Table 2 layout: burst 1 -> 5 -> 1 QPS, 10 min each ({res['burst_requests']} requests)")
    for name, r in res["burst"].items():
        lines.append(f"    {name:<11s} {r['mean_latency_s']:9.1f} {r['p95_latency_s']:9.1f} {r['throughput_qps']:7.3f} "
                     f"{r['slo_pct']:6.1f} {r['accuracy_pct']:6.1f}")
    lines.append("Ablation (Section 5.4 layout), QPS=2: mean latency (s), throughput, accuracy (%)")
    for name, r in res["ablation"].items():
        lines.append(f"    {name:<16s} {r['mean_latency_s']:9.1f} {r['throughput_qps']:7.3f} {r['accuracy_pct']:6.1f}")
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--costs", default=DEFAULT_COSTS, help="a bench.py JSON line with sim_costs")
    ap.add_argument("--n", type=int, default=125, help="requests per QPS run")
    ap.add_argument("--json", action="store_true")
    args = ap.parse_args(argv)
    costs = load_costs(args.costs)
    res = run(costs, n=args.n)
    if args.json:
        print(json.dumps({"costs": costs, **{k: v for k, v in res.items()}}, default=str))
    else:
        print("costs (ms): " + ", ".join(f"{k}={v:g}" for k, v in costs.items()))
        print(format_tables(res))


if __name__ == "__main__":
    sys.exit(main())
