#!/usr/bin/env python3
"""Throughput of the LASER decode + confidence-probe hot path on one MI355X.

One step = one chain-of-thought decode token for every request of the batch; every
`probe_every` steps each request also runs the trial-answer probe (S=8 suffix tokens,
T=4 trial tokens) and the host takes the load-aware exit decision on its confidence,
as at an action transition point.  By default the probe rides along: the request is
forked at the ATP and the fork's suffix rows (one per forward by default) and fed-back
trial tokens join the next decode forwards, so the probe costs an extra row in those
forwards instead of its own weight passes; the decision follows S + T - 1 forwards later.  With
--probe-mode separate the probe runs as its own forwards between decode steps.  Inputs are synthetic and seeded: random-initialised
weights of the named shape and pre-filled random KV (stand-ins for the paper's trained
reasoners and their chains of thought, which are not available here).

Prints one JSON line.  `value` is whole-job decode throughput (tokens/s) with the
probes and exit decisions inside the timed region: ATPs are counted from the first timed
step (a probe at timed step 0, then every `probe_every` steps), so any run of at least
S/probe-rows + T - 1 steps times at least one whole riding probe.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
PAGE = 16
COST_CTX = 2048  # the shorter context of the cost-model pass


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default="7B-b1-kv14336")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-only", action="store_true", help="steps only, no reporting (for rocprofv3 runs)")
    ap.add_argument("--probe-mode", choices=["riding", "separate"], default="riding",
                    help="riding: each probe's rows ride along with the next decode forwards on a fork of the "
                         "request; separate: the probe runs as its own forwards between decode steps")
    ap.add_argument("--probe-rows", type=int, default=8, help="probe rows per forward in riding mode")
    ap.add_argument("--no-tiles", action="store_true", help="MFMA path reads the row-major weights (no tile copy)")
    ap.add_argument("--gemm-kernel", type=int, choices=[0, 1, 2], default=0,
                    help="matrix-core projections: 0 by cost, 1 K-split waves only, 2 row waves where they apply")
    ap.add_argument("--attn-merge", choices=["fused", "kernel"], default="kernel",
                    help="one-row attention groups: merged by the attention kernel's last workgroup (fused) or "
                         "by the separate merge kernel")
    ap.add_argument("--attn-splits", type=int, default=56, help="split bound of a fused one-row attention group")
    ap.add_argument("--oproj-merge", choices=["auto", "on", "off"], default="auto",
                    help="split merge of 1-2 row forwards: inside the O-projection's launch (on), as its own "
                         "kernel (off), or inside the launch for projections of at least 16 MiB of weights (auto)")
    ap.add_argument("--design-probes", action="store_true",
                    help="only run the design-probe program (streaming read, kernel boundary, cross-workgroup "
                         "hand-off, grid barrier, dependent products) and print its report")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device-to-device copy three times (scale for HBM byte counters)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    if args.design_probes:  # a child process: nothing here has touched the GPU
        import subprocess

        exe = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2606_31580_amd", "lib", "design_probes")
        if not os.path.exists(exe):
            print(f"{exe} is missing: build with `python -m paper_2606_31580_amd.build`", file=sys.stderr)
            sys.exit(2)
        sys.exit(subprocess.run([exe]).returncode)
    import numpy as np
    import torch

    if args.copy_calibration:
        n = 256 << 20
        src = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: 3 copies of {n} bytes", file=sys.stderr, flush=True)
        return

    from paper_2606_31580_amd import laser as L
    from paper_2606_31580_amd import synth
    from paper_2606_31580_amd.configs import WORKLOADS

    wl = WORKLOADS[args.workload]
    shape = wl.shape
    dev = torch.device("cuda:0")
    B = wl.batch
    S, T = wl.suffix_len, wl.trial_len
    lens = list(wl.kv_lens) if wl.kv_lens else synth.make_ragged_lengths(B, 3000, 14000)
    total_steps = args.warmup + args.steps
    max_pos = max(lens) + 2 * total_steps + S + T + 2 * PAGE
    max_pos = min(65536, (max_pos + 255) // 256 * 256)

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    log(f"workload {wl.name}: generating weights")
    weights = synth.make_weights(shape, device=dev)
    R = args.probe_rows
    if wl.mixed:  # every step: decode for the batch + probe chunks of a seeded half, one forward
        schedule = synth.make_mixed_schedule(B, total_steps + 64)
        if args.probe_mode == "riding":  # decode rows + new suffix chunks + one trial row per probe in flight
            rows = B + max(len(x) for x in schedule) * (S + T - 1)
        else:
            rows = max(B + max(len(x) for x in schedule) * S, B * S)
    else:
        rows = max(B + B * R, B * S)
    if rows > 64:
        log(f"{rows} rows per forward exceed the 64-row maximum; use fewer probe rows")
        sys.exit(2)
    # the workspace takes the full 64 rows so that prompt prefills run in 64-token chunks
    model = L.Model(shape, weights, max_rows=64, max_positions=max_pos, tiles=not args.no_tiles)
    model.set_gemm_kernel(args.gemm_kernel)
    model.set_attn_merge(args.attn_merge == "fused", args.attn_splits)
    model.set_oproj_merge({"off": 0, "auto": 1, "on": 2}[args.oproj_merge])
    pps = max_pos // PAGE + 1
    num_pages = sum((n + 2 * total_steps + S + T) // PAGE + 2 for n in lens) + B * ((S + T) // PAGE + 3) + 8
    num_pages += (COST_CTX + 512) // PAGE + 4  # the cost-model pass (a shorter request in a fork slot)
    # fork slots after the B requests: one per request, or (mixed workload, riding probes) one per
    # probe in flight: a seeded half of the batch starts a probe every step and each lives T forwards
    P_SLOTS = max(len(x) for x in schedule) * T if (wl.mixed and args.probe_mode == "riding") else B
    num_pages += P_SLOTS * ((S + T) // PAGE + 3)
    kv = L.KVCache(model, num_pages, B + P_SLOTS, pps)
    for i, n in enumerate(lens):
        k0, v0 = synth.make_prefill_kv(shape, n, i, device=dev)
        kv.add_seq(i, n)
        kv.import_kv(i, k0, v0)
        del k0, v0
    torch.cuda.synchronize()
    seqs = list(range(B))
    forks = [B + b for b in seqs]
    tokens = synth.make_tokens(B, shape.vocab, 3003).to(dev)
    nxt = tokens  # greedy feedback in place: each forward's next tokens overwrite its inputs
    pmax = torch.empty(B, device=dev)
    suffix = synth.make_suffix(S, shape.vocab).to(dev)
    conf = torch.empty(B, device=dev)
    argm = torch.empty(B * T, dtype=torch.int32, device=dev)
    ptrial = torch.empty(B * T, device=dev)
    params = L.laser_params_default()
    load_state = L.laser_load_state(0.0)
    stream = torch.cuda.current_stream()

    probe_ms = []  # riding: fork to confidence (device time, the decode forwards included); separate: the probe
    n_probes = [0]
    ride = {}  # progress of the riding probes in flight: suffix rows and trial tokens done

    def decide(c):
        for b in range(B):  # the controller needs the confidence on the host
            L.laser_exit_decision(params, load_state, float(c[b]), B, 0, 10)
        n_probes[0] += 1

    # Riding probes: the confidences go to the host by an asynchronous copy, and the exit
    # decisions are taken once the next forward is queued (settle), so the GPU never waits
    # for the host round trip.  A request that exits is told one decode step later.  Two
    # pinned buffers in turn; at most one copy is pending at a time.
    conf_h = [torch.empty(max(B, 1), pin_memory=True) for _ in range(2)]
    pend = []  # [copy event, host buffer, confidences, per-request decisions?, (fork, conf) events, timed]
    turn = [0]

    def send(n, per_request, evs, timed):
        hb = conf_h[turn[0]]
        turn[0] ^= 1
        hb[:n].copy_(conf[:n], non_blocking=True)
        ev = torch.cuda.Event()
        ev.record(stream)
        pend.append((ev, hb, n, per_request, evs, timed))

    def settle():
        while pend:
            ev, hb, n, per_request, evs, timed = pend.pop(0)
            ev.synchronize()
            c = hb[:n].numpy()
            if per_request:
                decide(c)
            else:
                for k in range(n):
                    L.laser_exit_decision(params, load_state, float(c[k]), B, 0, 10)
                n_probes[0] += n
            if timed:  # device time from the fork to the confidence (the decode forwards included)
                probe_ms.extend(e0.elapsed_time(e1) for e0, e1 in evs)

    # mixed workload, riding probes: each probe is a fork of its request (slot B + f) whose S
    # suffix rows ride in one forward and whose T-1 trial rows ride in the next forwards, all
    # beside the batch's decode rows.  tokbuf = [suffix | T trial tokens per slot]; the
    # trial tokens are written and read there, their probabilities at the same offsets of pbuf.
    tokbuf = torch.zeros(S + P_SLOTS * T, dtype=torch.int32, device=dev)
    tokbuf[:S].copy_(suffix)
    pbuf = torch.zeros(S + P_SLOTS * T, device=dev)
    free_slots = list(range(P_SLOTS))
    inflight = []  # [slot, request, trials done, fork event]
    skipped = [0]

    def step_mixed_riding(i, timed_probe, new_probes=True):
        spans = [L.span(b, 1, 0, b, out=(0, b)) for b in seqs]
        for pr in inflight:  # one trial row per probe in flight, fed its previous trial token
            f, j = pr[0], pr[2] + 1
            spans.append(L.span(B + f, 1, 1, S + f * T + j - 1, out=(1, S + f * T + j)))
            pr[2] = j
        if new_probes:
            for b in schedule[i % len(schedule)]:
                if not free_slots:
                    skipped[0] += 1
                    continue
                f = free_slots.pop()
                ev0 = torch.cuda.Event(enable_timing=True)
                ev0.record(stream)
                kv.fork(b, B + f)
                spans.append(L.span(B + f, S, 1, 0, out=(1, S + f * T)))
                inflight.append([f, b, 0, ev0])
        L.laser_forward(model, kv, spans, tokens, tokbuf, nxt, pmax, tokbuf, pbuf)
        settle()  # the previous step's decisions, this step's forward being queued
        done = [pr for pr in inflight if pr[2] == T - 1]
        if not done:
            return
        for k, pr in enumerate(done):
            L.laser_confidence(model, pbuf[S + pr[0] * T:], T, 1, conf[k:])
        ev1 = torch.cuda.Event(enable_timing=True)
        ev1.record(stream)
        send(len(done), False, [(pr[3], ev1) for pr in done], timed_probe)
        for pr in done:  # (later forwards are stream-ordered after this one's use of the pages)
            kv.free_seq(B + pr[0])
            free_slots.append(pr[0])
            inflight.remove(pr)

    def step(i, timed_probe):
        if wl.mixed and args.probe_mode == "riding":
            step_mixed_riding(i, timed_probe)
            return
        if wl.mixed:  # the probes of this step run in the same forwards as its decode
            pidx = schedule[i % len(schedule)]
            L.laser_step_mixed(model, kv, seqs, tokens, nxt, pmax, pidx, suffix, T, conf, argm)
            c = conf.cpu().numpy()
            for j in range(len(pidx)):
                L.laser_exit_decision(params, load_state, float(c[j]), B, 0, 10)
            n_probes[0] += len(pidx)
            return
        at_atp = wl.probe_every and i % wl.probe_every == 0
        if args.probe_mode == "separate":
            L.laser_decode_step(model, kv, seqs, tokens, nxt, pmax)
            if at_atp:
                if timed_probe:  # latency of the probe itself, not of decode steps still queued
                    torch.cuda.synchronize()
                t0 = time.perf_counter()
                L.laser_probe_confidence(model, kv, seqs, suffix, T, conf, argm)
                decide(conf.cpu().numpy())
                if timed_probe:
                    probe_ms.append((time.perf_counter() - t0) * 1e3)
            return
        if at_atp and not ride:  # fork every request at its current length
            ev0 = torch.cuda.Event(enable_timing=True)
            ev0.record(stream)
            for b in seqs:
                kv.fork(b, forks[b])
            ride.update(s=0, t=0, ev0=ev0)
        spans = [L.span(b, 1, 0, b, out=(0, b)) for b in seqs]
        tok1 = None
        if ride:
            if ride["s"] < S:
                k = min(R, S - ride["s"])
                last = ride["s"] + k == S
                spans += [L.span(forks[b], k, 1, ride["s"], out=(1, b * T) if last else None) for b in seqs]
                tok1 = suffix
                ride["s"] += k
            else:
                ride["t"] += 1
                j = ride["t"]
                spans += [L.span(forks[b], 1, 1, b * T + j - 1, out=(1, b * T + j)) for b in seqs]
                tok1 = argm
        L.laser_forward(model, kv, spans, tokens, tok1, nxt, pmax, argm, ptrial)
        settle()  # the previous step's decisions, this step's forward being queued
        if ride and ride["s"] == S and ride["t"] == T - 1:
            L.laser_confidence(model, ptrial, T, B, conf)
            ev1 = torch.cuda.Event(enable_timing=True)
            ev1.record(stream)
            send(B, True, [(ride["ev0"], ev1)], timed_probe)
            for b in seqs:  # (later forwards are stream-ordered after this one's use of the pages)
                kv.free_seq(forks[b])
            ride.clear()

    # ATPs fall on step indices counted from the start of each phase (warm-up, timed), so the
    # timed region begins with a probe whatever the warm-up length.
    log("warmup")
    for i in range(args.warmup):
        step(i, False)
    while ride:  # no probe crosses into the timed region
        step(-1, False)
    while inflight:
        step_mixed_riding(-1, False, new_probes=False)
    settle()
    torch.cuda.synchronize()
    n_probes[0] = 0

    if args.profile_only:  # the timed loop's work (decode steps with their probes), nothing else
        for i in range(args.steps):
            step(i, False)
        while inflight:
            step_mixed_riding(-1, False, new_probes=False)
        settle()
        torch.cuda.synchronize()
        log("profile loop done")
        return

    # ---- whole job: decode + probes + host exit decisions (forwards replay captured graphs)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    cap0 = model.graph_stats()[0]
    e0.record(stream)
    w0 = time.perf_counter()
    for i in range(args.steps):
        step(i, True)
    settle()  # the last step's decisions
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_total = e0.elapsed_time(e1)
    ms_per_step = ms_total / args.steps
    captures_timed = model.graph_stats()[0] - cap0  # forwards captured into new graphs while timed
    value = args.steps * B / (ms_total / 1e3)
    probes_timed = n_probes[0]
    while ride:  # a probe still riding: finish it outside the timed region
        step(-1, False)
    while inflight:
        step_mixed_riding(-1, False, new_probes=False)
    settle()
    # reference: the probe run as separate forwards (the cost it has when nothing rides along),
    # device time between stream events around the call
    sep_ms = []
    for _ in range(3):
        torch.cuda.synchronize()
        e0.record(stream)
        L.laser_probe_confidence(model, kv, seqs, suffix, T, conf, argm)
        e1.record(stream)
        torch.cuda.synchronize()
        sep_ms.append(e0.elapsed_time(e1))
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step, {value:.1f} tok/s (wall {wall:.2f}s)")

    # ---- decode only (same cache, no probes)
    n_dec = min(args.steps, 128)
    ctx_dec = kv.seq_len(0) + n_dec / 2.0
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(n_dec):
        L.laser_decode_step(model, kv, seqs, tokens, nxt, pmax)
    e1.record(stream)
    torch.cuda.synchronize()
    dec_ms = e0.elapsed_time(e1) / n_dec

    # ---- kernel timing pass: the same decode steps launched kernel by kernel, each launch
    # ending in a fence-free HIP event on the stream it runs on; a class's launch is timed
    # from the end of the previous kernel to the end of its own last kernel
    classes = {"embed": L.K_EMBED, "qkv": L.K_QKV, "attn+merge": L.K_ATTN, "o_proj": L.K_OPROJ,
               "gate_up": L.K_GATEUP, "down": L.K_DOWN, "lm_head+reduce": L.K_LMHEAD}
    for c in classes.values():
        model.timing_enable(c, True)
    n_kt = min(args.steps, 32)
    for i in range(n_kt):
        L.laser_decode_step(model, kv, seqs, tokens, nxt, pmax)
    kernel_us = {}
    for name, c in classes.items():
        tot_ms, n = model.timing_read(c)
        kernel_us[name] = {"avg_us": round(tot_ms * 1e3 / max(n, 1), 2), "launches": n}
        model.timing_enable(c, False)
    gu_avg_ms = kernel_us["gate_up"]["avg_us"] / 1e3
    gu_n = kernel_us["gate_up"]["launches"]

    # ---- cost model of the serving simulation (one-request workloads)
    sim_costs = None
    if B == 1:
        sim_costs = cost_model(L, synth, model, kv, shape, dev, forks[0], dec_ms, ctx_dec, suffix, T, log)

    # ---- algorithmic bytes
    es = 2 if shape.dtype == "bf16" else 4
    ctx = [kv.seq_len(i) for i in seqs]
    kv_tok = shape.kv_bytes_per_token()
    step_bytes = shape.weight_bytes() + sum(ctx) * kv_tok + B * kv_tok
    step_gbs = step_bytes / (dec_ms / 1e3) / 1e9
    gu_bytes = 2 * shape.d_ffn * shape.d_model * es + B * shape.d_model * 4 + B * shape.d_ffn * 4
    gu_gbs = gu_bytes / (gu_avg_ms / 1e3) / 1e9
    # every class of the kernel-timing pass against the same peak: its algorithmic bytes per
    # launch (the weights once; for attention the K and V of the context in one layer) over its
    # average launch time
    d, hd, F = shape.d_model, shape.head_dim, shape.d_ffn
    cls_bytes = {
        "qkv": (shape.n_q_heads + 2 * shape.n_kv_heads) * hd * d * es,
        "attn+merge": sum(ctx) * kv_tok // shape.n_layers,
        "o_proj": d * shape.n_q_heads * hd * es,
        "gate_up": 2 * F * d * es,
        "down": d * F * es,
        "lm_head+reduce": shape.vocab * d * es,
    }
    class_hbm = {n: {"bytes_per_launch": b,
                     "frac_of_peak": round(b / (kernel_us[n]["avg_us"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
                 for n, b in cls_bytes.items() if kernel_us[n]["avg_us"] > 0}

    traffic = None
    tf = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "gateup_traffic.json")
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2606_31580_amd", "csrc", "gemm.hip")
    if os.path.exists(tf):
        rec = json.load(open(tf))
        cur = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
        if rec.get("gemm_hip_sha256_16") == cur and rec.get("workload") == wl.name:
            traffic = rec.get("bytes_per_launch")

    # host exit decision (EMA, Eq. 5, Algorithm 1), timed outside the timed region through the
    # Python binding (the C call is scalar arithmetic; ctypes dominates)
    dec_state = L.laser_load_state(0.0)
    n_dec = 20000
    t0 = time.perf_counter()
    for i in range(n_dec):
        L.laser_exit_decision(params, dec_state, 0.9, 8, 0, 10)
    host_decision_us = (time.perf_counter() - t0) / n_dec * 1e6

    out = {
        "metric": "decode tok/s + probe latency, achieved HBM GB/s vs peak, 1 GPU",
        "value": round(value, 2),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 weights+KV, fp32 activations" if shape.dtype == "bf16" else "f32",
        "data": "synthetic: random-init weights, seeded pre-filled KV",
        "config": {"workload": wl.name, "model_shape": shape.name, "batch": B, "kv_lens": lens,
                   "probe_every": wl.probe_every, "suffix": S, "trials": T, "attn_merge": args.attn_merge,
                   "attn_splits": args.attn_splits, "oproj_merge": args.oproj_merge},
        "decode_only_ms_per_step": round(dec_ms, 4),
        "decode_only_tok_s": round(B / (dec_ms / 1e3), 2),
        "probe_latency_ms": {"mean": round(float(np.mean(probe_ms)), 3) if probe_ms else None,
                             "p50": round(float(np.median(probe_ms)), 3) if probe_ms else None,
                             "max": round(float(np.max(probe_ms)), 3) if probe_ms else None, "n": len(probe_ms)}
        if not (wl.mixed and args.probe_mode == "separate")
        else {"mean": round(ms_per_step, 3), "p50": None, "max": None, "n": probes_timed},
        "probe_latency_valid": (len(probe_ms) > 0) if not (wl.mixed and args.probe_mode == "separate") else probes_timed > 0,
        "host_decision_us": round(host_decision_us, 3),
        "graph_captures_timed": captures_timed,
        "probe": {"mode": "mixed, riding", "probes_in_timed_region": probes_timed, "forwards_per_probe": T,
                  "probes_skipped_no_slot": skipped[0],
                  "latency_meaning": "device time from the fork to the confidence: the probing half's suffix chunks "
                                     "ride in one forward with the batch's decode rows, each trial row in one of the "
                                     "next T-1",
                  "exit_decision": "on the host, once the next forward is queued (a request that exits stops one step later)",
                  "separate_probe_latency_ms": round(float(np.mean(sep_ms)), 3),
                  "separate_probe_latency_meaning": "device time between stream events around laser_probe_confidence"}
        if wl.mixed and args.probe_mode == "riding" else
                 {"mode": "mixed", "probes_in_timed_region": probes_timed,
                  "latency_meaning": "each step's probes finish within it: one forward with the decode rows and the "
                                     "probing half's suffix chunks, then T-1 forwards of trial rows",
                  "separate_probe_latency_ms": round(float(np.mean(sep_ms)), 3),
                  "separate_probe_latency_meaning": "device time between stream events around laser_probe_confidence"}
        if wl.mixed else
                 {"mode": args.probe_mode, "rows_per_forward": R if args.probe_mode == "riding" else S,
                  "forwards_per_probe": (-(-S // R) + T - 1) if args.probe_mode == "riding" else 1 + T - 1,
                  "probes_in_timed_region": probes_timed,
                  "latency_meaning": "device time from the ATP fork to the confidence, decode forwards included"
                  if args.probe_mode == "riding" else "host time of the probe call with its confidence copy",
                  "exit_decision": "on the host, once the next forward is queued (a request that exits stops one step later)"
                  if args.probe_mode == "riding" else "on the host, after the probe's confidence copy",
                  "separate_probe_latency_ms": round(float(np.mean(sep_ms)), 3),
                  "separate_probe_latency_meaning": "device time between stream events around laser_probe_confidence"},
        "step_hbm": {"bytes": step_bytes, "achieved_GBs": round(step_gbs, 1), "frac_of_peak": round(step_gbs / HBM_PEAK_GBS, 4)},
        "roofline": {"kernel": "gate/up projection + SwiGLU (k_gemv, EPI_SWIGLU)", "bound": "hbm",
                     "achieved": round(gu_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gu_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "avg_launch_us": round(gu_avg_ms * 1e3, 2), "launches": gu_n, "bytes_per_launch": gu_bytes},
        "kernel_us_per_launch": kernel_us,
        "kernel_hbm_frac": class_hbm,
        "sim_costs": sim_costs,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, weights, kv, lens, model, dev, log, S, T)
    print(json.dumps(out), flush=True)


def cost_model(L, synth, model, kv, shape, dev, slot, dec_long_ms, ctx_long, suffix, T, log):
    """Per-token decode, probe and prefill times of this engine, each fitted as a + b * x from
    two measured points: decode steps and probes at the workload's context and at COST_CTX,
    prompt prefills of 64 and 256 tokens.  These drive the serving simulation (Eq. 2)."""
    import torch

    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn, reps):
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(reps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / reps

    log(f"cost model: decode and probe at context {COST_CTX}")
    k0, v0 = synth.make_prefill_kv(shape, COST_CTX, 9, device=dev)
    kv.add_seq(slot, COST_CTX)
    kv.import_kv(slot, k0, v0)
    del k0, v0
    tok = synth.make_tokens(1, shape.vocab, 3005).to(dev)
    pm = torch.empty(1, device=dev)
    conf = torch.empty(1, device=dev)
    argm = torch.empty(T, dtype=torch.int32, device=dev)

    def dec():
        L.laser_decode_step(model, kv, [slot], tok, tok, pm)  # next token in place

    timed(dec, 4)
    n = 32
    ctx_short = kv.seq_len(slot) + n / 2.0
    dec_short_ms = timed(dec, n)
    probe_short_ms = timed(lambda: L.laser_probe_confidence(model, kv, [slot], suffix, T, conf, argm), 3)
    ctx_probe_long = kv.seq_len(0)
    probe_long_ms = timed(lambda: L.laser_probe_confidence(model, kv, [0], suffix, T, conf, argm), 3)
    kv.free_seq(slot)
    log("cost model: prompt prefill of 64 and 256 tokens")
    pre = {}
    for n_p in (64, 256):
        ptok = synth.make_tokens(n_p, shape.vocab, 3006).to(dev)

        def run():
            kv.add_seq(slot, 0)
            L.laser_prefill(model, kv, slot, ptok)
            torch.cuda.synchronize()
            kv.free_seq(slot)

        run()
        t0 = time.perf_counter()
        for _ in range(2):
            run()
        pre[n_p] = (time.perf_counter() - t0) * 1e3 / 2

    def fit(x0, y0, x1, y1):
        b = (y1 - y0) / (x1 - x0)
        return y0 - b * x0, b

    dec_a, dec_b = fit(ctx_short, dec_short_ms, ctx_long, dec_long_ms)
    pr_a, pr_b = fit(COST_CTX, probe_short_ms, ctx_probe_long, probe_long_ms)
    pf_a, pf_b = fit(64, pre[64], 256, pre[256])
    return {"decode_ms": round(dec_a, 5), "decode_ms_per_ctx": round(dec_b, 9),
            "probe_ms": round(pr_a, 4), "probe_ms_per_ctx": round(pr_b, 8),
            "prefill_ms": round(max(pf_a, 0.0), 3), "prefill_ms_per_token": round(pf_b, 5),
            "points": {"decode_ms": [[round(ctx_short, 1), round(dec_short_ms, 4)], [round(ctx_long, 1), round(dec_long_ms, 4)]],
                       "probe_ms": [[COST_CTX, round(probe_short_ms, 3)], [ctx_probe_long, round(probe_long_ms, 3)]],
                       "prefill_ms": [[64, round(pre[64], 3)], [256, round(pre[256], 3)]]},
            "meaning": "ms per decoded token = decode_ms + decode_ms_per_ctx * context; per probe (separate forwards) = "
                       "probe_ms + probe_ms_per_ctx * context; per prompt = prefill_ms + prefill_ms_per_token * tokens"}


def cpu_baseline(shape, weights, kv, lens, model, dev, log, S, T):
    """The oracle, as written (float64 numpy), timed on this host: two decode tokens of request
    0 at its context, BLAS threads set to the cores this process may run on.  A probe of the
    oracle is S + T - 1 such token forwards (its suffix tokens, then the fed-back trial
    tokens) plus a softmax statistic per trial token, so its latency is reported as that many
    measured token times."""
    import platform

    import numpy as np
    import torch
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle.transformer import DecoderOracle, SeqState
    from paper_2606_31580_amd import synth

    cores = len(os.sched_getaffinity(0))
    cpu_model = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    log("cpu baseline: copying weights and the request's KV to the host")
    host = {k: synth.to_numpy(v) for k, v in weights.items()}
    n = kv.seq_len(0)
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    K = torch.empty((shape.n_layers, n, shape.n_kv_heads, shape.head_dim), dtype=dt, device=dev)
    V = torch.empty_like(K)
    kv.export_kv(0, K, V)
    torch.cuda.synchronize()
    st = SeqState.from_prefill(shape, synth.to_numpy(K), synth.to_numpy(V), n + 2)
    del K, V
    orc = DecoderOracle(shape, host)
    toks = [int(t) for t in synth.make_tokens(2, shape.vocab, 3004)]
    log(f"cpu baseline: two oracle decode tokens ({cores} cores)")
    with threadpool_limits(limits=cores, user_api="blas"):
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        secs = []
        for tok in toks:
            t0 = time.perf_counter()
            orc.decode_token(st, tok)
            secs.append(time.perf_counter() - t0)
    sec = float(np.mean(secs))
    blas = ", ".join(sorted({f"{i.get('internal_api', '?')} {i.get('version', '')}".strip() for i in info})) or "unknown"
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    return {"value": round(1.0 / sec, 5), "unit": "tok/s", "cores": threads, "kind": "oracle",
            "sample": f"2 decode tokens of request 0 at context {n}-{n + 1} (float64 numpy, {sum(secs):.1f} s)",
            "probe_latency_ms": round((S + T - 1) * sec * 1e3, 1),
            "probe_latency_meaning": f"{S + T - 1} oracle token forwards (S={S} suffix + T-1={T - 1} trial) at the "
                                     f"measured token time",
            "affinity_cores": cores, "blas_threads": threads, "blas": blas, "cpu_model": cpu_model}


if __name__ == "__main__":
    main()
