"""Confidence, max-probability and exit-decision parity where the confidence spans (0, 1).

A random-initialised decoder has nearly flat next-token distributions: every max-softmax
probability is about 1/V (about 1e-3 at the 7B shape), so an absolute confidence tolerance
of 1e-3 alone cannot fail and no confidence comes near an exit threshold.  Scaling the
final RMSNorm gain by g scales every logit by g (the norm's output feeds the LM head
linearly); the logits' spread is about 0.02 g sqrt(d_model), so g = 4, 8, 16 (and 32 at the
tiny shape's d_model of 256) spread the max-probabilities over (0, 1).  Powers of two are
exact in bf16, so both sides hold the same weights.

Each probe is checked two ways against the oracle's probe at the same state (Section 3.1):
  * as laser_probe_confidence runs it (trial tokens fed back on the device): logits and
    tokens while they agree, tokens exact where the oracle's top-2 margin exceeds 1e-2, the
    confidence whenever all trial tokens agree;
  * teacher-forced (forced_probe: a fork whose trial inputs are the oracle's tokens), so every
    p_j and the confidence are compared in every case.
Max-probabilities and confidences are held to 1e-3 absolute and to the relative bound that
the 2e-2 logit tolerance implies.  The confidences then drive laser_exit_decision over a
threshold grid against the oracle controller (Algorithm 1, Eq. 5): identical decisions
wherever |C - lambda| > 1e-3.
"""
import gc
import sys
import time

import numpy as np
import pytest
import torch

from gpu_helpers import (MARGIN, check_exit_decisions, check_prob, check_token, compare_forced_probe,
                         compare_logits, forced_probe, kv_pair, make_pair, require_gpu, riding_forwards,
                         set_final_gain)
from oracle.transformer import SeqState, lm_stats
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import QWEN_1P5B, QWEN_7B, TINY

pytestmark = pytest.mark.gpu

S, T = 8, 4
T0 = [time.time()]


def log(*a):
    print(f"[{time.time() - T0[0]:6.1f}s]", *a, flush=True)
    sys.stdout.flush()


def decode_and_check(model, kv, opool, orc, states, seqs, toks, what):
    """One teacher-forced decode step (the oracle's tokens in), checked row by row."""
    B, V = len(seqs), model.shape.vocab
    d_tok = torch.tensor(toks, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(B, dtype=torch.int32, device="cuda")
    d_p = torch.zeros(B, device="cuda")
    d_logits = torch.zeros(B, V, device="cuda")
    L.laser_decode_step(model, kv, seqs, d_tok, d_next, d_p, d_logits)
    torch.cuda.synchronize()
    lg = d_logits.cpu().numpy()
    for i, b in enumerate(seqs):
        opool.append(b, 1)
        ref = orc.decode_token(states[b], toks[i])
        compare_logits(lg[i], ref, f"{what} seq {b}")
        check_token(d_next[i].item(), ref, f"{what} seq {b}")
        check_prob(d_p[i].item(), lm_stats(ref)[1], f"{what} seq {b} p_max")
        toks[i] = lm_stats(ref)[0]
        assert kv.page_table(b) == opool.tables[b]


def probe_both_ways(model, kv, opool, orc, states, seqs, fork, suffix, d_suffix, what):
    """Runs the probe of every request as laser_probe_confidence and teacher-forced; returns
    the (GPU confidence, oracle confidence) pairs of the teacher-forced runs."""
    B, V = len(seqs), model.shape.vocab
    d_conf = torch.zeros(B, device="cuda")
    d_arg = torch.zeros(B * T, dtype=torch.int32, device="cuda")
    d_log = torch.zeros(B * T, V, device="cuda")
    L.laser_probe_confidence(model, kv, seqs, d_suffix, T, d_conf, d_arg, d_log)
    torch.cuda.synchronize()
    conf, arg = d_conf.cpu().numpy(), d_arg.cpu().numpy().reshape(B, T)
    lg = d_log.cpu().numpy().reshape(B, T, V)
    pairs, n_untaught = [], 0
    for i, b in enumerate(seqs):
        res = orc.probe(states[b], suffix, T, keep_logits=True)
        agree = True
        for j in range(T):
            if not agree:
                break
            compare_logits(lg[i, j], res.logits[j], f"{what} seq {b} trial {j}")
            if res.margins[j] > MARGIN:
                assert arg[i, j] == res.tokens[j], f"{what} seq {b} trial {j}: {arg[i, j]} vs {res.tokens[j]}"
            agree = int(arg[i, j]) == res.tokens[j]
        if agree:
            check_prob(conf[i], res.confidence, f"{what} seq {b} confidence (device feedback)")
            n_untaught += 1
        got = forced_probe(model, kv, b, fork, d_suffix, res.tokens, T, V)
        compare_forced_probe(res, got, f"{what} seq {b} (teacher-forced)")
        pairs.append((got[2], res.confidence))
        assert kv.page_table(b) == opool.tables[b] and kv.seq_len(b) == states[b].length, f"{what}: cache changed"
        log(f"{what} seq {b}: C gpu {got[2]:.6g} (device feedback {conf[i]:.6g}) oracle {res.confidence:.6g}, "
            f"p_max {np.round(res.pmax, 4).tolist()}")
    return pairs, n_untaught


def spread_check(pairs, what):
    """The confidences reach well into (0, 1) and differ from each other, so the checks above
    and the exit decisions are exercised away from the flat random-init regime."""
    cs = [co for _, co in pairs]
    assert max(cs) > 0.3 and max(cs) - min(cs) > 0.2, f"{what}: confidences {cs}"


def test_peaked_tiny():
    T0[0] = time.time()
    require_gpu()
    V = TINY.vocab
    model, orc, _ = make_pair(TINY, max_rows=32, max_positions=1024)
    kv, opool = kv_pair(model, TINY, num_pages=200, max_seqs=8, max_pages_per_seq=64)
    lens = [40, 100, 250]
    states = []
    for s, n in enumerate(lens):
        K0, V0 = synth.make_prefill_kv(TINY, n, 60 + s)
        kv.add_seq(s, n)
        opool.add_seq(s, n)
        kv.import_kv(s, K0.cuda(), V0.cuda())
        states.append(SeqState.from_prefill(TINY, K0.numpy(), V0.numpy(), 1024))
    seqs = [0, 1, 2]
    suffix = [int(t) for t in synth.make_suffix(S, V)]
    d_suffix = torch.tensor(suffix, dtype=torch.int32, device="cuda")
    toks = [int(t) for t in synth.make_tokens(3, V, 3020)]
    pairs, untaught = [], 0
    for g in (4, 8, 16, 32):
        set_final_gain(model, orc, float(g))
        for step in range(2):
            decode_and_check(model, kv, opool, orc, states, seqs, toks, f"tiny g={g} step {step}")
        pr, nu = probe_both_ways(model, kv, opool, orc, states, seqs, 5, suffix, d_suffix, f"tiny g={g}")
        pairs += pr
        untaught += nu
    spread_check(pairs, "tiny")
    assert untaught >= len(pairs) // 2
    n = check_exit_decisions(pairs, "tiny")
    log(f"tiny: {len(pairs)} confidences, {n} exit decisions compared")


def test_peaked_qwen1p5b_kv4096():
    T0[0] = time.time()
    require_gpu()
    shape = QWEN_1P5B
    V = shape.vocab
    n0, cap = 4096, 4096 + 64
    model, orc, _ = make_pair(shape, max_rows=16, max_positions=cap, weights_on_device=True, cache_oracle=True)
    kv, opool = kv_pair(model, shape, num_pages=n0 // 16 + 24, max_seqs=2, max_pages_per_seq=cap // 16 + 1)
    K0, V0 = synth.make_prefill_kv(shape, n0, 0, device="cuda")
    kv.add_seq(0, n0)
    opool.add_seq(0, n0)
    kv.import_kv(0, K0, V0)
    states = [SeqState.from_prefill(shape, synth.to_numpy(K0), synth.to_numpy(V0), cap)]
    del K0, V0
    suffix = [int(t) for t in synth.make_suffix(S, V)]
    d_suffix = torch.tensor(suffix, dtype=torch.int32, device="cuda")
    toks = [int(synth.make_tokens(1, V, 3021)[0])]
    log("1.5B setup done")
    pairs = []
    for g in (4, 8, 16):
        set_final_gain(model, orc, float(g))
        decode_and_check(model, kv, opool, orc, states, [0], toks, f"1.5B g={g}")
        pr, _ = probe_both_ways(model, kv, opool, orc, states, [0], 1, suffix, d_suffix, f"1.5B g={g}")
        pairs += pr
    spread_check(pairs, "1.5B")
    n = check_exit_decisions(pairs, "1.5B")
    log(f"1.5B: {n} exit decisions compared")
    kv.destroy()
    model.destroy()
    del orc, states
    gc.collect()
    torch.cuda.empty_cache()


def test_peaked_qwen7b_b1_kv14336_and_riding():
    # The benchmark's configuration: 7B shape, batch 1, 14,336 positions.  Probes at
    # g = 4, 8, 16 both ways, then (g = 8) the benchmark's riding pattern: a fork at the ATP
    # whose 8 suffix rows ride beside the decode row (a 9-row forward over one shared-prefix
    # group plus the fork's own copied page), then one trial row per forward (2 rows).
    T0[0] = time.time()
    require_gpu()
    shape = QWEN_7B
    V = shape.vocab
    n0, cap = 14336, 14336 + 64
    model, orc, _ = make_pair(shape, max_rows=16, max_positions=cap, weights_on_device=True, cache_oracle=True,
                              oracle_dtype=np.float32)
    kv, opool = kv_pair(model, shape, num_pages=n0 // 16 + 32, max_seqs=3, max_pages_per_seq=cap // 16 + 1)
    K0, V0 = synth.make_prefill_kv(shape, n0, 0, device="cuda")
    kv.add_seq(0, n0)
    opool.add_seq(0, n0)
    kv.import_kv(0, K0, V0)
    states = [SeqState.from_prefill(shape, synth.to_numpy(K0), synth.to_numpy(V0), cap, dtype=np.float32)]
    del K0, V0
    suffix = [int(t) for t in synth.make_suffix(S, V)]
    d_suffix = torch.tensor(suffix, dtype=torch.int32, device="cuda")
    log("7B setup done")
    pairs = []
    for g in (4, 8, 16):
        set_final_gain(model, orc, float(g))
        pr, _ = probe_both_ways(model, kv, opool, orc, states, [0], 1, suffix, d_suffix, f"7B g={g}")
        pairs += pr
    # one decode step first, so the fork copies a partial last page
    set_final_gain(model, orc, 8.0)
    toks = [int(synth.make_tokens(1, V, 3022)[0])]
    decode_and_check(model, kv, opool, orc, states, [0], toks, "7B g=8 decode")
    pairs += riding_forwards(model, orc, kv, opool, states, [0], [[0], [], [], []], {(0, 0)}, [1, 2], suffix, S, T,
                             5022, "7B riding g=8", log=log)
    spread_check(pairs, "7B")
    n = check_exit_decisions(pairs, "7B")
    log(f"7B: {n} exit decisions compared")
    kv.destroy()
    model.destroy()
    del orc, states
    gc.collect()
    torch.cuda.empty_cache()
