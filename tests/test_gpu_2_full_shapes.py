"""GPU parity at full model sizes by state injection.

The GPU runs the real configuration (same kernels and launch plans the benchmark
times); the oracle starts from the same pre-filled KV and weights (host copies) and
computes the sampled outputs one token at a time: decode logits, greedy tokens,
max-probabilities, the probe's confidence and trial tokens, page tables.
"""
import sys
import time

import numpy as np
import pytest
import torch

from gpu_helpers import PROB_TOL, check_token, compare_logits, export_seq, make_pair, require_gpu
from oracle.transformer import SeqState, lm_stats
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import QWEN_1P5B

pytestmark = pytest.mark.gpu

S, T = 8, 4


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_state_injection(shape, lens, n_steps, probe_seq=0, max_rows=16):
    dev = require_gpu()
    t0 = time.time()
    max_pos = max(lens) + n_steps + S + T + 64
    model, orc, _ = make_pair(shape, max_rows=max_rows, max_positions=max_pos, weights_on_device=True,
                              cache_oracle=True)
    pps = max_pos // 16 + 1
    kv = L.KVCache(model, sum(n // 16 + 4 for n in lens) + 8, len(lens), pps)
    states = []
    for i, n in enumerate(lens):
        k0, v0 = synth.make_prefill_kv(shape, n, i, device=dev)
        kv.add_seq(i, n)
        kv.import_kv(i, k0, v0)
        states.append(SeqState.from_prefill(shape, synth.to_numpy(k0), synth.to_numpy(v0), max_pos))
        del k0, v0
    log(f"{shape.name}: setup {time.time() - t0:.1f}s")
    B = len(lens)
    V = shape.vocab
    seqs = list(range(B))
    toks = [int(t) for t in synth.make_tokens(B, V, 3003)]
    d_tok = torch.zeros(B, dtype=torch.int32, device=dev)
    d_next = torch.zeros(B, dtype=torch.int32, device=dev)
    d_p = torch.zeros(B, device=dev)
    d_logits = torch.zeros(B, V, device=dev)
    for step in range(n_steps):
        d_tok.copy_(torch.tensor(toks, dtype=torch.int32))
        L.laser_decode_step(model, kv, seqs, d_tok, d_next, d_p, d_logits)
        torch.cuda.synchronize()
        for b in seqs:
            ref = orc.decode_token(states[b], toks[b])
            err = compare_logits(d_logits[b].cpu().numpy(), ref, f"step {step} seq {b}")
            check_token(d_next[b].item(), ref, f"step {step} seq {b}")
            assert abs(d_p[b].item() - lm_stats(ref)[1]) <= PROB_TOL
            toks[b] = lm_stats(ref)[0]
            log(f"{shape.name} step {step} seq {b}: logits err {err:.3g} ({time.time() - t0:.0f}s)")
    # the probe of one request at full size
    suffix = [int(t) for t in synth.make_suffix(S, V)]
    d_suffix = torch.tensor(suffix, dtype=torch.int32, device=dev)
    table = kv.page_table(probe_seq)
    d_conf = torch.zeros(1, device=dev)
    d_arg = torch.zeros(T, dtype=torch.int32, device=dev)
    d_plog = torch.zeros(T, V, device=dev)
    L.laser_probe_confidence(model, kv, [probe_seq], d_suffix, T, d_conf, d_arg, d_plog)
    torch.cuda.synchronize()
    res = orc.probe(states[probe_seq], suffix, T, keep_logits=True)
    agree = True
    for j in range(T):
        if not agree:
            break
        compare_logits(d_plog[j].cpu().numpy(), res.logits[j], f"probe trial {j}")
        tok, _, margin = lm_stats(res.logits[j])
        agree = int(d_arg[j].item()) == tok
        if margin > 1e-2:
            assert agree
    if agree:
        assert abs(d_conf.item() - res.confidence) <= PROB_TOL
    assert kv.page_table(probe_seq) == table
    log(f"{shape.name}: probe conf gpu {d_conf.item():.6g} oracle {res.confidence:.6g} ({time.time() - t0:.0f}s)")
    return model, kv


def test_qwen1p5b_kv4096_state_injection():
    run_state_injection(QWEN_1P5B, [4096], n_steps=2)
