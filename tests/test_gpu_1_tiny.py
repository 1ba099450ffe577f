"""GPU parity on the tiny decoder (2 layers, d 256, 4/2 heads of 64, FFN 688, vocab 2048, fp32).

Full run against the oracle: 128-token prompt through the chunked forward, 128 greedy
decode steps (teacher-forced with the oracle's tokens), a confidence probe (S=8, T=4)
every 32 steps; batched and mixed steps; page tables checked bit-exact throughout.
"""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import (LOGIT_TOL, check_prob, check_token, compare_logits, export_seq, kv_pair, make_pair,
                         require_gpu)
from oracle.transformer import SeqState, lm_stats
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import TINY

pytestmark = pytest.mark.gpu

S, T = 8, 4


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def probe_and_compare(model, kv, orc, states, seqs, suffix, d_suffix, what):
    B = len(seqs)
    V = TINY.vocab
    d_conf = torch.empty(B, device="cuda")
    d_arg = torch.empty(B * T, dtype=torch.int32, device="cuda")
    d_log = torch.empty(B * T * V, device="cuda")
    tables = [kv.page_table(s) for s in seqs]
    lens = [kv.seq_len(s) for s in seqs]
    L.laser_probe_confidence(model, kv, seqs, d_suffix, T, d_conf, d_arg, d_log)
    torch.cuda.synchronize()
    conf, arg, lg = d_conf.cpu().numpy(), d_arg.cpu().numpy().reshape(B, T), d_log.cpu().numpy().reshape(B, T, V)
    for b, s in enumerate(seqs):
        res = orc.probe(states[b], suffix, T, keep_logits=True)
        agree = True
        for j in range(T):
            if not agree:
                break
            compare_logits(lg[b, j], res.logits[j], f"{what} seq {s} trial {j}")
            tok, _, margin = lm_stats(res.logits[j])
            if margin > 1e-2:
                assert arg[b, j] == tok, f"{what}: trial token {j}"
            agree = arg[b, j] == tok
        if agree:
            check_prob(conf[b], res.confidence, (what, conf[b], res.confidence))
        assert 0.0 <= conf[b] <= 1.0
        assert kv.page_table(s) == tables[b] and kv.seq_len(s) == lens[b], f"{what}: probe changed the cache state"
    return conf


def test_tiny_full_run():
    require_gpu()
    V = TINY.vocab
    model, orc, _ = make_pair(TINY, max_rows=64, max_positions=512)
    kv, opool = kv_pair(model, TINY, num_pages=64, max_seqs=4, max_pages_per_seq=32)
    kv.add_seq(0, 0)
    opool.add_seq(0, 0)
    prompt = synth.make_tokens(128, V, 3000)
    suffix = [int(t) for t in synth.make_suffix(S, V)]
    d_suffix = torch.tensor(suffix, dtype=torch.int32, device="cuda")
    st = SeqState(TINY, 512)
    for t in prompt:
        ref = orc.decode_token(st, int(t))
    d_last = torch.empty(V, device="cuda")
    L.laser_prefill(model, kv, 0, prompt.cuda(), d_last)
    opool.append(0, 128)
    torch.cuda.synchronize()
    err = compare_logits(d_last.cpu().numpy(), ref, "prefill")
    log(f"prefill logits max err {err:.3g}")
    K, Vv = export_seq(kv, TINY, 0)
    assert np.max(np.abs(K - st.K[:, :128])) < 1e-4 and np.max(np.abs(Vv - st.V[:, :128])) < 1e-4
    assert kv.page_table(0) == opool.tables[0]

    tok = lm_stats(ref)[0]
    d_tok = torch.zeros(1, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(1, dtype=torch.int32, device="cuda")
    d_p = torch.zeros(1, device="cuda")
    d_logits = torch.zeros(1, V, device="cuda")
    worst = 0.0
    for step in range(1, 129):
        d_tok.fill_(tok)
        L.laser_decode_step(model, kv, [0], d_tok, d_next, d_p, d_logits)
        opool.append(0, 1)
        ref = orc.decode_token(st, tok)
        torch.cuda.synchronize()
        worst = max(worst, compare_logits(d_logits[0].cpu().numpy(), ref, f"step {step}"))
        rtok, rp, _ = lm_stats(ref)
        check_token(d_next.item(), ref, f"step {step}")
        check_prob(d_p.item(), rp)
        assert kv.page_table(0) == opool.tables[0] and kv.seq_len(0) == st.length
        tok = rtok
        if step % 32 == 0:
            probe_and_compare(model, kv, orc, [st], [0], suffix, d_suffix, f"probe@{step}")
    log(f"decode logits max err {worst:.3g}")
    K, Vv = export_seq(kv, TINY, 0)
    assert np.max(np.abs(K - st.K[:, :256])) < 1e-4


# gemm_kernel: the matrix-core projections with the K-split kernel (1) and the row-wave kernel
# (2), fp32 weights (two 16-byte loads per step, split into hi/lo)
@pytest.mark.parametrize("gemm_kernel", [1, 2])
def test_tiny_batched_decode_probe_and_mixed(gemm_kernel):
    require_gpu()
    V = TINY.vocab
    model, orc, _ = make_pair(TINY, max_rows=64, max_positions=1024)
    model.set_gemm_kernel(gemm_kernel)
    kv, opool = kv_pair(model, TINY, num_pages=200, max_seqs=8, max_pages_per_seq=64)
    lens = [15, 16, 37, 250]  # page-boundary edge cases and a longer context
    states = []
    for s, n in enumerate(lens):
        K0, V0 = synth.make_prefill_kv(TINY, n, s)
        kv.add_seq(s, n)
        opool.add_seq(s, n)
        kv.import_kv(s, K0.cuda(), V0.cuda())
        states.append(SeqState.from_prefill(TINY, K0.numpy(), V0.numpy(), 1024))
    toks = [int(t) for t in synth.make_tokens(len(lens), V, 3002)]
    seqs = list(range(len(lens)))
    suffix = [int(t) for t in synth.make_suffix(S, V)]
    d_suffix = torch.tensor(suffix, dtype=torch.int32, device="cuda")
    B = len(seqs)
    d_tok = torch.zeros(B, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(B, dtype=torch.int32, device="cuda")
    d_p = torch.zeros(B, device="cuda")
    d_logits = torch.zeros(B, V, device="cuda")
    for step in range(3):
        d_tok.copy_(torch.tensor(toks, dtype=torch.int32))
        L.laser_decode_step(model, kv, seqs, d_tok, d_next, d_p, d_logits)
        torch.cuda.synchronize()
        for b in seqs:
            opool.append(b, 1)
            ref = orc.decode_token(states[b], toks[b])
            compare_logits(d_logits[b].cpu().numpy(), ref, f"batch step {step} seq {b}")
            check_token(d_next[b].item(), ref)
            toks[b] = lm_stats(ref)[0]
            assert kv.page_table(b) == opool.tables[b]
    # batched probe: 4 requests x 8 suffix rows = 32 rows through the MFMA path
    probe_and_compare(model, kv, orc, states, seqs, suffix, d_suffix, "batched probe")
    # mixed step: all decode, requests 1 and 3 also probe in the same forward
    pidx = [1, 3]
    d_conf = torch.empty(len(pidx), device="cuda")
    d_arg = torch.empty(len(pidx) * T, dtype=torch.int32, device="cuda")
    d_tok.copy_(torch.tensor(toks, dtype=torch.int32))
    L.laser_step_mixed(model, kv, seqs, d_tok, d_next, d_p, pidx, d_suffix, T, d_conf, d_arg)
    torch.cuda.synchronize()
    for b in seqs:
        opool.append(b, 1)
    for b in seqs:
        ref = orc.decode_token(states[b], toks[b])
        check_token(d_next[b].item(), ref, f"mixed decode seq {b}")
        check_prob(d_p[b].item(), lm_stats(ref)[1])
    for i, b in enumerate(pidx):
        # scratch pages are taken after every request's committed page and returned afterwards
        opool.append(b, S + T - 1)
    for i, b in enumerate(pidx):
        opool.truncate(b, states[b].length)
    for i, b in enumerate(pidx):
        res = orc.probe(states[b], suffix, T)
        if list(d_arg[i * T:(i + 1) * T].cpu().numpy()) == res.tokens:
            check_prob(d_conf[i].item(), res.confidence)
    for b in seqs:
        assert kv.page_table(b) == opool.tables[b] and kv.seq_len(b) == states[b].length


def test_tiny_determinism_and_errors():
    require_gpu()
    V = TINY.vocab
    model, orc, _ = make_pair(TINY, max_rows=16, max_positions=512)
    outs = []
    for rep in range(2):
        kv, _ = kv_pair(model, TINY, num_pages=40, max_seqs=2, max_pages_per_seq=32)
        K0, V0 = synth.make_prefill_kv(TINY, 300, 9)
        kv.add_seq(1, 300)
        kv.import_kv(1, K0.cuda(), V0.cuda())
        d_tok = torch.tensor([5], dtype=torch.int32, device="cuda")
        d_next = torch.zeros(1, dtype=torch.int32, device="cuda")
        d_p = torch.zeros(1, device="cuda")
        d_logits = torch.zeros(1, V, device="cuda")
        L.laser_decode_step(model, kv, [1], d_tok, d_next, d_p, d_logits)
        torch.cuda.synchronize()
        outs.append(d_logits.clone())
        # errors leave state unchanged
        with pytest.raises(L.LaserError) as e:
            L.laser_decode_step(model, kv, [1, 1], torch.zeros(2, dtype=torch.int32, device="cuda"),
                                torch.zeros(2, dtype=torch.int32, device="cuda"), torch.zeros(2, device="cuda"))
        assert e.value.code == L.ERR_INVALID_ARG and kv.seq_len(1) == 301
        with pytest.raises(L.LaserError) as e:
            L.laser_probe_confidence(model, kv, [1], torch.zeros(17, dtype=torch.int32, device="cuda"), 4,
                                     torch.zeros(1, device="cuda"), torch.zeros(4, dtype=torch.int32, device="cuda"))
        assert e.value.code == L.ERR_INVALID_ARG and kv.seq_len(1) == 301
        kv.destroy()
    assert torch.equal(outs[0], outs[1])  # fixed merge orders: bitwise repeatable
    # pool exhaustion is reported and changes nothing
    kv, _ = kv_pair(model, TINY, num_pages=2, max_seqs=2, max_pages_per_seq=32)
    kv.add_seq(0, 32)
    with pytest.raises(L.LaserError) as e:
        L.laser_decode_step(model, kv, [0], torch.zeros(1, dtype=torch.int32, device="cuda"),
                            torch.zeros(1, dtype=torch.int32, device="cuda"), torch.zeros(1, device="cuda"))
    assert e.value.code == L.ERR_OUT_OF_PAGES and kv.seq_len(0) == 32 and kv.page_table(0) == [0, 1]


def test_tiny_batched_decode_fused_attention_merge():
    # One-row attention groups merged by their last workgroup inside the attention kernel
    # (laser_model_set_attn_merge), batch 4 at 15-700 positions (1 to several splits each).
    require_gpu()
    V = TINY.vocab
    model, orc, _ = make_pair(TINY, max_rows=16, max_positions=1024)
    model.set_attn_merge(True, 4)
    kv, opool = kv_pair(model, TINY, num_pages=200, max_seqs=4, max_pages_per_seq=64)
    lens = [15, 130, 433, 700]
    states = []
    for s, n in enumerate(lens):
        K0, V0 = synth.make_prefill_kv(TINY, n, 80 + s)
        kv.add_seq(s, n)
        opool.add_seq(s, n)
        kv.import_kv(s, K0.cuda(), V0.cuda())
        states.append(SeqState.from_prefill(TINY, K0.numpy(), V0.numpy(), 1024))
    toks = [int(t) for t in synth.make_tokens(len(lens), V, 3040)]
    seqs = list(range(len(lens)))
    B = len(seqs)
    d_tok = torch.zeros(B, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(B, dtype=torch.int32, device="cuda")
    d_p = torch.zeros(B, device="cuda")
    d_logits = torch.zeros(B, V, device="cuda")
    for step in range(3):
        d_tok.copy_(torch.tensor(toks, dtype=torch.int32))
        L.laser_decode_step(model, kv, seqs, d_tok, d_next, d_p, d_logits)
        torch.cuda.synchronize()
        for b in seqs:
            opool.append(b, 1)
            ref = orc.decode_token(states[b], toks[b])
            compare_logits(d_logits[b].cpu().numpy(), ref, f"fused merge step {step} seq {b}")
            check_token(d_next[b].item(), ref, f"fused merge step {step} seq {b}")
            check_prob(d_p[b].item(), lm_stats(ref)[1], f"fused merge step {step} seq {b}")
            toks[b] = lm_stats(ref)[0]
            assert kv.page_table(b) == opool.tables[b]
