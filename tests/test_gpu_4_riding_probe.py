"""A probe that rides along with decode steps on a fork of the request.

At an ATP each probing request is forked (full pages shared, the partial last page copied);
the following forwards carry, beside every request's decode row, a few of the fork's suffix
rows and then its fed-back trial rows (laser_forward spans).  Checked against the oracle:

Cases: tiny at 1, 3 and 8 probe rows per forward; 1.5B bf16 at 8 (the benchmark's setting:
all suffix rows in one forward beside the decode row, then the trial rows one per forward).

* every decode row equals plain decoding of the request (the fork's rows never touch it);
* the confidence and trial tokens equal the oracle's probe of the request's state at the
  ATP (Section 3.1): with the trial rows fed back on the device (the benchmark's way; the
  confidence compared whenever the trial tokens agree) and teacher-forced with the oracle's
  trial tokens (every trial's max-probability and the confidence compared);
* decode rows take the oracle's greedy tokens as inputs (teacher forcing);
* page tables (request, fork, and the pool after the fork is freed) equal the oracle page
  model's, bit for bit.
"""
import pytest
import torch

from gpu_helpers import check_prob, check_token, kv_pair, make_pair, require_gpu
from oracle.transformer import SeqState, lm_stats
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import QWEN_1P5B, TINY

pytestmark = pytest.mark.gpu

S, T = 8, 4


def riding_probe_run(shape, model, orc, kv, opool, states, seqs, probing, forks, per_step, toks, suffix, tag,
                     forced=False):
    """Runs decode steps for `seqs` (inputs: the oracle's greedy tokens) while requests
    `probing` (forked into `forks`) carry their probe rows, per_step rows per forward.  The
    trial rows read t_j as the device wrote it (forced=False: the benchmark's feedback, the
    confidence compared whenever every trial token agrees) or the oracle's t_j (forced=True:
    teacher forcing, every p_j and the confidence compared).  Returns (forwards, the next
    input tokens)."""
    V = shape.vocab
    B, P = len(seqs), len(probing)
    d_tok = torch.tensor(toks, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(B, dtype=torch.int32, device="cuda")
    d_p = torch.zeros(B, device="cuda")
    d_suffix = torch.tensor(suffix, dtype=torch.int32, device="cuda")
    d_arg = torch.zeros(P * T, dtype=torch.int32, device="cuda")
    d_pp = torch.zeros(P * T, device="cuda")
    d_conf = torch.zeros(P, device="cuda")
    res = {b: orc.probe(states[b], suffix, T) for b in probing}  # the oracle's probe at the ATP
    d_forced = torch.tensor([t for b in probing for t in res[b].tokens], dtype=torch.int32, device="cuda")
    for b, f in zip(probing, forks):
        kv.fork(b, f)
        opool.fork(b, f)
        assert kv.page_table(f) == opool.tables[f], f"{tag}: fork table"
    toks = list(toks)
    done_s, done_t, n_fwd = 0, 0, 0
    while done_t < T - 1 or done_s < S:
        spans = [L.span(b, 1, 0, i, out=(0, i)) for i, b in enumerate(seqs)]
        if done_s < S:
            k = min(per_step, S - done_s)
            last = done_s + k == S
            for i, f in enumerate(forks):
                spans.append(L.span(f, k, 1, done_s, out=(1, i * T) if last else None))
            tok1, done_s = d_suffix, done_s + k
            adv = k
        else:
            done_t += 1
            for i, f in enumerate(forks):  # trial j = done_t reads t_j, writes t_{j+1}
                spans.append(L.span(f, 1, 1, i * T + done_t - 1, out=(1, i * T + done_t)))
            tok1, adv = (d_forced if forced else d_arg), 1
        L.laser_forward(model, kv, spans, d_tok, tok1, d_next, d_p, d_arg, d_pp)
        torch.cuda.synchronize()
        n_fwd += 1
        for i, b in enumerate(seqs):
            opool.append(b, 1)
            ref = orc.decode_token(states[b], toks[i])
            check_token(d_next[i].item(), ref, f"{tag}: decode seq {b} forward {n_fwd}")
            check_prob(d_p[i].item(), lm_stats(ref)[1], f"{tag}: decode seq {b} forward {n_fwd}")
            assert kv.page_table(b) == opool.tables[b]
            toks[i] = lm_stats(ref)[0]
        for f in forks:
            opool.append(f, adv)
            assert kv.page_table(f) == opool.tables[f], f"{tag}: fork table after forward {n_fwd}"
        d_tok.copy_(torch.tensor(toks, dtype=torch.int32))
    L.laser_confidence(model, d_pp, T, P, d_conf)
    torch.cuda.synchronize()
    pp = d_pp.cpu().numpy()
    for i, b in enumerate(probing):
        r = res[b]
        got = [int(x) for x in d_arg[i * T:(i + 1) * T].cpu().numpy()]
        print(f"{tag}: probe seq {b}: conf gpu {d_conf[i].item():.6g} oracle {r.confidence:.6g}", flush=True)
        for j in range(T):
            if r.margins[j] > 1e-2:
                assert got[j] == r.tokens[j], f"{tag}: trial {j} token {got[j]} vs {r.tokens[j]}"
        if forced or got == r.tokens:
            for j in range(T):
                check_prob(pp[i * T + j], r.pmax[j], f"{tag}: probe seq {b} trial {j}")
            check_prob(d_conf[i].item(), r.confidence, f"{tag}: probe seq {b} confidence")
        else:  # device feedback: a trial token may differ only where the oracle's top-2 margin is tiny
            assert any(m <= 1e-2 for m in r.margins), f"{tag}: trial tokens {got} vs {r.tokens}"
    for f in forks:
        kv.free_seq(f)
        opool.free_seq(f)
    for b in seqs:
        assert kv.page_table(b) == opool.tables[b] and kv.seq_len(b) == states[b].length
    return n_fwd, toks


def test_riding_probe_tiny():
    require_gpu()
    model, orc, _ = make_pair(TINY, max_rows=32, max_positions=1024)
    kv, opool = kv_pair(model, TINY, num_pages=160, max_seqs=8, max_pages_per_seq=64)
    lens = [37, 48, 250]  # a partial last page, a page boundary, a longer context
    states = []
    for s, n in enumerate(lens):
        K0, V0 = synth.make_prefill_kv(TINY, n, 30 + s)
        kv.add_seq(s, n)
        opool.add_seq(s, n)
        kv.import_kv(s, K0.cuda(), V0.cuda())
        states.append(SeqState.from_prefill(TINY, K0.numpy(), V0.numpy(), 1024))
    toks = [int(t) for t in synth.make_tokens(len(lens), TINY.vocab, 3010)]
    suffix = [int(t) for t in synth.make_suffix(S, TINY.vocab)]
    for per_step, forced in ((1, False), (3, False), (8, False), (3, True), (8, True)):
        n, toks = riding_probe_run(TINY, model, orc, kv, opool, states, [0, 1, 2], [0, 1], [5, 6], per_step,
                                   toks, suffix, f"tiny per_step={per_step} forced={forced}", forced=forced)
        assert n == -(-S // per_step) + T - 1


def test_riding_probe_1p5b_bf16():
    require_gpu()
    shape = QWEN_1P5B
    model, orc, _ = make_pair(shape, max_rows=16, max_positions=4352, weights_on_device=True, cache_oracle=True)
    kv, opool = kv_pair(model, shape, num_pages=600, max_seqs=4, max_pages_per_seq=272)
    n0 = 4093  # partial last page: the fork copies it
    K0, V0 = synth.make_prefill_kv(shape, n0, 0, device="cuda")
    kv.add_seq(0, n0)
    opool.add_seq(0, n0)
    kv.import_kv(0, K0, V0)
    states = [SeqState.from_prefill(shape, synth.to_numpy(K0), synth.to_numpy(V0), 4352)]
    del K0, V0
    toks = [int(synth.make_tokens(1, shape.vocab, 3011)[0])]
    suffix = [int(t) for t in synth.make_suffix(S, shape.vocab)]
    # the benchmark's setting: the 8 suffix rows ride in one forward (9 rows: the MFMA path)
    riding_probe_run(shape, model, orc, kv, opool, states, [0], [0], [2], 8, toks, suffix, "1.5B")


def test_riding_probes_staggered_tiny():
    # A new probe starts on every forward (rotating over the requests, so one request has
    # several forks in flight); each probe's suffix chunk rides in its first forward and its
    # trial rows in the next T-1, all beside the decode rows (the batch serving pattern).
    require_gpu()
    model, orc, _ = make_pair(TINY, max_rows=32, max_positions=1024)
    P = T  # probe slots: one probe starts per forward and lives T forwards
    kv, opool = kv_pair(model, TINY, num_pages=200, max_seqs=3 + P, max_pages_per_seq=64)
    lens = [30, 64, 131]
    states = []
    for s, n in enumerate(lens):
        K0, V0 = synth.make_prefill_kv(TINY, n, 40 + s)
        kv.add_seq(s, n)
        opool.add_seq(s, n)
        kv.import_kv(s, K0.cuda(), V0.cuda())
        states.append(SeqState.from_prefill(TINY, K0.numpy(), V0.numpy(), 1024))
    seqs = [0, 1, 2]
    suffix = [int(t) for t in synth.make_suffix(S, TINY.vocab)]
    toks = [int(t) for t in synth.make_tokens(3, TINY.vocab, 3011)]
    d_tok = torch.tensor(toks, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(3, dtype=torch.int32, device="cuda")
    d_p = torch.zeros(3, device="cuda")
    # inputs: the suffix, then each slot's trial inputs (the oracle's t_1..t_{T-1}: teacher forcing)
    tokbuf = torch.zeros(S + P * T, dtype=torch.int32, device="cuda")
    tokbuf[:S] = torch.tensor(suffix, dtype=torch.int32)
    outbuf = torch.zeros(P * T, dtype=torch.int32, device="cuda")
    pbuf = torch.zeros(P * T, device="cuda")
    d_conf = torch.zeros(1, device="cuda")
    free, inflight, checked = list(range(P)), [], 0
    n_fwd = 10
    for fwd in range(n_fwd + T - 1):
        spans = [L.span(b, 1, 0, i, out=(0, i)) for i, b in enumerate(seqs)]
        fork_rows = []  # (fork slot, rows) in span order: pages are taken in that order
        for pr in inflight:  # [slot, request, trials done, the oracle's probe at the fork]
            f, j = pr[0], pr[2] + 1
            spans.append(L.span(3 + f, 1, 1, S + f * T + j - 1, out=(1, f * T + j)))
            fork_rows.append((3 + f, 1))
            pr[2] = j
        if fwd < n_fwd:
            b = seqs[fwd % 3]
            f = free.pop()
            res = orc.probe(states[b], suffix, T)
            tokbuf[S + f * T:S + (f + 1) * T] = torch.tensor(res.tokens, dtype=torch.int32)
            kv.fork(b, 3 + f)
            opool.fork(b, 3 + f)
            assert kv.page_table(3 + f) == opool.tables[3 + f], f"fork table at forward {fwd}"
            spans.append(L.span(3 + f, S, 1, 0, out=(1, f * T)))
            fork_rows.append((3 + f, S))
            inflight.append([f, b, 0, res])
        L.laser_forward(model, kv, spans, d_tok, tokbuf, d_next, d_p, outbuf, pbuf)
        torch.cuda.synchronize()
        for b in seqs:
            opool.append(b, 1)
        for f, n in fork_rows:
            opool.append(f, n)
        for i, b in enumerate(seqs):
            ref = orc.decode_token(states[b], toks[i])
            check_token(d_next[i].item(), ref, f"staggered: decode seq {b} forward {fwd}")
            check_prob(d_p[i].item(), lm_stats(ref)[1], f"staggered: decode seq {b} forward {fwd}")
            assert kv.page_table(b) == opool.tables[b]
            toks[i] = lm_stats(ref)[0]
        for pr in inflight:
            assert kv.page_table(3 + pr[0]) == opool.tables[3 + pr[0]], f"fork table after forward {fwd}"
        d_tok.copy_(torch.tensor(toks, dtype=torch.int32))
        for pr in [p for p in inflight if p[2] == T - 1]:
            f, b, res = pr[0], pr[1], pr[3]
            L.laser_confidence(model, pbuf[f * T:], T, 1, d_conf)
            torch.cuda.synchronize()
            got = [int(x) for x in outbuf[f * T:(f + 1) * T].cpu().numpy()]
            pp = pbuf[f * T:(f + 1) * T].cpu().numpy()
            for j in range(T):
                if res.margins[j] > 1e-2:
                    assert got[j] == res.tokens[j], f"probe of seq {b} (slot {f}) trial {j}"
                check_prob(pp[j], res.pmax[j], f"probe of seq {b} (slot {f}) trial {j}")
            check_prob(d_conf.item(), res.confidence, f"probe of seq {b} (slot {f})")
            kv.free_seq(3 + f)
            opool.free_seq(3 + f)
            free.append(f)
            inflight.remove(pr)
            checked += 1
    assert checked == n_fwd and not inflight
    for b in seqs:
        assert kv.page_table(b) == opool.tables[b] and kv.seq_len(b) == states[b].length


def test_fork_with_long_own_tail_tiny():
    # A fork that has decoded far past its fork point: its own pages outnumber what its own
    # row group may split into (the split count beside a shared-prefix group is bounded), so
    # the planner lengthens that group's page runs.  Then the request and the fork decode in
    # one forward: one group over their shared pages, one group each over its own pages,
    # partials merged per row.  Every decode row and page table is checked.
    require_gpu()
    model, orc, _ = make_pair(TINY, max_rows=16, max_positions=1024)
    kv, opool = kv_pair(model, TINY, num_pages=120, max_seqs=2, max_pages_per_seq=64)
    K0, V0 = synth.make_prefill_kv(TINY, 100, 50)
    kv.add_seq(0, 100)
    opool.add_seq(0, 100)
    kv.import_kv(0, K0.cuda(), V0.cuda())
    states = [SeqState.from_prefill(TINY, K0.numpy(), V0.numpy(), 1024)]
    kv.fork(0, 1)
    opool.fork(0, 1)
    states.append(states[0].copy())
    assert kv.page_table(1) == opool.tables[1]
    toks = [int(t) for t in synth.make_tokens(2, TINY.vocab, 3012)]

    def steps(seqs, n, tag):
        B = len(seqs)
        d_tok = torch.tensor([toks[b] for b in seqs], dtype=torch.int32, device="cuda")
        d_next = torch.zeros(B, dtype=torch.int32, device="cuda")
        d_p = torch.zeros(B, device="cuda")
        for step in range(n):
            L.laser_decode_step(model, kv, seqs, d_tok, d_next, d_p)
            torch.cuda.synchronize()
            for i, b in enumerate(seqs):
                opool.append(b, 1)
                ref = orc.decode_token(states[b], toks[b])
                check_token(d_next[i].item(), ref, f"{tag} step {step} seq {b}")
                check_prob(d_p[i].item(), lm_stats(ref)[1])
                toks[b] = lm_stats(ref)[0]
                assert kv.page_table(b) == opool.tables[b], f"{tag} step {step}: page table of seq {b}"
            d_tok.copy_(torch.tensor([toks[b] for b in seqs], dtype=torch.int32))

    steps([1], 560, "fork alone")  # 35 own pages past the 6 shared ones
    steps([0, 1], 4, "request and fork")
    steps([1, 0], 2, "fork and request")
