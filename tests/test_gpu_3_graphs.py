"""Graph replay of forwards: bitwise equal to launching the same kernels one by one.

Two KV caches hold the same state; every decode step, probe and mixed step runs once with
graphs on (cache A) and once with graphs off (cache B), with host synchronisation and
eager work between the replays, and every replay is compared bitwise.  Output buffers are
swapped between calls (they travel in the plan, not in the captured kernel arguments), and
the contexts grow across page and attention-grid boundaries so that several graph keys
are captured and reused.
"""
import pytest
import torch

from gpu_helpers import require_gpu
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import TINY

pytestmark = pytest.mark.gpu


def _state(model, lens):
    kv = L.KVCache(model, 96, 4, 48, poison=True)
    for i, n in enumerate(lens):
        k0, v0 = synth.make_prefill_kv(TINY, n, 50 + i)
        kv.add_seq(i, n)
        kv.import_kv(i, k0.cuda(), v0.cuda())
    return kv


def test_graph_replay_matches_eager():
    require_gpu()
    w = {k: v.cuda() for k, v in synth.make_weights(TINY).items()}
    model = L.Model(TINY, w, max_rows=32, max_positions=768, poison=True)
    lens = [31, 250]
    kv_a, kv_b = _state(model, lens), _state(model, lens)
    B, V, S, T = len(lens), TINY.vocab, 8, 4
    seqs = list(range(B))
    tok = synth.make_tokens(B, V, 77).cuda()
    bufs = [(torch.zeros(B, dtype=torch.int32, device="cuda"), torch.zeros(B, device="cuda"),
             torch.zeros(B, V, device="cuda")) for _ in range(2)]
    ref = (torch.zeros(B, dtype=torch.int32, device="cuda"), torch.zeros(B, device="cuda"),
           torch.zeros(B, V, device="cuda"))
    suffix = synth.make_suffix(S, V).cuda()
    tok_a, tok_b = tok.clone(), tok.clone()
    n_steps = 40
    for step in range(n_steps):
        nxt, p, lg = bufs[step % 2]
        model.set_graphs(True)
        L.laser_decode_step(model, kv_a, seqs, tok_a, nxt, p, lg)
        model.set_graphs(False)
        L.laser_decode_step(model, kv_b, seqs, tok_b, ref[0], ref[1], ref[2])
        torch.cuda.synchronize()
        assert torch.equal(nxt, ref[0]) and torch.equal(p, ref[1]) and torch.equal(lg, ref[2]), f"step {step}"
        tok_a.copy_(nxt)
        tok_b.copy_(ref[0])
        if step % 10 == 9:
            out = []
            for on, kv in ((True, kv_a), (False, kv_b)):
                model.set_graphs(on)
                conf = torch.zeros(B, device="cuda")
                arg = torch.zeros(B * T, dtype=torch.int32, device="cuda")
                L.laser_probe_confidence(model, kv, seqs, suffix, T, conf, arg)
                torch.cuda.synchronize()
                out.append((conf, arg))
            assert torch.equal(out[0][0], out[1][0]) and torch.equal(out[0][1], out[1][1]), f"probe at {step}"
        if step % 10 == 4:
            out = []
            for on, kv in ((True, kv_a), (False, kv_b)):
                model.set_graphs(on)
                t_in = tok_a if on else tok_b
                nx = torch.zeros(B, dtype=torch.int32, device="cuda")
                pm = torch.zeros(B, device="cuda")
                conf = torch.zeros(1, device="cuda")
                arg = torch.zeros(T, dtype=torch.int32, device="cuda")
                L.laser_step_mixed(model, kv, seqs, t_in, nx, pm, [1], suffix, T, conf, arg)
                torch.cuda.synchronize()
                out.append((nx, pm, conf, arg))
            for x, y in zip(out[0], out[1]):
                assert torch.equal(x, y), f"mixed at {step}"
            tok_a.copy_(out[0][0])
            tok_b.copy_(out[1][0])
    assert kv_a.seq_len(0) == kv_b.seq_len(0) == lens[0] + n_steps + 4
    assert kv_a.page_table(1) == kv_b.page_table(1)
    # timing forces one-by-one launches and still gives the same tokens
    model.set_graphs(True)
    model.timing_enable(L.K_GATEUP, True)
    nxt, p, lg = bufs[0]
    L.laser_decode_step(model, kv_a, seqs, tok_a, nxt, p, lg)
    model.set_graphs(False)
    L.laser_decode_step(model, kv_b, seqs, tok_b, ref[0], ref[1], ref[2])
    torch.cuda.synchronize()
    ms, n = model.timing_read(L.K_GATEUP)
    model.timing_enable(L.K_GATEUP, False)
    assert n == 2 * TINY.n_layers and ms > 0  # both decodes ran inside the timing session
    assert torch.equal(lg, ref[2])


def test_forward_next_tokens_in_place():
    """laser_forward whose output tokens overwrite its input tokens at the same indices (the
    forward reads every input before it writes an output) against separate output buffers."""
    require_gpu()
    w = {k: v.cuda() for k, v in synth.make_weights(TINY).items()}
    model = L.Model(TINY, w, max_rows=32, max_positions=768, poison=True)
    lens = [31, 250, 77]
    kv_a, kv_b = _state(model, lens), _state(model, lens)
    B = len(lens)
    tok_a = synth.make_tokens(B, TINY.vocab, 78).cuda()
    tok_b, nxt_b = tok_a.clone(), torch.zeros(B, dtype=torch.int32, device="cuda")
    p_a, p_b = torch.zeros(B, device="cuda"), torch.zeros(B, device="cuda")
    spans = [L.span(b, 1, 0, b, out=(0, b)) for b in range(B)]
    for step in range(24):
        L.laser_forward(model, kv_a, spans, tok_a, None, tok_a, p_a)
        L.laser_forward(model, kv_b, spans, tok_b, None, nxt_b, p_b)
        torch.cuda.synchronize()
        assert torch.equal(tok_a, nxt_b) and torch.equal(p_a, p_b), f"step {step}"
        tok_b.copy_(nxt_b)
    kv_a.destroy()
    kv_b.destroy()
    model.destroy()


def test_graph_eviction_matches_eager():
    """More forward shapes than the captured-graph cache holds (16): evicted graphs are
    released while later forwards are queued, and every replay still matches the eager
    launch of the same forward bitwise."""
    require_gpu()
    w = {k: v.cuda() for k, v in synth.make_weights(TINY).items()}
    model = L.Model(TINY, w, max_rows=32, max_positions=768, poison=True)
    n = 20
    lens = [10 + 7 * i for i in range(n)]

    def caches():
        kv = L.KVCache(model, 200, n, 48, poison=True)
        for i, ln in enumerate(lens):
            k0, v0 = synth.make_prefill_kv(TINY, ln, 90 + i)
            kv.add_seq(i, ln)
            kv.import_kv(i, k0.cuda(), v0.cuda())
        return kv
    kv_a, kv_b = caches(), caches()
    tok = synth.make_tokens(n, TINY.vocab, 79).cuda()
    for rnd in range(3):
        for b in range(1, n + 1):  # b rows: a new graph key per batch size
            seqs = list(range(b))
            outs = []
            for on, kv in ((True, kv_a), (False, kv_b)):
                model.set_graphs(on)
                nxt = torch.zeros(b, dtype=torch.int32, device="cuda")
                p = torch.zeros(b, device="cuda")
                L.laser_decode_step(model, kv, seqs, tok[:b], nxt, p)
                outs.append((nxt, p))
            torch.cuda.synchronize()
            assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1]), f"round {rnd}, {b} rows"
    model.set_graphs(True)
    captures, cached = model.graph_stats()
    assert captures > 16 and cached <= 16
    kv_a.destroy()
    kv_b.destroy()
    model.destroy()
