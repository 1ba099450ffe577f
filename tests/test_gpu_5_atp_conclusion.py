"""Device-side ATP cue detection and the forced conclusion (Section 3.1, Algorithm 1).

* laser_atp_match against the oracle's set membership, bit for bit, on tokens in and out
  of the vocabulary, and in place (flags written over the tokens);
* during greedy decoding of the tiny decoder, the flag of every generated token equals the
  oracle's membership of that token;
* after an exit, the closing delimiter and an answer prompt are appended with laser_prefill
  and the conclusion is decoded greedily: logits, tokens and max-probabilities against the
  oracle fed the same tokens, page tables against the oracle page model.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import check_prob, check_token, compare_logits, kv_pair, make_pair, require_gpu
from oracle import atp as A
from oracle.transformer import SeqState, lm_stats
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import TINY

pytestmark = pytest.mark.gpu


def test_atp_match_bitwise():
    require_gpu()
    rng = np.random.default_rng(3)
    for vocab in (1, 33, 2048, 152064):
        cues = rng.integers(0, vocab, size=min(vocab, 97)).tolist()
        words = torch.tensor(L.laser_atp_bitmap(cues, vocab).view(np.int32), device="cuda")
        toks = rng.integers(-40, vocab + 40, size=1000).astype(np.int32)
        toks[:len(cues)] = cues  # members for sure
        d_tok = torch.tensor(toks, device="cuda")
        d_flags = torch.full_like(d_tok, -7)
        L.laser_atp_match(d_tok, words, vocab, d_flags)
        torch.cuda.synchronize()
        assert d_flags.cpu().tolist() == A.cue_flags(toks.tolist(), cues, vocab), f"vocab {vocab}"
        L.laser_atp_match(d_tok, words, vocab, d_tok)  # in place
        torch.cuda.synchronize()
        assert d_tok.cpu().tolist() == A.cue_flags(toks.tolist(), cues, vocab)
    with pytest.raises(L.LaserError):
        L.laser_atp_match(d_tok, words, vocab, d_flags, n=0)


def test_cues_during_decode_and_forced_conclusion():
    require_gpu()
    V = TINY.vocab
    model, orc, _ = make_pair(TINY, max_rows=16, max_positions=512)
    kv, opool = kv_pair(model, TINY, num_pages=32, max_seqs=2, max_pages_per_seq=32)
    n0 = 40
    K0, V0 = synth.make_prefill_kv(TINY, n0, 61)
    kv.add_seq(0, n0)
    opool.add_seq(0, n0)
    kv.import_kv(0, K0.cuda(), V0.cuda())
    st = SeqState.from_prefill(TINY, K0.numpy(), V0.numpy(), 512)
    # a quarter of the vocabulary are cues, so detections happen within a few steps
    cues = synth.make_tokens(V // 4, V, 3100).tolist()
    words = torch.tensor(L.laser_atp_bitmap(cues, V).view(np.int32), device="cuda")
    d_tok = synth.make_tokens(1, V, 3101).cuda()
    d_next = torch.empty(1, dtype=torch.int32, device="cuda")
    d_p = torch.empty(1, device="cuda")
    d_flag = torch.empty(1, dtype=torch.int32, device="cuda")
    hits = 0
    tok = int(d_tok[0].item())  # a seeded input; afterwards the oracle's greedy tokens (teacher forcing)
    for step in range(24):
        L.laser_decode_step(model, kv, [0], d_tok, d_next, d_p)
        L.laser_atp_match(d_next, words, V, d_flag)
        torch.cuda.synchronize()
        opool.append(0, 1)
        ref = orc.decode_token(st, tok)
        check_token(d_next[0].item(), ref, f"decode {step}")
        check_prob(d_p[0].item(), lm_stats(ref)[1], f"decode {step}")
        tok = lm_stats(ref)[0]
        flag = d_flag[0].item()
        if d_next[0].item() == tok:  # the device's flag is of the device's token
            assert flag == A.cue_flags([tok], cues, V)[0], f"step {step}"
            hits += flag
        d_tok.fill_(tok)
    assert 0 < hits < 24
    # exit: the closing delimiter and an answer prompt, then the conclusion
    forced = synth.make_tokens(3, V, 3102)
    d_last = torch.empty(V, device="cuda")
    seq_in = torch.cat([torch.tensor([tok]), forced]).to(torch.int32)  # the pending token, then the forced ones
    L.laser_prefill(model, kv, 0, seq_in.cuda(), d_last)
    torch.cuda.synchronize()
    opool.append(0, len(seq_in))
    for t in seq_in.tolist():
        ref = orc.decode_token(st, int(t))
    compare_logits(d_last.cpu().numpy(), ref, "conclusion prompt")
    assert kv.page_table(0) == opool.tables[0] and kv.seq_len(0) == st.length
    tok = int(lm_stats(ref)[0])
    d_tok[0] = tok
    check_token(int(np.argmax(d_last.cpu().numpy())), ref, "first conclusion token")
    for step in range(8):
        L.laser_decode_step(model, kv, [0], d_tok, d_next, d_p)
        torch.cuda.synchronize()
        opool.append(0, 1)
        ref = orc.decode_token(st, tok)
        check_token(d_next[0].item(), ref, f"conclusion {step}")
        check_prob(d_p[0].item(), lm_stats(ref)[1], f"conclusion {step}")
        tok = lm_stats(ref)[0]
        d_tok.fill_(tok)
    assert kv.page_table(0) == opool.tables[0]
