"""The allocation-free decode step (laser_decode_step_static) against laser_decode_step.

Two caches with the same pre-filled K/V and the same input tokens: one advanced by
laser_decode_step (scratch in the model's workspace), the other by laser_decode_step_static
(scratch in the library's static device array).  Two calls in a row, the second with a
smaller batch (the array keeps the first call's contents, including its arrival counters'
state); each compared with the existing entry point's outputs to the parity bar: greedy
tokens exact, logits within 2e-2 and max-probabilities within 1e-3 (the same kernels run, so
the results are expected to be identical).  Contexts of 250-700 positions split each row's
attention over several workgroups, so the partials and the merge use the scratch.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import LOGIT_TOL, PROB_TOL, make_pair, require_gpu
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import TINY

pytestmark = pytest.mark.gpu


def test_static_scratch_decode_matches_decode_step():
    require_gpu()
    V = TINY.vocab
    model, _, _ = make_pair(TINY, max_rows=8, max_positions=1024)
    lens = [250, 433, 700, 512]
    kvs = []
    for _ in range(2):
        kv = L.KVCache(model, 200, 4, 64, poison=True)
        for s, n in enumerate(lens):
            K0, V0 = synth.make_prefill_kv(TINY, n, 70 + s)
            kv.add_seq(s, n)
            kv.import_kv(s, K0.cuda(), V0.cuda())
        kvs.append(kv)
    for call, seqs in enumerate(([0, 1, 2, 3], [2, 0])):  # the second call is smaller
        B = len(seqs)
        toks = synth.make_tokens(B, V, 3030 + call).cuda()
        outs = []
        for kv, fn in ((kvs[0], L.laser_decode_step), (kvs[1], L.laser_decode_step_static)):
            nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
            p = torch.zeros(B, device="cuda")
            lg = torch.zeros(B, V, device="cuda")
            fn(model, kv, seqs, toks, nxt, p, lg)
            torch.cuda.synchronize()
            outs.append((nxt.cpu().numpy(), p.cpu().numpy(), lg.cpu().numpy()))
        (t0, p0, l0), (t1, p1, l1) = outs
        assert np.array_equal(t0, t1), f"call {call}: tokens {t0} vs {t1}"
        err = float(np.max(np.abs(l0 - l1)))
        assert err <= LOGIT_TOL, f"call {call}: logits differ by {err}"
        assert float(np.max(np.abs(p0 - p1))) <= PROB_TOL
        print(f"call {call} (batch {B}): max logit difference {err:.3g}", flush=True)
        for s in seqs:
            assert kvs[0].page_table(s) == kvs[1].page_table(s) and kvs[0].seq_len(s) == kvs[1].seq_len(s)
    for kv in kvs:
        kv.destroy()
    model.destroy()


def test_static_scratch_size_limit():
    """A batch whose scratch exceeds the static array is refused before anything changes; a
    batch just under the limit runs and matches laser_decode_step.  (A 1-layer bf16 decoder
    with 64 query / 8 KV heads of 128: 4 MiB of attention partials per row.)"""
    require_gpu()
    from paper_2606_31580_amd.configs import ModelShape

    wide = ModelShape("wide-heads-1L", 1, 512, 64, 8, 128, 512, 1024, False, False, "bf16", 1.0e4, 1.0e-6)
    V = wide.vocab
    model, _, _ = make_pair(wide, max_rows=8, max_positions=256)
    kvs = []
    for _ in range(2):
        kv = L.KVCache(model, 64, 8, 16, poison=True)
        for s in range(8):
            K0, V0 = synth.make_prefill_kv(wide, 20 + s, 90 + s, device="cuda")
            kv.add_seq(s, 20 + s)
            kv.import_kv(s, K0, V0)
        kvs.append(kv)
    toks = synth.make_tokens(8, V, 3050).cuda()
    nxt = torch.zeros(8, dtype=torch.int32, device="cuda")
    p = torch.zeros(8, device="cuda")
    with pytest.raises(L.LaserError) as e:
        L.laser_decode_step_static(model, kvs[1], list(range(8)), toks, nxt, p)
    assert e.value.code == L.ERR_UNSUPPORTED
    assert all(kvs[1].seq_len(s) == 20 + s for s in range(8))
    seqs = list(range(7))  # 28 MiB of partials: within the array
    outs = []
    for kv, fn in ((kvs[0], L.laser_decode_step), (kvs[1], L.laser_decode_step_static)):
        n7 = torch.zeros(7, dtype=torch.int32, device="cuda")
        p7 = torch.zeros(7, device="cuda")
        lg = torch.zeros(7, V, device="cuda")
        fn(model, kv, seqs, toks[:7], n7, p7, lg)
        torch.cuda.synchronize()
        outs.append((n7.cpu().numpy(), p7.cpu().numpy(), lg.cpu().numpy()))
    (t0, p0, l0), (t1, p1, l1) = outs
    assert np.array_equal(t0, t1)
    assert float(np.max(np.abs(l0 - l1))) <= LOGIT_TOL and float(np.max(np.abs(p0 - p1))) <= PROB_TOL
    for kv in kvs:
        kv.destroy()
    model.destroy()
