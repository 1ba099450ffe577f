"""The attention split merge run inside the O-projection's launch (forced on: by default only
projections of at least 16 MiB of weights take it) against the separate merge kernel.

One model, two KV caches holding the same state; each decode step runs once with the merge in
the projection's launch (cache A) and once with the merge kernel (cache B).  The two combine
the split partials in different orders, so logits agree to float rounding carried through
the layers, greedy tokens agree wherever the top two logits are not within rounding of each
other, and the appended K/V agree to one rounding step of their largest values.  Steps of one and
of two requests, replayed graphs, and switching back and forth on one model (the merge
counters keep counting across forwards that do not use them).  Oracle parity of the default
path is covered by the end-to-end tests.  Shapes: tiny (fp32, head dim 64), 1.5B (3-wave
projection workgroups, one round of partials for 96 splits), 7B (4 waves, up to 112 splits,
GQA group 7), 8B (group 4; the default takes this path there too).
"""
import numpy as np
import pytest
import torch

from gpu_helpers import export_seq, require_gpu
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import LLAMA_8B, QWEN_1P5B, QWEN_7B, TINY

pytestmark = pytest.mark.gpu


def _caches(model, shape, lens, steps):
    out = []
    for _ in range(2):
        pages = sum(n // 16 + 3 for n in lens) + len(lens) * (steps // 16 + 2) + 8
        kv = L.KVCache(model, pages, len(lens), (max(lens) + steps + 64) // 16 + 2, poison=True)
        for i, n in enumerate(lens):
            k0, v0 = synth.make_prefill_kv(shape, n, 90 + i, device="cuda")
            kv.add_seq(i, n)
            kv.import_kv(i, k0, v0)
        out.append(kv)
    torch.cuda.synchronize()
    return out


def _step(model, shape, kv, seqs, tok, on):
    model.set_oproj_merge(2 if on else 0)
    B = len(seqs)
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    p = torch.zeros(B, device="cuda")
    lg = torch.zeros(B, shape.vocab, device="cuda")
    L.laser_decode_step(model, kv, seqs, tok, nxt, p, lg)
    torch.cuda.synchronize()
    return nxt, p, lg


def _run(shape, lens, seq_sets, steps, tol):
    require_gpu()
    w = synth.make_weights(shape, device="cuda")
    model = L.Model(shape, w, max_rows=16, max_positions=max(lens) + steps * len(seq_sets) + 128, poison=True)
    kvs = _caches(model, shape, lens, steps * len(seq_sets))
    worst = 0.0
    for it in range(steps):
        for si, seqs in enumerate(seq_sets):
            tok = synth.make_tokens(len(seqs), shape.vocab, 500 + 7 * it + si).cuda()
            a = _step(model, shape, kvs[0], seqs, tok, True)
            b = _step(model, shape, kvs[1], seqs, tok, False)
            what = f"{shape.name} step {it} rows {seqs}"
            assert torch.isfinite(a[2]).all(), f"{what}: non-finite logits with the merge in the projection"
            d = (a[2] - b[2]).abs().max().item()
            worst = max(worst, d)
            assert d <= tol, f"{what}: logits differ by {d:.3g} (tolerance {tol})"
            assert torch.allclose(a[1], b[1], rtol=1e-4, atol=1e-6), f"{what}: max-prob"
            top2 = b[2].topk(2, dim=1).values
            clear = (top2[:, 0] - top2[:, 1]) > 4 * tol
            assert torch.equal(a[0][clear], b[0][clear]), f"{what}: greedy tokens"
    for s in sorted({x for ss in seq_sets for x in ss}):
        ka, va = export_seq(kvs[0], shape, s)
        kb, vb = export_seq(kvs[1], shape, s)
        # against the tensor's scale: one rounding step of the largest stored values (an element
        # may sit at a near-cancellation of the rotation, where relative error means nothing)
        step = 2.0 ** -7 if shape.dtype == "bf16" else 1e-5
        for x, y, n in ((ka, kb, "K"), (va, vb, "V")):
            dmax, scale = float(np.max(np.abs(x - y))), float(np.max(np.abs(y)))
            assert dmax <= step * scale, f"{shape.name}: {n} of request {s} differs by {dmax:.3g} (scale {scale:.3g})"
    print(f"{shape.name}: largest logit difference {worst:.3g} over {steps * len(seq_sets)} steps")
    model.set_oproj_merge(1)
    model.destroy()


def test_oproj_merge_tiny_fp32():
    _run(TINY, [700, 250, 40], [[0], [0, 1], [2], [1, 2]], 3, 1e-4)


def test_oproj_merge_1p5b():
    _run(QWEN_1P5B, [14336, 4093], [[0], [0, 1]], 3, 2e-3)


def test_oproj_merge_7b():
    # request 2 (24 positions) fits one attention workgroup, whose output needs no merge: its
    # merge workgroups only count their arrival, beside request 0's 112 splits
    _run(QWEN_7B, [14336, 3000, 24], [[0], [1, 0], [2, 0]], 3, 2e-3)


def test_oproj_merge_8b():
    _run(LLAMA_8B, [6000, 1500], [[0], [0, 1]], 2, 2e-3)
