"""Matrix-core weight tiles: forwards that run on the MFMA path give bitwise the same results
with the tile-order weight copy as with the row-major tensors.

One model, two KV caches holding the same state; each forward runs once with tiles on
(cache A) and once with tiles off (cache B), and every output is compared bit for bit.
Covers fp32 weights with a K that is not a multiple of 32 (tiny: d_ffn 688), bf16 at 1.5B
(two row groups per workgroup) and 7B (four), batches of 6, probe chunks, mixed steps, the
matrix-core LM head (8B batch-8 mixed: 12 outputs) and prompt prefill.
"""
import pytest
import torch

from gpu_helpers import require_gpu
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import LLAMA_8B, QWEN_1P5B, QWEN_7B, TINY

pytestmark = pytest.mark.gpu
S, T = 8, 4


def _caches(model, shape, lens, extra=96):
    out = []
    for _ in range(2):
        pages = sum(n // 16 + 3 for n in lens) + len(lens) * ((extra + S + T) // 16 + 3) + 8
        kv = L.KVCache(model, pages, len(lens), (max(lens) + extra + 64) // 16 + 2, poison=True)
        for i, n in enumerate(lens):
            k0, v0 = synth.make_prefill_kv(shape, n, 70 + i, device="cuda")
            kv.add_seq(i, n)
            kv.import_kv(i, k0, v0)
        out.append(kv)
    torch.cuda.synchronize()
    return out


def _both(model, kvs, fn):
    res = []
    for on, kv in zip((True, False), kvs):
        model.set_tiles(on)
        res.append(fn(kv))
        torch.cuda.synchronize()
    model.set_tiles(True)
    for x, y in zip(res[0], res[1]):
        assert torch.equal(x, y)


def _decode(model, shape, seqs, tok):
    def fn(kv):
        B = len(seqs)
        nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
        p = torch.zeros(B, device="cuda")
        lg = torch.zeros(B, shape.vocab, device="cuda")
        L.laser_decode_step(model, kv, seqs, tok, nxt, p, lg)
        return nxt, p, lg
    return fn


def _probe(model, shape, seqs, suffix):
    def fn(kv):
        B = len(seqs)
        conf = torch.zeros(B, device="cuda")
        arg = torch.zeros(B * T, dtype=torch.int32, device="cuda")
        lg = torch.zeros(B * T, shape.vocab, device="cuda")
        L.laser_probe_confidence(model, kv, seqs, suffix, T, conf, arg, lg)
        return conf, arg, lg
    return fn


def _mixed(model, seqs, tok, probe_idx, suffix):
    def fn(kv):
        B = len(seqs)
        nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
        p = torch.zeros(B, device="cuda")
        conf = torch.zeros(len(probe_idx), device="cuda")
        arg = torch.zeros(len(probe_idx) * T, dtype=torch.int32, device="cuda")
        L.laser_step_mixed(model, kv, seqs, tok, nxt, p, probe_idx, suffix, T, conf, arg)
        return nxt, p, conf, arg
    return fn


def test_tiles_tiny_fp32():
    require_gpu()
    w = {k: v.cuda() for k, v in synth.make_weights(TINY).items()}
    model = L.Model(TINY, w, max_rows=64, max_positions=768, poison=True)
    lens = [31, 250, 16, 77, 100, 5]
    kvs = _caches(model, TINY, lens)
    seqs = list(range(6))
    tok = synth.make_tokens(6, TINY.vocab, 81).cuda()
    suffix = synth.make_suffix(S, TINY.vocab).cuda()
    _both(model, kvs, _decode(model, TINY, seqs, tok))                 # 6 rows
    _both(model, kvs, _probe(model, TINY, [1, 4], suffix))              # 16-row chunk
    _both(model, kvs, _mixed(model, seqs, tok, [0, 2, 5], suffix))      # 30 rows
    prompt = synth.make_tokens(64, TINY.vocab, 82).cuda()

    def pre(kv):
        lg = torch.zeros(TINY.vocab, device="cuda")
        L.laser_prefill(model, kv, 2, prompt, lg)  # 64 prompt rows appended to request 2
        return (lg,)
    _both(model, kvs, pre)


@pytest.mark.parametrize("shape,lens", [(QWEN_1P5B, [4096]), (QWEN_7B, [14336])])
def test_tiles_probe_chunk(shape, lens):
    require_gpu()
    w = synth.make_weights(shape, device="cuda")
    model = L.Model(shape, w, max_rows=16, max_positions=max(lens) + 256)
    kvs = _caches(model, shape, lens)
    suffix = synth.make_suffix(S, shape.vocab).cuda()
    _both(model, kvs, _probe(model, shape, [0], suffix))
    model.destroy()
    del kvs, w, model
    torch.cuda.empty_cache()


def test_tiles_8b_mixed_and_lm_head():
    require_gpu()
    w = synth.make_weights(LLAMA_8B, device="cuda")
    model = L.Model(LLAMA_8B, w, max_rows=64, max_positions=14400)
    lens = synth.make_ragged_lengths(8, 3000, 14000)
    kvs = _caches(model, LLAMA_8B, lens)
    seqs = list(range(8))
    tok = synth.make_tokens(8, LLAMA_8B.vocab, 83).cuda()
    suffix = synth.make_suffix(S, LLAMA_8B.vocab).cuda()
    _both(model, kvs, _mixed(model, seqs, tok, synth.make_mixed_schedule(8, 1)[0], suffix))
    _both(model, kvs, _decode(model, LLAMA_8B, seqs, tok))  # 8 rows: MFMA projections and LM head
    model.destroy()
    del kvs, w, model
    torch.cuda.empty_cache()
