"""The fp8 (OCP E4M3) KV-cache variant against the oracle that rounds K/V the same way.

State injection at full size, as in test_gpu_2_full_shapes, with the KV cache in E4M3:
* pre-filled K/V survive import and export bit for bit;
* decode logits, greedy tokens, max-probabilities and the probe's confidence and trial
  tokens match the oracle (which stores every appended key and value rounded to E4M3,
  ties to even, saturating at 448) within the usual tolerances;
* the appended keys and values equal the oracle's rounded ones, allowing one E4M3 step
  where the fp32 and fp64 pre-rounding values fall on different sides of a rounding
  boundary;
* the 8B batch-8 mixed step (the configuration where KV bytes matter most).
"""
import numpy as np
import pytest
import torch

from gpu_helpers import check_prob, check_token, require_gpu
from oracle.numerics import round_fp8_e4m3
from oracle.transformer import lm_stats
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import LLAMA_8B_FP8KV, QWEN_1P5B_FP8KV, QWEN_7B_FP8KV
from test_gpu_2_full_shapes import S, T, Setup, log

pytestmark = pytest.mark.gpu


def _export(st, seq):
    n = st.kv.seq_len(seq)
    sh = st.shape
    K = torch.empty((sh.n_layers, n, sh.n_kv_heads, sh.head_dim), dtype=torch.float8_e4m3fn, device="cuda")
    V = torch.empty_like(K)
    st.kv.export_kv(seq, K, V)
    torch.cuda.synchronize()
    return K, V


def _fp8_step(x):
    # spacing of the E4M3 grid at |x|
    a = np.maximum(np.abs(x), 2.0 ** -6)
    return np.ldexp(1.0, np.floor(np.log2(a)).astype(np.int64) - 3)


def test_qwen1p5b_fp8kv_state_injection():
    require_gpu()
    n0 = 4096
    st = Setup(QWEN_1P5B_FP8KV, [n0])
    k0, v0 = synth.make_prefill_kv(QWEN_1P5B_FP8KV, n0, 0, device="cuda")
    K, V = _export(st, 0)
    assert torch.equal(K.view(torch.uint8), k0.view(torch.uint8)) and torch.equal(V.view(torch.uint8), v0.view(torch.uint8))
    del k0, v0, K, V
    st.decode(3)
    st.probe([0])
    K, V = _export(st, 0)
    k = synth.to_numpy(K)
    v = synth.to_numpy(V)
    from oracle.numerics import fp8_e4m3_bits_to_float
    kg, vg = fp8_e4m3_bits_to_float(k[:, n0:n0 + 3]), fp8_e4m3_bits_to_float(v[:, n0:n0 + 3])
    ko, vo = st.states[0].K[:, n0:n0 + 3], st.states[0].V[:, n0:n0 + 3]
    assert np.array_equal(round_fp8_e4m3(ko), ko) and np.array_equal(round_fp8_e4m3(vo), vo)  # oracle stores E4M3
    for g, o in ((kg, ko), (vg, vo)):
        diff = np.abs(g - o)
        assert np.all(diff <= _fp8_step(o) + 1e-12), float(diff.max())
        log(f"appended K/V: {int((diff > 0).sum())} of {diff.size} one step apart")
    st.release()


def test_qwen7b_fp8kv_b1_kv14336_state_injection():
    st = Setup(QWEN_7B_FP8KV, [14336])
    st.decode(1)
    st.probe([0])
    st.release()


def test_llama8b_fp8kv_b8_mixed_step_state_injection():
    lens = synth.make_ragged_lengths(8, 3000, 14000)
    st = Setup(LLAMA_8B_FP8KV, lens)
    probe_idx = synth.make_mixed_schedule(8, 1)[0]
    B = 8
    d_tok = torch.tensor(st.toks, dtype=torch.int32, device=st.dev)
    d_next = torch.zeros(B, dtype=torch.int32, device=st.dev)
    d_p = torch.zeros(B, device=st.dev)
    d_conf = torch.zeros(len(probe_idx), device=st.dev)
    d_arg = torch.zeros(len(probe_idx) * T, dtype=torch.int32, device=st.dev)
    L.laser_step_mixed(st.model, st.kv, st.seqs, d_tok, d_next, d_p, probe_idx, st.d_suffix, T, d_conf, d_arg)
    torch.cuda.synchronize()
    for b in st.seqs:
        st.opool.append(b, 1)
    for b in probe_idx:
        st.opool.append(b, S + T - 1)
    for b in st.seqs:
        ref = st.orc.decode_token(st.states[b], st.toks[b])
        check_token(d_next[b].item(), ref, f"mixed decode seq {b}")
        check_prob(d_p[b].item(), lm_stats(ref)[1])
    for b in probe_idx:
        st.opool.truncate(b, st.states[b].length)
    arg = d_arg.cpu().numpy().reshape(len(probe_idx), T)
    for i, b in enumerate(probe_idx):
        st.compare_probe(b, arg[i], d_conf[i].item())
    st.check_tables()
    st.release()
