"""Seeded synthetic inputs shared by the GPU path's tests/bench and the CPU oracle.

This module only draws random numbers (torch generators with fixed seeds) and
names tensors; it holds none of the method's arithmetic.  Weights follow the
random-init recipe: every matrix, embedding and bias ~N(0, 0.02) rounded to the
storage dtype (bf16 round-to-nearest-even, or fp32), norm gains 1.0.
Pre-filled KV entries ~N(0, 1) stand for an already-generated chain of thought
(post-RoPE keys), tokens are uniform over the vocabulary.

Seeds: weights 1000 + tensor index (fixed name order), pre-filled KV 2000 +
request index, prompt/first tokens/suffix 3000.., ragged lengths and the
mixed-step schedule 4000, serving-simulation traces 6000 and arrivals 7000.

Serving-simulation traces (the paper's per-sample profiles of trained models are not
available, so these stand in for them; shapes from the paper):
  * prompt length uniform in [50, 275] tokens (the p_min..p_max range of Section 4.3);
  * reasoning length uniform in [3000, 14000] tokens (the CoT lengths of Section 1), cut
    into chunks of lognormal length (median 900 tokens) at ATPs;
  * the trial answer settles early, as reasoning models overthink (Section 3.1): at chunk
    g - 1 with g geometric (p = 0.45), at most the last chunk; from there on it is the final
    answer (right with probability 0.85), before it right with probability 0.35;
  * confidences are polarised (Section 4.2's rationale for tanh): after settling, 85%
    are drawn from [0.95, 1) and the rest from [0.5, 0.95); before settling, 10% from
    [0.9, 1) and the rest from [0.2, 0.9);
  * conclusion length uniform in [100, 400] tokens; the answer without reasoning is
    right with probability 0.35.
Arrivals: exponential gaps at the given rate (Poisson), or phases of given rates and
durations (the 1 -> 5 -> 1 QPS burst of Section 5.1).
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np
import torch

from .configs import ModelShape

WEIGHT_STD = 0.02


def _tdtype(shape: ModelShape) -> torch.dtype:
    return torch.bfloat16 if shape.dtype == "bf16" else torch.float32


def _kv_tdtype(shape: ModelShape) -> torch.dtype:
    if shape.kv_storage == "fp8":
        return torch.float8_e4m3fn
    return _tdtype(shape)


def tensor_specs(shape: ModelShape) -> List[tuple]:
    """(name, dims, kind) in the fixed order that defines each tensor's seed.

    kind: "w" matrix/embedding/bias ~N(0, std); "g" norm gain = 1.
    """
    d, hd, F = shape.d_model, shape.head_dim, shape.d_ffn
    hq, hkv = shape.n_q_heads, shape.n_kv_heads
    specs = [("embed", (shape.vocab, d), "w")]
    for i in range(shape.n_layers):
        p = f"layers.{i}."
        specs += [
            (p + "attn_norm", (d,), "g"),
            (p + "wq", (hq * hd, d), "w"),
            (p + "wk", (hkv * hd, d), "w"),
            (p + "wv", (hkv * hd, d), "w"),
        ]
        if shape.qkv_bias:
            specs += [(p + "bq", (hq * hd,), "w"), (p + "bk", (hkv * hd,), "w"), (p + "bv", (hkv * hd,), "w")]
        specs += [
            (p + "wo", (d, hq * hd), "w"),
            (p + "mlp_norm", (d,), "g"),
            (p + "w_gate", (F, d), "w"),
            (p + "w_up", (F, d), "w"),
            (p + "w_down", (d, F), "w"),
        ]
    specs.append(("final_norm", (d,), "g"))
    if not shape.tied_embeddings:
        specs.append(("lm_head", (shape.vocab, d), "w"))
    return specs


def make_weights(shape: ModelShape, device="cpu", seed_base: int = 1000, std: float = WEIGHT_STD) -> Dict[str, torch.Tensor]:
    """Random-init weights in the storage dtype on `device` (tied models have no lm_head)."""
    out = {}
    dt = _tdtype(shape)
    for idx, (name, dims, kind) in enumerate(tensor_specs(shape)):
        if kind == "g":
            out[name] = torch.ones(dims, dtype=dt, device=device)
            continue
        g = torch.Generator(device=device)
        g.manual_seed(seed_base + idx)
        t = torch.randn(dims, generator=g, device=device, dtype=torch.float32)
        t.mul_(std)
        out[name] = t.to(dt)
    return out


def make_prefill_kv(shape: ModelShape, length: int, request: int, device="cpu", seed_base: int = 2000):
    """Pre-filled (K, V) for one request: two tensors [n_layers, length, n_kv_heads, head_dim], ~N(0,1),
    in the KV-cache storage type."""
    g = torch.Generator(device=device)
    g.manual_seed(seed_base + request)
    dims = (shape.n_layers, length, shape.n_kv_heads, shape.head_dim)
    k = torch.randn(dims, generator=g, device=device, dtype=torch.float32).to(_kv_tdtype(shape))
    v = torch.randn(dims, generator=g, device=device, dtype=torch.float32).to(_kv_tdtype(shape))
    return k, v


def make_tokens(n: int, vocab: int, seed: int) -> torch.Tensor:
    """n uniform token ids in [0, vocab) as int32 (CPU)."""
    g = torch.Generator()
    g.manual_seed(seed)
    return torch.randint(0, vocab, (n,), generator=g, dtype=torch.int64).to(torch.int32)


def make_suffix(S: int, vocab: int, seed: int = 3001) -> torch.Tensor:
    """The fixed answer-inducing suffix (S ids, shared by every request)."""
    return make_tokens(S, vocab, seed)


def make_ragged_lengths(batch: int, lo: int, hi: int, seed: int = 4000) -> List[int]:
    g = torch.Generator()
    g.manual_seed(seed)
    return [int(x) for x in torch.randint(lo, hi + 1, (batch,), generator=g)]


def make_mixed_schedule(batch: int, steps: int, seed: int = 4001) -> List[List[int]]:
    """For each step, a seeded random half of the requests that also run a probe chunk (sorted ids)."""
    g = torch.Generator()
    g.manual_seed(seed)
    out = []
    for _ in range(steps):
        perm = torch.randperm(batch, generator=g)[: batch // 2]
        out.append(sorted(int(x) for x in perm))
    return out


def bf16_bits(t: torch.Tensor):
    """Raw storage bits of a bf16 tensor as a numpy uint16 array (CPU copy)."""
    assert t.dtype == torch.bfloat16
    return t.detach().cpu().view(torch.int16).numpy().view("uint16")


def to_numpy(t: torch.Tensor):
    """Host copy of a tensor for the oracle: bf16 tensors come back as uint16 bit patterns, fp8 (E4M3)
    tensors as uint8 bit patterns, fp32 as float32."""
    if t.dtype == torch.bfloat16:
        return bf16_bits(t)
    if t.dtype == torch.float8_e4m3fn:
        return t.detach().view(torch.uint8).cpu().numpy()
    return t.detach().cpu().numpy()


def make_sim_traces(n: int, seed: int = 6000) -> Dict[str, np.ndarray]:
    """n synthetic reasoning traces: per-request and concatenated per-chunk arrays."""
    rng = np.random.default_rng(seed)
    prompt = rng.integers(50, 276, size=n)
    concl = rng.integers(100, 401, size=n)
    nothink = rng.random(n) < 0.35
    n_chunks, tokens, conf, correct = [], [], [], []
    for _ in range(n):
        total = int(rng.integers(3000, 14001))
        lens = []
        while sum(lens) < total:
            lens.append(max(1, int(round(rng.lognormal(np.log(900.0), 0.6)))))
        lens[-1] -= sum(lens) - total
        if lens[-1] < 1:
            lens.pop()
            lens[-1] += total - sum(lens)
        K = len(lens)
        settle = min(K - 1, int(rng.geometric(0.45)) - 1)
        final = rng.random() < 0.85
        for c in range(K):
            if c >= settle:
                ok = final
                cf = rng.uniform(0.95, 1.0) if rng.random() < 0.85 else rng.uniform(0.5, 0.95)
            else:
                ok = rng.random() < 0.35
                cf = rng.uniform(0.9, 1.0) if rng.random() < 0.10 else rng.uniform(0.2, 0.9)
            conf.append(cf)
            correct.append(ok)
        n_chunks.append(K)
        tokens += lens
    return {
        "prompt_len": prompt.astype(np.int32),
        "n_chunks": np.asarray(n_chunks, dtype=np.int32),
        "conclusion_tokens": concl.astype(np.int32),
        "nothink_correct": nothink.astype(np.int32),
        "chunk_tokens": np.asarray(tokens, dtype=np.int32),
        "confidence": np.asarray(conf, dtype=np.float32),
        "correct": np.asarray(correct, dtype=np.uint8),
    }


def make_poisson_arrivals(n: int, qps: float, seed: int = 7000) -> np.ndarray:
    """Arrival times (s) of n requests with exponential gaps of mean 1/qps, from t = 0."""
    rng = np.random.default_rng(seed)
    return np.cumsum(rng.exponential(1.0 / qps, size=n))


def make_phased_arrivals(rates: Sequence[float], durations_s: Sequence[float], seed: int = 7001) -> np.ndarray:
    """Poisson arrivals whose rate is rates[k] during the k-th phase of durations_s[k] seconds."""
    rng = np.random.default_rng(seed)
    out, t0 = [], 0.0
    for rate, dur in zip(rates, durations_s):
        t = t0
        while True:
            t += rng.exponential(1.0 / rate)
            if t >= t0 + dur:
                break
            out.append(t)
        t0 += dur
    return np.asarray(out, dtype=np.float64)
