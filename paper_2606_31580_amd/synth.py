"""Seeded synthetic inputs shared by the GPU path's tests/bench and the CPU oracle.

This module only draws random numbers (torch generators with fixed seeds) and
names tensors; it holds none of the method's arithmetic.  Weights follow the
random-init recipe: every matrix, embedding and bias ~N(0, 0.02) rounded to the
storage dtype (bf16 round-to-nearest-even, or fp32), norm gains 1.0.
Pre-filled KV entries ~N(0, 1) stand for an already-generated chain of thought
(post-RoPE keys), tokens are uniform over the vocabulary.

Seeds: weights 1000 + tensor index (fixed name order), pre-filled KV 2000 +
request index, prompt/first tokens/suffix 3000.., ragged lengths and the
mixed-step schedule 4000.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import torch

from .configs import ModelShape

WEIGHT_STD = 0.02


def _tdtype(shape: ModelShape) -> torch.dtype:
    return torch.bfloat16 if shape.dtype == "bf16" else torch.float32


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
    """Pre-filled (K, V) for one request: two tensors [n_layers, length, n_kv_heads, head_dim], ~N(0,1)."""
    g = torch.Generator(device=device)
    g.manual_seed(seed_base + request)
    dims = (shape.n_layers, length, shape.n_kv_heads, shape.head_dim)
    k = torch.randn(dims, generator=g, device=device, dtype=torch.float32).to(_tdtype(shape))
    v = torch.randn(dims, generator=g, device=device, dtype=torch.float32).to(_tdtype(shape))
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
    """Host copy of a tensor for the oracle: bf16 tensors come back as uint16 bit patterns, fp32 as float32."""
    if t.dtype == torch.bfloat16:
        return bf16_bits(t)
    return t.detach().cpu().numpy()
