"""Model shapes and synthetic workloads for the LASER decode + confidence-probe path.

The paper evaluates distilled reasoning models of 1.5B-8B parameters whose
chain-of-thought runs 3,000-14,000 tokens (Introduction), served from one GPU
(Section 3), and probes confidence at action transition points (Section 3.1,
Eq. 1).  The shapes below are random-initialised stand-ins with the
dimensions of those model families (Qwen2-style 1.5B/7B, Llama-style 8B) plus
a tiny decoder that the CPU oracle runs in seconds.  Nothing here holds any of
the method's arithmetic: these are plain records.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    tied_embeddings: bool
    qkv_bias: bool
    dtype: str  # "bf16" or "f32": weight storage type (and the KV cache's unless kv_dtype is set)
    rope_theta: float
    rms_eps: float
    kv_dtype: str = ""  # "" = dtype, or "fp8" (OCP E4M3 KV cache, bf16 models)

    @property
    def kv_storage(self) -> str:
        return self.kv_dtype or self.dtype

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def weight_bytes(self) -> int:
        """Bytes of every weight matrix read once per decode step (norm gains/biases included)."""
        es = 2 if self.dtype == "bf16" else 4
        d, hd = self.d_model, self.head_dim
        per_layer = (d * (self.n_q_heads + 2 * self.n_kv_heads) * hd + self.n_q_heads * hd * d + 3 * d * self.d_ffn)
        per_layer += 2 * d  # norm gains
        if self.qkv_bias:
            per_layer += (self.n_q_heads + 2 * self.n_kv_heads) * hd
        return es * (self.n_layers * per_layer + self.vocab * d + d)

    def kv_bytes_per_token(self) -> int:
        es = {"fp8": 1, "bf16": 2}.get(self.kv_storage, 4)
        return self.n_layers * 2 * self.n_kv_heads * self.head_dim * es


@dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    batch: int
    kv_lens: tuple  # pre-filled KV length per request (empty -> prompt prefill)
    decode_steps: int
    probe_every: int
    suffix_len: int = 8   # S: answer-inducing suffix tokens
    trial_len: int = 4    # T: trial-answer tokens scored for confidence
    prompt_len: int = 0   # >0: the prompt is prefilled through the chunked forward
    mixed: bool = False   # every step, a seeded half of the batch also runs a probe chunk
    page_size: int = 16


TINY = ModelShape("tiny-2L-d256", 2, 256, 4, 2, 64, 688, 2048, False, False, "f32", 1.0e4, 1.0e-5)
QWEN_1P5B = ModelShape("qwen2-1.5B-shape", 28, 1536, 12, 2, 128, 8960, 151936, True, True, "bf16", 1.0e4, 1.0e-6)
QWEN_7B = ModelShape("qwen2-7B-shape", 28, 3584, 28, 4, 128, 18944, 152064, False, True, "bf16", 1.0e4, 1.0e-6)
LLAMA_8B = ModelShape("llama-8B-shape", 32, 4096, 32, 8, 128, 14336, 128256, False, False, "bf16", 5.0e5, 1.0e-5)

# the same shapes with an fp8 (E4M3) KV cache
QWEN_1P5B_FP8KV = replace(QWEN_1P5B, name="qwen2-1.5B-shape-fp8kv", kv_dtype="fp8")
QWEN_7B_FP8KV = replace(QWEN_7B, name="qwen2-7B-shape-fp8kv", kv_dtype="fp8")
LLAMA_8B_FP8KV = replace(LLAMA_8B, name="llama-8B-shape-fp8kv", kv_dtype="fp8")

SHAPES = {s.name: s for s in (TINY, QWEN_1P5B, QWEN_7B, LLAMA_8B, QWEN_1P5B_FP8KV, QWEN_7B_FP8KV, LLAMA_8B_FP8KV)}

WORKLOADS = {
    w.name: w
    for w in (
        Workload("tiny-b1-prompt128", TINY, 1, (), 128, 32, prompt_len=128),
        Workload("1.5B-b1-kv4096", QWEN_1P5B, 1, (4096,), 512, 256),
        Workload("1.5B-b1-kv14336", QWEN_1P5B, 1, (14336,), 512, 128),
        Workload("7B-b4-ragged", QWEN_7B, 4, (3000, 6000, 10000, 14000), 256, 64),
        Workload("7B-b1-kv14336", QWEN_7B, 1, (14336,), 256, 64),
        Workload("7B-b1-kv14336-fp8kv", QWEN_7B_FP8KV, 1, (14336,), 256, 64),
        Workload("8B-b8-mixed", LLAMA_8B, 8, (), 64, 1, mixed=True),
        Workload("8B-b8-mixed-fp8kv", LLAMA_8B_FP8KV, 8, (), 64, 1, mixed=True),
    )
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]
