"""Decoder-only transformer decode step and trial-answer confidence probe (oracle).

Oracle (test infrastructure): plain numpy, float64 by default, no blocking,
fusion or reordering.  It follows the paper's statement of what runs at an
action transition point (ATP, Section 3.1, Eq. 1): the model keeps generating
its chain of thought token by token (the reasoning chunks T_k whose cost the
latency model Eq. 2 sums), and at an ATP an answer-inducing suffix makes it
emit a trial answer whose confidence is computed from the token probabilities.

The paper gives no model equations; the decoder below is the standard
Qwen2/Llama-style block that the distilled reasoners it evaluates use
(Section 5.1): RMSNorm, grouped-query attention with rotary position
embedding (half-split pairs), SwiGLU MLP, final RMSNorm and an LM head.
Readings of points the paper leaves open (each listed in the design doc):
  * confidence = arithmetic mean over the T trial tokens of the maximum
    softmax probability of the distribution that produced each token
    (temperature 1, greedy trial tokens);
  * the probe's suffix and trial tokens are discarded afterwards: the cache
    length and contents below the snapshot length are unchanged;
  * K and V are rounded to the cache's storage type when appended (bf16 for
    bf16 models, fp32 otherwise); queries and activations are not rounded.

Parity status: the building blocks (RMSNorm, RoPE, attention, SwiGLU, softmax
statistics) are pinned by closed forms, special cases and brute force; the
cached decode is pinned against the independent full-recompute form below.
Whole-model logits are "parity unpinned" with respect to the paper, which has
no worked example.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Mapping, Optional, Sequence

import numpy as np

from .numerics import as_dtype, as_float64, round_bf16, round_fp8_e4m3


# --------------------------------------------------------------------------- blocks

def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope_angles(pos: int, head_dim: int, theta: float) -> np.ndarray:
    """Rotation angle of pair i (i < head_dim/2) at position pos: pos * theta^(-2i/head_dim)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return float(pos) * theta ** (-2.0 * i / head_dim)


def rope(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate each head vector (last axis) at position pos; pairs are (i, i + head_dim/2)."""
    hd = x.shape[-1]
    half = hd // 2
    a = rope_angles(pos, hd, theta)
    c, s = np.cos(a), np.sin(a)
    lo, hi = x[..., :half], x[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def softmax(s: np.ndarray) -> np.ndarray:
    e = np.exp(s - np.max(s))
    return e / np.sum(e)


def gqa_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Grouped-query attention of one position.

    q [n_q_heads, hd]; K, V [n_ctx, n_kv_heads, hd] (every cached position is visible).
    Query head h reads KV head h // (n_q_heads / n_kv_heads).
    """
    hq, hd = q.shape
    hkv = K.shape[1]
    G = hq // hkv
    out = np.empty_like(q)
    for kv in range(hkv):
        # the keys and values of one KV head, read by its G query heads (a contiguous copy,
        # so each product below reads them densely)
        Kh = np.ascontiguousarray(K[:, kv, :])
        Vh = np.ascontiguousarray(V[:, kv, :])
        for h in range(kv * G, (kv + 1) * G):
            scores = Kh @ q[h] / math.sqrt(hd)  # (a Python float keeps the working precision)
            out[h] = softmax(scores) @ Vh
    return out


def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def lm_stats(logits: np.ndarray):
    """(greedy token, max softmax probability, top-2 logit margin) of one logit row.

    The greedy token is the lowest index among the maxima.  The maximum softmax
    probability is exp(l_max) / sum_j exp(l_j) = 1 / sum_j exp(l_j - l_max).
    """
    l = np.asarray(logits, dtype=np.float64)
    tok = int(np.argmax(l))  # numpy returns the first maximum
    lmax = l[tok]
    pmax = 1.0 / np.sum(np.exp(l - lmax))
    top2 = np.partition(l, -2)[-2:]
    margin = float(top2[1] - top2[0])
    return tok, float(pmax), margin


# --------------------------------------------------------------------------- state

class SeqState:
    """KV cache of one request: K, V [n_layers, capacity, n_kv_heads, head_dim] plus a length."""

    def __init__(self, shape, capacity: int, dtype=np.float64):
        dims = (shape.n_layers, capacity, shape.n_kv_heads, shape.head_dim)
        self.K = np.zeros(dims, dtype=dtype)
        self.V = np.zeros(dims, dtype=dtype)
        self.length = 0

    @classmethod
    def from_prefill(cls, shape, K0, V0, capacity: int, dtype=np.float64) -> "SeqState":
        """State holding pre-filled post-RoPE keys and values for positions 0..L0-1."""
        K0 = as_float64(K0)
        V0 = as_float64(V0)
        st = cls(shape, capacity, dtype)
        L0 = K0.shape[1]
        st.K[:, :L0] = K0
        st.V[:, :L0] = V0
        st.length = L0
        return st

    def truncate(self, n: int) -> None:
        self.length = n

    def copy(self) -> "SeqState":
        c = object.__new__(SeqState)
        c.K, c.V, c.length = self.K.copy(), self.V.copy(), self.length
        return c


@dataclass
class ProbeResult:
    confidence: float
    tokens: List[int]
    pmax: List[float]
    margins: List[float]
    logits: List[np.ndarray] = field(default_factory=list)


# --------------------------------------------------------------------------- model

class DecoderOracle:
    """Random-initialised decoder in float64 (or float32) with the storage rounding of its KV cache.

    weights: name -> array; uint16 arrays are bf16 bit patterns, other arrays are values.
    kv_storage: "bf16", "fp8" (E4M3), "f32" or None (no rounding, for the exact recompute invariant);
    defaults to the shape's storage dtype.
    """

    def __init__(self, shape, weights: Mapping[str, np.ndarray], dtype=np.float64, kv_storage: Optional[str] = "auto",
                 cache_weights: bool = False):
        self.shape = shape
        self.weights = weights
        self.dtype = dtype
        if kv_storage == "auto":
            kv_storage = getattr(shape, "kv_storage", shape.dtype)
        self.kv_storage = kv_storage
        # cache_weights keeps each tensor's decoded value after first use (memory for speed)
        self._cache = {} if cache_weights else None

    def set_weight(self, name: str, value: np.ndarray) -> None:
        """Replaces one input tensor (same encoding as the constructor's) and drops its cached value."""
        self.weights = dict(self.weights)
        self.weights[name] = value
        if self._cache is not None:
            self._cache.pop(name, None)

    def W(self, name: str) -> np.ndarray:
        if self._cache is not None:
            w = self._cache.get(name)
            if w is None:
                w = self._cache[name] = as_dtype(self.weights[name], self.dtype)
            return w
        return as_dtype(self.weights[name], self.dtype)

    def store_kv(self, x: np.ndarray) -> np.ndarray:
        if self.kv_storage == "bf16":
            return round_bf16(x).astype(self.dtype)
        if self.kv_storage == "fp8":
            return round_fp8_e4m3(x).astype(self.dtype)
        if self.kv_storage == "f32":
            return x.astype(np.float32).astype(self.dtype)
        return x

    def lm_weight(self) -> np.ndarray:
        return self.W("embed") if self.shape.tied_embeddings else self.W("lm_head")

    def decode_token(self, st: SeqState, token: int) -> np.ndarray:
        """Run one token at position st.length, append its K/V, return the logits [vocab]."""
        s = self.shape
        hq, hkv, hd = s.n_q_heads, s.n_kv_heads, s.head_dim
        pos = st.length
        h = self.W("embed")[int(token)].copy()
        for i in range(s.n_layers):
            p = f"layers.{i}."
            x = rmsnorm(h, self.W(p + "attn_norm"), s.rms_eps)
            q = self.W(p + "wq") @ x
            k = self.W(p + "wk") @ x
            v = self.W(p + "wv") @ x
            if s.qkv_bias:
                q = q + self.W(p + "bq")
                k = k + self.W(p + "bk")
                v = v + self.W(p + "bv")
            # (the rotation angles are float64; results are kept in the oracle's working precision)
            q = rope(q.reshape(hq, hd), pos, s.rope_theta).astype(self.dtype, copy=False)
            k = rope(k.reshape(hkv, hd), pos, s.rope_theta).astype(self.dtype, copy=False)
            st.K[i, pos] = self.store_kv(k)
            st.V[i, pos] = self.store_kv(v.reshape(hkv, hd))
            o = gqa_attention(q, st.K[i, : pos + 1], st.V[i, : pos + 1]).astype(self.dtype, copy=False)
            h = h + self.W(p + "wo") @ o.reshape(hq * hd)
            x = rmsnorm(h, self.W(p + "mlp_norm"), s.rms_eps)
            a = silu(self.W(p + "w_gate") @ x) * (self.W(p + "w_up") @ x)
            h = h + self.W(p + "w_down") @ a
        st.length = pos + 1
        return self.lm_weight() @ rmsnorm(h, self.W("final_norm"), s.rms_eps)

    def full_recompute(self, tokens: Sequence[int], K0=None, V0=None) -> np.ndarray:
        """Logits [n, vocab] of `tokens` placed after an optional pre-filled prefix, computed
        without a KV cache: every layer recomputes all chunk rows at once with a causal mask.
        K/V are not rounded here (exact reference for the cached decode invariant)."""
        s = self.shape
        hq, hkv, hd = s.n_q_heads, s.n_kv_heads, s.head_dim
        G = hq // hkv
        n = len(tokens)
        L0 = 0 if K0 is None else np.asarray(K0).shape[1]
        Kp = None if K0 is None else as_float64(K0)
        Vp = None if V0 is None else as_float64(V0)
        H = self.W("embed")[np.asarray(tokens, dtype=np.int64)].copy()  # [n, d]
        for i in range(s.n_layers):
            p = f"layers.{i}."
            X = rmsnorm(H, self.W(p + "attn_norm"), s.rms_eps)
            Q = X @ self.W(p + "wq").T
            Kc = X @ self.W(p + "wk").T
            Vc = X @ self.W(p + "wv").T
            if s.qkv_bias:
                Q, Kc, Vc = Q + self.W(p + "bq"), Kc + self.W(p + "bk"), Vc + self.W(p + "bv")
            Q = np.stack([rope(Q[r].reshape(hq, hd), L0 + r, s.rope_theta) for r in range(n)])
            Kc = np.stack([rope(Kc[r].reshape(hkv, hd), L0 + r, s.rope_theta) for r in range(n)])
            Vc = Vc.reshape(n, hkv, hd)
            if Kp is not None:
                Kall = np.concatenate([Kp[i], Kc], axis=0)
                Vall = np.concatenate([Vp[i], Vc], axis=0)
            else:
                Kall, Vall = Kc, Vc
            # mask[r, t]: chunk row r (position L0 + r) sees cache positions t <= L0 + r
            visible = np.arange(L0 + n)[None, :] <= (L0 + np.arange(n))[:, None]
            O = np.empty((n, hq, hd))
            for h in range(hq):
                S = Q[:, h, :] @ Kall[:, h // G, :].T / np.sqrt(hd)  # [n, L0+n]
                S = np.where(visible, S, -np.inf)
                S = S - S.max(axis=1, keepdims=True)
                P = np.exp(S)
                P = P / P.sum(axis=1, keepdims=True)
                O[:, h, :] = P @ Vall[:, h // G, :]
            H = H + O.reshape(n, hq * hd) @ self.W(p + "wo").T
            X = rmsnorm(H, self.W(p + "mlp_norm"), s.rms_eps)
            A = silu(X @ self.W(p + "w_gate").T) * (X @ self.W(p + "w_up").T)
            H = H + A @ self.W(p + "w_down").T
        return rmsnorm(H, self.W("final_norm"), s.rms_eps) @ self.lm_weight().T

    def probe(self, st: SeqState, suffix: Sequence[int], T: int, keep_logits: bool = False) -> ProbeResult:
        """Trial-answer confidence at an ATP (Section 3.1).

        The S suffix tokens run at positions L..L+S-1; the last one's distribution gives
        trial token t_1 and its max probability p_1; each t_j (j < T) is fed back to give
        t_{j+1}, p_{j+1}.  Confidence = (p_1 + ... + p_T) / T.  The cache is then cut back
        to length L, so the probe leaves the committed state unchanged.
        """
        L = st.length
        logits = None
        for tok in suffix:
            logits = self.decode_token(st, int(tok))
        toks, ps, margins, kept = [], [], [], []
        for j in range(T):
            if j > 0:
                logits = self.decode_token(st, toks[-1])
            t, pm, mg = lm_stats(logits)
            toks.append(t)
            ps.append(pm)
            margins.append(mg)
            if keep_logits:
                kept.append(logits.copy())
        st.truncate(L)
        conf = 0.0
        for pm in ps:
            conf += pm
        return ProbeResult(conf / T, toks, ps, margins, kept)
