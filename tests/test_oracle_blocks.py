"""Pins for the oracle's transformer building blocks: closed forms, special cases, brute force."""
import math

import numpy as np
import pytest
from scipy.special import expit, softmax as sp_softmax

from oracle import transformer as T


def test_rmsnorm_closed_form_and_scale_invariance():
    g = np.linspace(0.5, 2.0, 8)
    c = -3.0
    out = T.rmsnorm(np.full(8, c), g, 1e-6)
    assert np.allclose(out, g * c / math.sqrt(c * c + 1e-6), rtol=0, atol=1e-15)
    rng = np.random.default_rng(0)
    x = rng.standard_normal(64)
    # with eps = 0 the norm is exactly scale invariant
    assert np.allclose(T.rmsnorm(x, 1.0, 0.0), T.rmsnorm(7.5 * x, 1.0, 0.0), atol=1e-14)
    # unit RMS after normalisation (eps = 0, unit gain)
    assert math.isclose(np.sqrt(np.mean(T.rmsnorm(x, 1.0, 0.0) ** 2)), 1.0, rel_tol=1e-14)


def test_rope_half_split_hand_example():
    # head_dim 4, theta 100: pair 0 = (x0, x2) rotates by pos * 100^0 = pos,
    # pair 1 = (x1, x3) rotates by pos * 100^(-2/4) = pos / 10
    x = np.array([1.0, 2.0, 3.0, 4.0])
    pos = 1
    a0, a1 = 1.0, 0.1
    expect = np.array([
        1.0 * math.cos(a0) - 3.0 * math.sin(a0),
        2.0 * math.cos(a1) - 4.0 * math.sin(a1),
        3.0 * math.cos(a0) + 1.0 * math.sin(a0),
        4.0 * math.cos(a1) + 2.0 * math.sin(a1),
    ])
    assert np.allclose(T.rope(x, pos, 100.0), expect, atol=1e-15)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((3, 64))
    k = rng.standard_normal((3, 64))
    assert np.array_equal(T.rope(q, 0, 1e4), q)
    for pos in (1, 17, 4096, 14335):
        r = T.rope(q, pos, 1e4)
        half = 32
        # each (i, i+half) pair keeps its length
        assert np.allclose(r[:, :half] ** 2 + r[:, half:] ** 2, q[:, :half] ** 2 + q[:, half:] ** 2, atol=1e-12)
    # <R_m q, R_n k> depends only on m - n
    for m, n in ((5, 2), (300, 297), (9000, 8997)):
        lhs = np.sum(T.rope(q, m, 1e4) * T.rope(k, n, 1e4), axis=-1)
        rhs = np.sum(T.rope(q, m - n, 1e4) * k, axis=-1)
        assert np.allclose(lhs, rhs, atol=1e-9)


def test_softmax_and_lm_stats():
    rng = np.random.default_rng(2)
    l = rng.standard_normal(2048) * 3
    p = T.softmax(l)
    assert math.isclose(p.sum(), 1.0, rel_tol=1e-14)
    assert np.allclose(p, sp_softmax(l), atol=1e-15)
    tok, pmax, margin = T.lm_stats(l)
    assert pmax == pytest.approx(sp_softmax(l).max(), rel=1e-13)
    assert 1.0 / l.size <= pmax <= 1.0
    srt = np.sort(l)
    assert margin == pytest.approx(srt[-1] - srt[-2])
    assert l[tok] == srt[-1]
    # uniform logits -> 1/V; ties break to the lowest index
    tok, pmax, margin = T.lm_stats(np.zeros(100))
    assert tok == 0 and pmax == pytest.approx(0.01, rel=1e-14) and margin == 0.0
    l2 = np.array([0.0, 5.0, 1.0, 5.0])
    assert T.lm_stats(l2)[0] == 1
    # one dominant logit -> probability close to 1
    assert T.lm_stats(np.array([0.0, 0.0, 60.0]))[1] == pytest.approx(1.0, abs=1e-15)
    assert T.lm_stats(np.array([0.0, 0.0, 3.0]))[1] == pytest.approx(1.0 / (1.0 + 2.0 * np.exp(-3.0)), rel=1e-14)


def _attention_brute(q, K, V):
    hq, hd = q.shape
    n, hkv, _ = K.shape
    G = hq // hkv
    out = np.zeros_like(q)
    for h in range(hq):
        kv = h // G
        scores = []
        for t in range(n):
            s = 0.0
            for d in range(hd):
                s += q[h, d] * K[t, kv, d]
            scores.append(s / math.sqrt(hd))
        m = max(scores)
        w = [math.exp(s - m) for s in scores]
        tot = sum(w)
        for d in range(hd):
            out[h, d] = sum(w[t] * V[t, kv, d] for t in range(n)) / tot
    return out


def test_gqa_attention_brute_force():
    rng = np.random.default_rng(4)
    for hq, hkv, n in ((4, 2, 9), (6, 1, 5), (3, 3, 7)):
        q = rng.standard_normal((hq, 8))
        K = rng.standard_normal((n, hkv, 8))
        V = rng.standard_normal((n, hkv, 8))
        assert np.allclose(T.gqa_attention(q, K, V), _attention_brute(q, K, V), atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((4, 16))
    K1 = rng.standard_normal((1, 2, 16))
    V1 = rng.standard_normal((1, 2, 16))
    o = T.gqa_attention(q, K1, V1)
    # a single visible token returns its value vector
    assert np.allclose(o[0], V1[0, 0]) and np.allclose(o[3], V1[0, 1])
    # identical keys -> uniform weights -> mean of the values
    K = np.repeat(K1, 6, axis=0)
    V = rng.standard_normal((6, 2, 16))
    o = T.gqa_attention(q, K, V)
    assert np.allclose(o[1], V[:, 0].mean(axis=0), atol=1e-14)
    # G = 1 (one KV head per query head) equals per-head attention
    Kf = rng.standard_normal((5, 4, 16))
    Vf = rng.standard_normal((5, 4, 16))
    o = T.gqa_attention(q, Kf, Vf)
    for h in range(4):
        w = T.softmax(Kf[:, h] @ q[h] / 4.0)
        assert np.allclose(o[h], w @ Vf[:, h], atol=1e-14)


def test_silu_closed_forms():
    x = np.linspace(-30, 30, 601)
    assert np.allclose(T.silu(x), x * expit(x), atol=1e-14)
    assert T.silu(np.array([0.0]))[0] == 0.0
    assert np.allclose(T.silu(-x), T.silu(x) - x, atol=1e-12)
