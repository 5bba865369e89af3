"""Pins of the decode-attention oracle (C7)."""
import math

import numpy as np
import pytest

import synth
from oracle import attention as oa
from oracle.gemv import bf16_to_f32


def bf(a):
    return synth.round_bf16(np.asarray(a, dtype=np.float32))


def test_single_token_returns_v0():
    rng = np.random.default_rng(0)
    q = synth.normal_bf16(rng, (2, 4, 16), 1.0)
    ks = [synth.normal_bf16(rng, (1, 2, 16), 1.0) for _ in range(2)]
    vs = [synth.normal_bf16(rng, (1, 2, 16), 1.0) for _ in range(2)]
    o = oa.decode_attention(q, ks, vs)
    for b in range(2):
        for h in range(4):
            assert np.array_equal(o[b, h], bf16_to_f32(vs[b][0, h // 2]).astype(np.float64))


def test_zero_query_gives_mean_of_values():
    rng = np.random.default_rng(1)
    q = bf(np.zeros((1, 2, 8)))
    ks = [synth.normal_bf16(rng, (37, 1, 8), 1.0)]
    vs = [synth.normal_bf16(rng, (37, 1, 8), 1.0)]
    o = oa.decode_attention(q, ks, vs)
    mean = bf16_to_f32(vs[0][:, 0]).astype(np.float64).mean(axis=0)
    assert np.allclose(o[0, 0], mean, atol=1e-14) and np.allclose(o[0, 1], mean, atol=1e-14)


def test_two_token_closed_form():
    """o = (1 - s) v0 + s v1 with s = sigmoid(scale * q.(k1 - k0))."""
    D = 4
    q = bf([[[1.0, 2.0, 0.0, 0.0]]])
    k = bf([[[0.0, 0.0, 0.0, 0.0]], [[1.5, 0.25, 3.0, -1.0]]])
    v = bf([[[1.0, 0.0, -1.0, 2.0]], [[0.0, 4.0, 1.0, 0.5]]])
    o = oa.decode_attention(q, [k], [v])[0, 0]
    z = (1.0 * 1.5 + 2.0 * 0.25) / math.sqrt(D)
    s = 1.0 / (1.0 + math.exp(-z))
    v0, v1 = np.array([1.0, 0.0, -1.0, 2.0]), np.array([0.0, 4.0, 1.0, 0.5])
    assert np.allclose(o, (1 - s) * v0 + s * v1, atol=1e-14)
    # an explicit scale replaces 1/sqrt(D)
    o2 = oa.decode_attention(q, [k], [v], scale=1.0)[0, 0]
    s2 = 1.0 / (1.0 + math.exp(-(1.5 + 0.5)))
    assert np.allclose(o2, (1 - s2) * v0 + s2 * v1, atol=1e-14)


def test_dominant_score_selects_value():
    D = 8
    q = bf(np.full((1, 1, D), 4.0))
    k = np.zeros((5, 1, D), dtype=np.float32)
    k[3] = 8.0
    v = np.arange(5 * D, dtype=np.float32).reshape(5, 1, D)
    o = oa.decode_attention(q, [bf(k)], [bf(v)])[0, 0]
    assert np.allclose(o, v[3, 0], atol=1e-9)


def test_gqa_group_mapping():
    """Query head h reads KV head h // G (groups contiguous)."""
    B, Hq, H, D, L = 1, 8, 2, 4, 3
    q = bf(np.ones((B, Hq, D)))
    k = bf(np.zeros((L, H, D)))
    v = np.zeros((L, H, D), dtype=np.float32)
    for g in range(H):
        v[:, g, :] = g + 1
    o = oa.decode_attention(q, [k], [bf(v)])
    for h in range(Hq):
        assert np.all(o[0, h] == h // (Hq // H) + 1)


def test_f32_close_to_f64_and_subset():
    lengths, q, ks, vs = synth.attention_inputs(3, 8, 2, 32, 5, 70, seed=3)
    o64 = oa.decode_attention(q, ks, vs)
    o32 = oa.decode_attention(q, ks, vs, dtype=np.float32)
    assert np.max(np.abs(o32 - o64)) < 1e-5
    sub = oa.decode_attention(q, ks, vs, heads=[(2, 5), (0, 0)])
    assert np.array_equal(sub[(2, 5)], o64[2, 5]) and np.array_equal(sub[(0, 0)], o64[0, 0])


def test_empty_context_gives_zero_row():
    rng = np.random.default_rng(2)
    q = synth.normal_bf16(rng, (2, 2, 8), 1.0)
    ks = [np.zeros((0, 1, 8), np.uint16), synth.normal_bf16(rng, (3, 1, 8), 1.0)]
    vs = [np.zeros((0, 1, 8), np.uint16), synth.normal_bf16(rng, (3, 1, 8), 1.0)]
    o = oa.decode_attention(q, ks, vs)
    assert np.all(o[0] == 0) and np.all(np.isfinite(o[1])) and np.any(o[1] != 0)
