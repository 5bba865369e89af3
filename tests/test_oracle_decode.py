"""Pins of the full decode-step oracle (C8) and its parts."""
import math

import numpy as np
import pytest

import synth
from oracle import decode_step as ods
from oracle.gemv import bf16_to_f32


def bf(a):
    return synth.round_bf16(np.asarray(a, dtype=np.float32))


def test_rmsnorm_constant_vector():
    """x = c * 1 gives w * c / sqrt(c^2 + eps)."""
    d = 64
    w = bf(np.linspace(0.5, 2.0, d))
    for c in (3.0, -0.25):
        x = np.full((1, d), c)
        y = ods.rmsnorm(x, w)
        wf = bf16_to_f32(w).astype(np.float64)
        assert np.allclose(y[0], wf * c / math.sqrt(c * c + ods.EPS), rtol=1e-14)


def test_rope_position_zero_is_identity_and_norm_preserved():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((3, 4, 128))
    assert np.array_equal(ods.rope(x, np.zeros(3)), x)
    y = ods.rope(x, np.array([1, 77, 4095]))
    half = 64
    n0 = x[..., :half] ** 2 + x[..., half:] ** 2
    n1 = y[..., :half] ** 2 + y[..., half:] ** 2
    assert np.allclose(n0, n1, rtol=1e-12)


def test_rope_closed_form_two_dims():
    """D = 2: one pair rotated by exactly the position (inv freq 1)."""
    x = np.array([[[0.6, -1.3]]])
    y = ods.rope(x, np.array([1.0]), theta=10000.0)[0, 0]
    c, s = math.cos(1.0), math.sin(1.0)
    assert np.allclose(y, [0.6 * c + 1.3 * s, 0.6 * s - 1.3 * c], rtol=1e-14)
    # D = 4: the second pair turns at theta^(-1/2)
    x4 = np.array([[[1.0, 0.0, 0.0, 0.0]]])
    y4 = ods.rope(x4, np.array([3.0]), theta=100.0)[0, 0]
    assert np.allclose(y4, [math.cos(3.0), 0.0, math.sin(3.0), 0.0], atol=1e-15)
    x4b = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    y4b = ods.rope(x4b, np.array([3.0]), theta=100.0)[0, 0]
    assert np.allclose(y4b, [0.0, math.cos(0.3), 0.0, math.sin(0.3)], atol=1e-15)


def test_rope_relative_position_property():
    """<rope(q, m), rope(k, n)> depends only on m - n."""
    rng = np.random.default_rng(1)
    q = rng.standard_normal((1, 1, 128))
    k = rng.standard_normal((1, 1, 128))
    dots = [float(np.sum(ods.rope(q, np.array([m])) * ods.rope(k, np.array([m - 5]))))
            for m in (5, 17, 300, 2047)]
    assert max(dots) - min(dots) < 1e-9 * max(1.0, abs(dots[0]))


def test_silu_identities():
    g = np.linspace(-20, 20, 401)
    assert ods.silu(np.array([0.0]))[0] == 0.0
    assert np.allclose(ods.silu(-g), ods.silu(g) - g, atol=1e-12)
    assert abs(ods.silu(np.array([30.0]))[0] - 30.0) < 1e-10


def test_argmax_ties_lowest():
    lg = np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0]])
    assert ods.argmax_lowest(lg).tolist() == [1, 0]


DIMS = dict(layers=2, d=64, hq=4, hkv=2, hd=16, ffn=96, vocab=50)


def tiny_model(seed, zero=()):
    rng = np.random.default_rng(seed)
    d, Hq, H, D, F, V = (DIMS[k] for k in ("d", "hq", "hkv", "hd", "ffn", "vocab"))
    w = {"embed": synth.normal_bf16(rng, (V, d), 1.0),
         "norm_f": bf(1 + 0.1 * rng.standard_normal(d)),
         "lm_head": synth.normal_bf16(rng, (V, d), 0.1)}
    for l in range(DIMS["layers"]):
        w[f"norm1.{l}"] = bf(1 + 0.1 * rng.standard_normal(d))
        w[f"norm2.{l}"] = bf(1 + 0.1 * rng.standard_normal(d))
        w[f"qkv.{l}"] = synth.normal_bf16(rng, ((Hq + 2 * H) * D, d), 0.1)
        w[f"o.{l}"] = synth.normal_bf16(rng, (d, Hq * D), 0.1)
        w[f"gate_up.{l}"] = synth.normal_bf16(rng, (2 * F, d), 0.1)
        w[f"down.{l}"] = synth.normal_bf16(rng, (d, F), 0.1)
    for name in zero:
        for key in list(w):
            if key.split(".")[0] == name:
                w[key] = np.zeros_like(w[key])
    return w


def caches(seed, lengths):
    rng = np.random.default_rng(seed)
    H, D = DIMS["hkv"], DIMS["hd"]
    kc = [[synth.normal_bf16(rng, (L - 1, H, D), 1.0) for L in lengths]
          for _ in range(DIMS["layers"])]
    vc = [[synth.normal_bf16(rng, (L - 1, H, D), 1.0) for L in lengths]
          for _ in range(DIMS["layers"])]
    return kc, vc


def test_step_without_block_outputs_reduces_to_embedding():
    """Zero attention and MLP output projections: the residual stream stays
    at the embedding, so logits = lm_head . rmsnorm(embed[token])."""
    w = tiny_model(2, zero=("o", "down"))
    tokens = np.array([3, 17, 49])
    lengths = [5, 1, 40]
    kc, vc = caches(3, lengths)
    logits, ids, _ = ods.decode_step(w, tokens, kc, vc, lengths, DIMS)
    x = ods.f64(w["embed"][tokens])
    exp = ods.f64(ods.to_bf16(ods.rmsnorm(x, w["norm_f"]))) @ ods.f64(w["lm_head"]).T
    assert np.allclose(logits, exp, rtol=1e-13, atol=1e-13)
    # tied lm_head with unit final norm: each token predicts itself
    w2 = dict(w)
    w2["lm_head"] = w["embed"]
    w2["norm_f"] = bf(np.ones(DIMS["d"]))
    _, ids2, _ = ods.decode_step(w2, tokens, kc, vc, lengths, DIMS)
    assert ids2.tolist() == tokens.tolist()


def test_zero_qkv_attends_uniformly_including_new_token():
    """q = k = v = 0: attention weights are uniform over the L_b tokens, the
    new token's value is zero, so the attention output is sum(cache v)/L_b."""
    w = tiny_model(4, zero=("qkv", "down"))
    tokens = np.array([1, 2])
    lengths = [7, 3]
    kc, vc = caches(5, lengths)
    _, _, app = ods.decode_step(w, tokens, kc, vc, lengths, DIMS)
    # (rotating zeros may give -0.0: compare values, not bit patterns)
    assert all(np.all(ods.f64(k) == 0) and np.all(ods.f64(v) == 0) for k, v in app)
    # reproduce layer 0's residual update by hand
    Hq, H, D = DIMS["hq"], DIMS["hkv"], DIMS["hd"]
    G = Hq // H
    x = ods.f64(w["embed"][tokens])
    for l in range(DIMS["layers"]):
        o = np.zeros((2, Hq, D))
        for b, L in enumerate(lengths):
            for h in range(Hq):
                o[b, h] = ods.f64(vc[l][b][:, h // G, :]).sum(axis=0) / L
        x = x + ods.f64(ods.to_bf16(o)).reshape(2, Hq * D) @ ods.f64(w[f"o.{l}"]).T
    exp = ods.f64(ods.to_bf16(ods.rmsnorm(x, w["norm_f"]))) @ ods.f64(w["lm_head"]).T
    logits, _, _ = ods.decode_step(w, tokens, kc, vc, lengths, DIMS)
    assert np.allclose(logits, exp, rtol=1e-12, atol=1e-12)


def test_mlp_only_layer_closed_form():
    """With zero attention output, each layer adds down . (silu(gate) * up)."""
    w = tiny_model(6, zero=("o",))
    tokens = np.array([0, 9])
    lengths = [2, 2]
    kc, vc = caches(7, lengths)
    F = DIMS["ffn"]
    x = ods.f64(w["embed"][tokens])
    for l in range(DIMS["layers"]):
        h2 = ods.f64(ods.to_bf16(ods.rmsnorm(x, w[f"norm2.{l}"])))
        gu = h2 @ ods.f64(w[f"gate_up.{l}"]).T
        g, u = gu[:, :F], gu[:, F:]
        act = ods.f64(ods.to_bf16(g / (1 + np.exp(-g)) * u))
        x = x + act @ ods.f64(w[f"down.{l}"]).T
    exp = ods.f64(ods.to_bf16(ods.rmsnorm(x, w["norm_f"]))) @ ods.f64(w["lm_head"]).T
    logits, _, _ = ods.decode_step(w, tokens, kc, vc, lengths, DIMS)
    assert np.allclose(logits, exp, rtol=1e-12, atol=1e-12)


SMALL = dict(layers=1, d=8, hq=2, hkv=1, hd=4, ffn=8, vocab=10)


def small_model(seed, qkv=None):
    rng = np.random.default_rng(seed)
    d, Hq, H, D, F, V = (SMALL[k] for k in ("d", "hq", "hkv", "hd", "ffn", "vocab"))
    w = {"embed": synth.normal_bf16(rng, (V, d), 1.0),
         "norm_f": bf(1 + 0.1 * rng.standard_normal(d)),
         "lm_head": synth.normal_bf16(rng, (V, d), 0.3),
         "norm1.0": bf(1 + 0.1 * rng.standard_normal(d)),
         "norm2.0": bf(1 + 0.1 * rng.standard_normal(d)),
         "qkv.0": synth.normal_bf16(rng, ((Hq + 2 * H) * D, d), 0.5),
         "o.0": synth.normal_bf16(rng, (d, Hq * D), 0.3),
         "gate_up.0": synth.normal_bf16(rng, (2 * F, d), 0.3),
         "down.0": synth.normal_bf16(rng, (d, F), 0.3)}
    if qkv is not None:
        w["qkv.0"] = qkv
    return w


def rot4(x, pos, theta=ods.THETA):
    """Half-split rotation of one D = 4 head written out: element 0 pairs
    with 2 at angle pos, element 1 with 3 at angle pos * theta^(-1/2)."""
    a0, a1 = pos, pos / math.sqrt(theta)
    c0, s0, c1, s1 = math.cos(a0), math.sin(a0), math.cos(a1), math.sin(a1)
    return np.array([x[0] * c0 - x[2] * s0, x[1] * c1 - x[3] * s1,
                     x[0] * s0 + x[2] * c0, x[1] * s1 + x[3] * c1])


def test_rope_position_is_context_length_minus_one():
    """Context of two tokens (one cached, one new): the new token sits at
    position 1.  Its query and key are the qkv rows rotated by exactly that
    position, and the attention output worked from them by hand matches;
    rotating by position 2 (or 0) would give other queries and another
    output."""
    w = small_model(11)
    kc = [[synth.normal_bf16(np.random.default_rng(12), (1, 1, 4), 1.0)]]
    vc = [[synth.normal_bf16(np.random.default_rng(13), (1, 1, 4), 1.0)]]
    tr = {}
    ods.decode_step(w, np.array([3]), kc, vc, [2], SMALL, trace=tr)
    raw = ods.f64(tr["h"]) @ ods.f64(w["qkv.0"]).T                  # [1, 16]
    q_raw = raw[0, :8].reshape(2, 4)
    k_raw = raw[0, 8:12]
    v_raw = raw[0, 12:16]
    exp_q = np.stack([rot4(q_raw[h], 1.0) for h in range(2)])
    assert np.array_equal(tr["q"][0], ods.to_bf16(exp_q))
    assert np.array_equal(tr["k"][0, 0], ods.to_bf16(rot4(k_raw, 1.0)))
    assert np.array_equal(tr["v"][0, 0], ods.to_bf16(v_raw))
    for wrong in (0.0, 2.0):
        bad = np.stack([rot4(q_raw[h], wrong) for h in range(2)])
        assert not np.array_equal(tr["q"][0], ods.to_bf16(bad))
    # the attention output of each query head over (cached, new), by hand
    k0, v0 = ods.f64(kc[0][0][0, 0]), ods.f64(vc[0][0][0, 0])
    k1, v1 = ods.f64(tr["k"][0, 0]), ods.f64(tr["v"][0, 0])

    def attend(q):
        s0, s1 = float(q @ k0) / 2.0, float(q @ k1) / 2.0      # 1/sqrt(D), D = 4
        e0, e1 = math.exp(s0 - max(s0, s1)), math.exp(s1 - max(s0, s1))
        return (e0 * v0 + e1 * v1) / (e0 + e1)

    got = ods.f64(tr["o"][0])
    for h in range(2):
        ref = attend(ods.f64(tr["q"][0, h]))
        assert np.all(np.abs(got[h] - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-30)
    # the same by hand with the query rotated to position 2 instead: far off
    q2 = ods.f64(ods.to_bf16(rot4(q_raw[0], 2.0)))
    assert np.max(np.abs(attend(q2) - got[0])) > 1e-2


def test_qkv_split_query_key_value_rows():
    """Fused qkv rows are Hq*D query rows, then H*D key rows, then H*D value
    rows, each head-major.  Row r of the weight is (r + 1) * e_0, so output
    r is (r + 1) * h[0]: query head 0 gets 1..4, head 1 5..8, the key 9..12
    and the value 13..16 (times h[0]).  At position 0 RoPE is the identity
    and one token's attention returns its value."""
    qkv = np.zeros((16, 8), np.float32)
    qkv[:, 0] = np.arange(1, 17)
    w = small_model(21, qkv=bf(qkv))
    tr = {}
    _, _, app = ods.decode_step(w, np.array([5]), [[np.zeros((0, 1, 4), np.uint16)]],
                                [[np.zeros((0, 1, 4), np.uint16)]], [1], SMALL, trace=tr)
    h0 = float(ods.f64(tr["h"])[0, 0])
    assert h0 != 0.0
    ramp = np.arange(1, 17, dtype=np.float64) * h0
    assert np.array_equal(tr["q"][0], ods.to_bf16(ramp[:8].reshape(2, 4)))
    assert np.array_equal(tr["k"][0, 0], ods.to_bf16(ramp[8:12]))
    assert np.array_equal(tr["v"][0, 0], ods.to_bf16(ramp[12:16]))
    assert np.array_equal(app[0][0], tr["k"]) and np.array_equal(app[0][1], tr["v"])
    assert np.array_equal(tr["o"][0], np.stack([tr["v"][0, 0]] * 2))
