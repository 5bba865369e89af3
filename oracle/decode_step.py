"""C8: one full decode step of a pre-norm Llama-style model (oracle, test-only).

The paper evaluates whole decode steps of Llama-style models (§5.1) but does
not restate the model; the step here is the standard pre-norm block, and its
constants are readings (the paper is silent on all of them):

  * RMSNorm:  y = x / sqrt(mean(x^2) + eps) * w, eps = 1e-5.
  * RoPE on query and key heads, half-split pairs (element i rotates with
    element i + D/2), angle = position * theta^(-2i/D), theta = 500000, no
    frequency scaling; position = context length - 1 (the new token).
  * SiLU(gate) * up with gate = first FFN rows of the fused gate_up weight.
  * Residual adds after attention and after the MLP; a final RMSNorm, the
    lm_head product and an argmax (ties: lowest index).
  * Fused qkv rows: Hq*D query rows, then H*D key rows, then H*D value rows,
    each head-major.
  * Precision points: every operand handed to a matrix product or to the
    attention (normed activations, q, k, v, attention output, SiLU product) is
    rounded to bf16 (round-to-nearest-even); the residual stream and all
    arithmetic here are float64.  The new token's k and v are appended to the
    cache in bf16.

Weights and inputs are bf16 bit patterns (uint16 arrays).
"""
from __future__ import annotations

import numpy as np

from .attention import decode_attention
from .gemv import bf16_to_f32, f32_to_bf16

EPS = 1e-5
THETA = 500000.0


def to_bf16(a64: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bits: round to float32 (nearest even), then to bf16
    (nearest even).  Values of interest are far from the double-rounding
    corner; both sides take the same two steps."""
    return f32_to_bf16(np.asarray(a64, dtype=np.float32))


def f64(u16: np.ndarray) -> np.ndarray:
    return bf16_to_f32(u16).astype(np.float64)


def rmsnorm(x: np.ndarray, w_u16: np.ndarray, eps: float = EPS) -> np.ndarray:
    """x [B, d] float64, w bf16 [d] -> float64 [B, d]."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * f64(w_u16)


def rope(x: np.ndarray, pos: np.ndarray, theta: float = THETA) -> np.ndarray:
    """x [B, heads, D] float64 rotated at positions pos [B] (half-split)."""
    B, nh, D = x.shape
    half = D // 2
    i = np.arange(half, dtype=np.float64)
    inv = theta ** (-2.0 * i / D)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]   # [B, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def silu(g: np.ndarray) -> np.ndarray:
    return g / (1.0 + np.exp(-g))


def argmax_lowest(logits: np.ndarray) -> np.ndarray:
    """Index of the maximum of every row; ties go to the lowest index."""
    return np.argmax(logits, axis=-1).astype(np.int64)


def decode_step(weights: dict, tokens: np.ndarray, k_cache, v_cache, lengths,
                dims: dict, trace: dict | None = None):
    """One decode step.

    weights: 'embed' [V, d]; per layer l: 'norm1.l' [d], 'qkv.l' [(Hq+2H)D, d],
      'o.l' [d, Hq D], 'norm2.l' [d], 'gate_up.l' [2F, d], 'down.l' [d, F];
      'norm_f' [d], 'lm_head' [V, d] (all bf16).
    tokens [B]: the token ids entering the step.
    k_cache[l][b], v_cache[l][b]: bf16 [L_b - 1, H, D], the context before the
      new token (lengths[b] = L_b counts the new token).
    dims: layers, d, hq, hkv, hd, ffn, vocab.
    Returns (logits float64 [B, V], ids [B], per-layer appended (k, v) bf16).
    trace, when given, receives the last layer's intermediates (diagnostics).
    """
    L, d = dims["layers"], dims["d"]
    Hq, H, D, F = dims["hq"], dims["hkv"], dims["hd"], dims["ffn"]
    B = len(tokens)
    pos = np.asarray(lengths, dtype=np.int64) - 1
    x = f64(weights["embed"][np.asarray(tokens)])                      # [B, d]
    appended = []
    for l in range(L):
        h = to_bf16(rmsnorm(x, weights[f"norm1.{l}"]))
        qkv = f64(h) @ f64(weights[f"qkv.{l}"]).T                      # [B, (Hq+2H)D]
        q = qkv[:, :Hq * D].reshape(B, Hq, D)
        k = qkv[:, Hq * D:(Hq + H) * D].reshape(B, H, D)
        v = qkv[:, (Hq + H) * D:].reshape(B, H, D)
        q16 = to_bf16(rope(q, pos))
        k16 = to_bf16(rope(k, pos))
        v16 = to_bf16(v)
        ks = [np.concatenate([k_cache[l][b], k16[b][None]], axis=0) for b in range(B)]
        vs = [np.concatenate([v_cache[l][b], v16[b][None]], axis=0) for b in range(B)]
        appended.append((k16, v16))
        o = to_bf16(decode_attention(q16, ks, vs))                     # [B, Hq, D]
        x = x + f64(o).reshape(B, Hq * D) @ f64(weights[f"o.{l}"]).T
        h2 = to_bf16(rmsnorm(x, weights[f"norm2.{l}"]))
        gu = f64(h2) @ f64(weights[f"gate_up.{l}"]).T
        act = to_bf16(silu(gu[:, :F]) * gu[:, F:])
        x = x + f64(act) @ f64(weights[f"down.{l}"]).T
        if trace is not None:
            trace.update(h=h, q=q16, k=k16, v=v16, o=o, h2=h2, act=act, x=x.copy())
    hf = to_bf16(rmsnorm(x, weights["norm_f"]))
    logits = f64(hf) @ f64(weights["lm_head"]).T
    return logits, argmax_lowest(logits), appended
