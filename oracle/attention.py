"""C7: GQA decode attention over logical K/V (oracle, test-only).

The paper's attention kernels (§3.3: KV head chunks per threadblock; §4.5:
paged attention addressing tensors through base pointers and strides) compute
ordinary scaled dot-product attention for one new query token per request;
placement and the paged layout never change the result.  Written out directly
(the textbook definition; readings: no mask, ALiBi, soft-cap or window; the
context length already counts the current token; query head h reads KV head
h // G with G = Hq / H):

    s_t = scale * sum_d q[b, h, d] * k[b, t, g, d]         t < L_b
    p_t = exp(s_t - max_t s_t) / sum_t exp(s_t - max_t s_t)
    o[b, h, :] = sum_t p_t * v[b, t, g, :]

K and V are given per request in logical order as [L_b, H, D] bf16.

Reading for the degenerate case the paper never meets: a request with an
empty context (L_b = 0) has no softmax; its output row is zero.
"""
from __future__ import annotations

import numpy as np

from .gemv import bf16_to_f32


def _attend(q, k, v, scale):
    # q [G, D], k [L, D], v [L, D] -> [G, D] in the dtype of the inputs
    if k.shape[0] == 0:
        return np.zeros_like(q)
    s = (q @ k.T) * scale
    s = s - s.max(axis=1, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=1, keepdims=True)
    return p @ v


def decode_attention(q_u16, ks_u16, vs_u16, scale=None, dtype=np.float64,
                     heads=None):
    """o [B, Hq, D] for queries q [B, Hq, D] and per-request K/V lists.
    ``heads`` restricts the computation to a list of (b, h) pairs and then
    returns a dict keyed by (b, h)."""
    B, Hq, D = q_u16.shape
    H = ks_u16[0].shape[1] if ks_u16 else 1
    G = Hq // H
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    q = bf16_to_f32(q_u16).astype(dtype)
    pairs = heads if heads is not None else [(b, h) for b in range(B)
                                              for h in range(Hq)]
    res = {}
    cache = {}
    for b, h in pairs:
        g = h // G
        key = (b, g)
        if key not in cache:
            cache[key] = (bf16_to_f32(ks_u16[b][:, g, :]).astype(dtype),
                          bf16_to_f32(vs_u16[b][:, g, :]).astype(dtype))
        k, v = cache[key]
        res[(b, h)] = _attend(q[b, h][None, :], k, v, dtype(scale))[0]
    if heads is not None:
        return res
    out = np.zeros((B, Hq, D), dtype=dtype)
    for (b, h), o in res.items():
        out[b, h] = o
    return out
