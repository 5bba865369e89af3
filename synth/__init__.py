"""Seeded synthetic inputs for the tiered-memory decode path.

This module is the only code shared by the product path and by the oracle.  It
draws random numbers and rounds them to the input dtype; it holds none of the
method's arithmetic (no placement, no allocation, no products or reductions).

Recipes (all values are synthetic; no dataset or checkpoint is used):

* bf16 inputs are ``rng.standard_normal(dtype=float32) * sigma`` rounded to
  bfloat16 with round-to-nearest-even on the float32 bit pattern, and handed
  around as ``uint16`` bit patterns.
* Weight tensors of the decode chain use ``sigma = 0.02`` and a per-tensor seed.
* Activations, queries and KV entries use ``sigma = 1``.
* Context lengths are uniform integers in a closed range.
"""
from __future__ import annotations

import numpy as np

PAGE_BYTES = 2 * 1024 * 1024


def round_bf16(a: np.ndarray) -> np.ndarray:
    """float32 array -> bfloat16 bit patterns (uint16), round-to-nearest-even."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # finite values stay below 2^32 after adding the rounding bias
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def uniforms(seed: int, n: int) -> np.ndarray:
    """n draws uniform on [0, 1) (float64) from ``default_rng(seed)``."""
    return np.random.default_rng(seed).random(int(n))


def normal_bf16(rng: np.random.Generator, shape, sigma: float) -> np.ndarray:
    f = rng.standard_normal(shape, dtype=np.float32)
    if sigma != 1.0:
        f *= np.float32(sigma)
    return round_bf16(f)


# ---------------------------------------------------------------- GEMV inputs
def gemv_inputs(seed: int, n: int, k: int, batch: int = 1,
                w_sigma: float = 0.02, x_sigma: float = 1.0):
    """W [n, k] then x [batch, k] from one stream ``default_rng(seed)``."""
    rng = np.random.default_rng(seed)
    w = normal_bf16(rng, (n, k), w_sigma)
    x = normal_bf16(rng, (batch, k), x_sigma)
    return w, x


def single_layer_inputs():
    """One bf16 linear layer W[4096 x 4096] ~N(0, 0.02) and x[4096] ~N(0, 1),
    seed 0 (16 pages of 2 MiB)."""
    return gemv_inputs(0, 4096, 4096, 1)


# Llama-3-8B-shaped decode weight chain (fused qkv and gate_up, nn.Linear
# layout [out, in]).
LLAMA8B = dict(layers=32, d=4096, ffn=14336, hq=32, hkv=8, head_dim=128,
               vocab=128256)
LLAMA70B = dict(layers=80, d=8192, ffn=28672, hq=64, hkv=8, head_dim=128,
                vocab=128256)
CHAIN_KINDS = ("qkv", "o", "gate_up", "down")


def chain_shapes(model: dict):
    """[(name, kind_index, N, K)] for one layer, then the lm_head."""
    d, f = model["d"], model["ffn"]
    hd = model["head_dim"]
    qkv = (model["hq"] + 2 * model["hkv"]) * hd
    per_layer = [("qkv", 0, qkv, d), ("o", 1, d, model["hq"] * hd),
                 ("gate_up", 2, 2 * f, d), ("down", 3, d, f)]
    return per_layer, ("lm_head", 9, model["vocab"], d)


def chain_seed(layer: int, kind_index: int) -> int:
    """Seed of tensor ``kind_index`` of ``layer``; the lm_head uses 9999."""
    if kind_index == 9:
        return 9999
    return 1000 + 10 * layer + kind_index


def chain_weight(layer: int, kind_index: int, n: int, k: int) -> np.ndarray:
    rng = np.random.default_rng(chain_seed(layer, kind_index))
    return normal_bf16(rng, (n, k), 0.02)


def chain_weight_torch(layer: int, kind_index: int, n: int, k: int, device):
    """Same recipe drawn on a device with torch's seeded generator (a
    different stream from the numpy one; used where gigabytes are needed)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(chain_seed(layer, kind_index))
    w = torch.randn((n, k), generator=g, device=device, dtype=torch.float32)
    w.mul_(0.02)
    return w.to(torch.bfloat16)


# ------------------------------------------------------- paged-attention inputs
def context_lengths(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(lo, hi, size=batch, endpoint=True).astype(np.int64)


def attention_inputs(batch: int, hq: int, hkv: int, head_dim: int,
                     lo: int, hi: int, seed: int = 0, kv_seed: int = 1,
                     lengths=None):
    """Context lengths and q from ``default_rng(seed)``; K/V of each request
    keyed by (request, token, kv head) from ``default_rng(kv_seed)`` drawn in
    logical order (request-major).  Returns lengths, q [B, Hq, D] and lists of
    K_b, V_b with shape [L_b, Hkv, D] (bf16 bit patterns)."""
    rng = np.random.default_rng(seed)
    if lengths is None:
        lengths = rng.integers(lo, hi, size=batch, endpoint=True).astype(np.int64)
    else:
        lengths = np.asarray(lengths, dtype=np.int64)
    q = normal_bf16(rng, (batch, hq, head_dim), 1.0)
    kr = np.random.default_rng(kv_seed)
    ks, vs = [], []
    for b in range(batch):
        ks.append(normal_bf16(kr, (int(lengths[b]), hkv, head_dim), 1.0))
        vs.append(normal_bf16(kr, (int(lengths[b]), hkv, head_dim), 1.0))
    return lengths, q, ks, vs


def attention_kv_torch(lengths, hkv: int, head_dim: int, kv_seed: int, device):
    """K and V of every request, all requests' tokens concatenated in logical
    order ([sum L_b, Hkv, D] bf16 each), drawn on a device with torch's seeded
    generator (used where gigabytes are needed; a different stream from
    ``attention_inputs``).  Request b's rows start at offsets[b]."""
    import torch
    lengths = np.asarray(lengths, dtype=np.int64)
    total = int(lengths.sum())
    g = torch.Generator(device=device)
    g.manual_seed(kv_seed)
    k = torch.randn((total, hkv, head_dim), generator=g, device=device,
                    dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn((total, hkv, head_dim), generator=g, device=device,
                    dtype=torch.float32).to(torch.bfloat16)
    offsets = np.concatenate([[0], np.cumsum(lengths)[:-1]]).astype(np.int64)
    return k, v, offsets


def churn_trace(seed: int, n_events: int, batch: int, lo: int, hi: int):
    """Replace events for KV-pool warm-up: (victim slot, new length) pairs."""
    rng = np.random.default_rng(seed)
    victims = rng.integers(0, batch, size=n_events)
    lengths = rng.integers(lo, hi, size=n_events, endpoint=True)
    return [(int(v), int(l)) for v, l in zip(victims, lengths)]


def poisson_arrivals(seed: int, steps: int, rate: float, prompt_lo: int, prompt_hi: int,
                     out_lo: int, out_hi: int):
    """Requests arriving over `steps` decode steps: the number arriving at each
    step is Poisson(rate); each request has a prompt length and an output
    length, uniform integers in the closed ranges.  Returns a list of
    (arrival step, prompt length, output length) in arrival order."""
    rng = np.random.default_rng(seed)
    counts = rng.poisson(rate, size=steps)
    n = int(counts.sum())
    prompts = rng.integers(prompt_lo, prompt_hi, size=n, endpoint=True)
    outs = rng.integers(out_lo, out_hi, size=n, endpoint=True)
    steps_of = np.repeat(np.arange(steps), counts)
    return [(int(s), int(p), int(o)) for s, p, o in zip(steps_of, prompts, outs)]
