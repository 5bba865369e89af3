"""C6: the decode GEMV / skinny GEMM y[b, n] = sum_k W[n, k] x[b, k] (oracle).

The paper's weight kernels (§3.1 handwritten matmul, §4.4 up/down projection)
compute an ordinary matrix product; placement changes where the bytes live,
never the result.  The definition is written out directly:

  * inputs are bfloat16 bit patterns (uint16); bf16 -> float is exact
    (the 16 bits become the high half of an IEEE binary32);
  * ``gemv_f64`` accumulates in float64 (the reference of record);
  * ``gemv_f32`` accumulates in float32 through NumPy's matmul (the
    fp32-accumulated CPU result the GPU output is compared with);
  * float -> bf16 output rounding is round-to-nearest-even on the bit pattern.

W is [N, K] row-major (nn.Linear layout: the K-vector of one output is
contiguous), x is [B, K], y is [B, N].
"""
from __future__ import annotations

import numpy as np


def bf16_to_f32(u16: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(u16, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32)


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even of float32 values to bf16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    keep = u >> 16
    rest = u & 0xFFFF
    up = (rest > 0x8000) | ((rest == 0x8000) & ((keep & 1) == 1))
    out = (keep + up.astype(np.uint64)).astype(np.uint16)
    out[np.isnan(a)] = 0x7FC0
    return out


def gemv_f64(w_u16: np.ndarray, x_u16: np.ndarray) -> np.ndarray:
    w = bf16_to_f32(w_u16).astype(np.float64)
    x = bf16_to_f32(x_u16).astype(np.float64)
    return x @ w.T


def gemv_f32(w_u16: np.ndarray, x_u16: np.ndarray) -> np.ndarray:
    w = bf16_to_f32(w_u16)
    x = bf16_to_f32(x_u16)
    return (x @ w.T).astype(np.float32)


def gemv_rows_f64(w_rows_u16: np.ndarray, row_ids, x_u16: np.ndarray):
    """Sampled outputs y[:, row_ids] (fp64), from the rows W[row_ids] only.

    ``w_rows_u16[i]`` must be row ``row_ids[i]`` of W, in the same order, so
    that a tensor too large to bring to the host is checked on the rows that
    matter (every row cut by a page boundary, plus random ones).  Column i of
    the result is output row ``row_ids[i]``."""
    w_rows_u16 = np.asarray(w_rows_u16)
    if w_rows_u16.ndim != 2 or w_rows_u16.shape[0] != len(row_ids):
        raise ValueError("one row of W per row id")
    w = bf16_to_f32(w_rows_u16).astype(np.float64)
    x = bf16_to_f32(x_u16).astype(np.float64)
    return x @ w.T


def rel_err(y: np.ndarray, ref: np.ndarray) -> float:
    """max_i |y_i - r_i| / max(|r_i|, 1e-3 * rms(r)): the error measure the
    parity tolerance (2e-2 for bf16 inputs) is stated in."""
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(r * r))) if r.size else 0.0
    den = np.maximum(np.abs(r), 1e-3 * rms)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(y - r) / den)) if r.size else 0.0
