"""Pins of the GEMV oracle (C6) and the bf16 conversions."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import gemv as og

WORKED = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "gemv_worked_example.json")))


def bf(a):
    return synth.round_bf16(np.asarray(a, dtype=np.float32))


def test_bf16_decode_known_patterns():
    u = np.array([0x3F80, 0xC000, 0x3F00, 0x0001, 0x7F80, 0x0000, 0x8000,
                  0x4049], dtype=np.uint16)
    f = og.bf16_to_f32(u)
    assert f[0] == 1.0 and f[1] == -2.0 and f[2] == 0.5
    assert f[3] == np.float32(2.0 ** -133)
    assert np.isinf(f[4]) and f[5] == 0.0 and np.signbit(f[6])
    assert f[7] == np.float32(3.140625)


def test_bf16_round_nearest_even():
    one = np.float32(1.0)
    vals = np.array([one + np.float32(2.0 ** -8),          # tie -> even (down)
                     one + np.float32(3 * 2.0 ** -8),      # tie -> even (up)
                     one + np.float32(2.0 ** -8 + 2.0 ** -20),  # above tie
                     np.float32(-1.5), np.float32(65504.0)],
                    dtype=np.float32)
    got = og.f32_to_bf16(vals)
    assert got.tolist() == [0x3F80, 0x3F82, 0x3F81, 0xBFC0, 0x4780]
    # the oracle's encoder and the input generator's agree (independent code)
    r = np.random.default_rng(0).standard_normal(100000).astype(np.float32)
    assert np.array_equal(og.f32_to_bf16(r), synth.round_bf16(r))
    # round trip of bf16 values is exact
    u = synth.round_bf16(r)
    assert np.array_equal(og.f32_to_bf16(og.bf16_to_f32(u)), u)


def test_worked_example():
    w, x = bf(WORKED["W"]), bf(WORKED["x"])
    y64 = og.gemv_f64(w, x)
    y32 = og.gemv_f32(w, x)
    assert y64.tolist() == WORKED["y"]
    assert y32.tolist() == WORKED["y"]


def test_identity_and_unit_vectors():
    n = 64
    rng = np.random.default_rng(1)
    x = synth.normal_bf16(rng, (3, n), 1.0)
    eye = bf(np.eye(n))
    assert np.array_equal(og.gemv_f64(eye, x), og.bf16_to_f32(x))
    w = synth.normal_bf16(rng, (40, n), 0.02)
    for j in (0, 17, n - 1):
        e = np.zeros((1, n), dtype=np.float32)
        e[0, j] = 1
        assert np.array_equal(og.gemv_f32(w, bf(e))[0], og.bf16_to_f32(w)[:, j])


def test_all_ones_exact():
    k = 4096
    w = bf(np.ones((8, k)))
    x = bf(np.ones((1, k)))
    assert np.all(og.gemv_f32(w, x) == k)


def test_nonsquare_catches_transpose():
    rng = np.random.default_rng(2)
    w = synth.normal_bf16(rng, (5, 7), 1.0)
    x = synth.normal_bf16(rng, (2, 7), 1.0)
    y = og.gemv_f64(w, x)
    assert y.shape == (2, 5)
    wf, xf = og.bf16_to_f32(w).astype(np.float64), og.bf16_to_f32(x).astype(np.float64)
    for b in range(2):
        for n in range(5):
            assert abs(y[b, n] - sum(wf[n, k] * xf[b, k] for k in range(7))) < 1e-12


@pytest.mark.parametrize("n,k", [(256, 4096), (64, 14336)])
def test_f32_within_rounding_bound_of_f64(n, k):
    """|y32 - y64| <= K * eps32 * sum |w x| (standard summation bound)."""
    rng = np.random.default_rng(4)
    w = synth.normal_bf16(rng, (n, k), 0.02)
    x = synth.normal_bf16(rng, (2, k), 1.0)
    y32, y64 = og.gemv_f32(w, x), og.gemv_f64(w, x)
    mag = np.abs(og.bf16_to_f32(x).astype(np.float64)) @ \
        np.abs(og.bf16_to_f32(w).astype(np.float64)).T
    assert np.all(np.abs(y32 - y64) <= k * 2 ** -24 * mag)
    assert og.rel_err(y32, y64) < 1e-3


def test_rel_err_measure():
    r = np.array([1.0, -2.0, 1e-9, 0.0])
    assert og.rel_err(r, r) == 0.0
    y = r.copy()
    y[1] = -2.04
    assert abs(og.rel_err(y, r) - 0.02) < 1e-12


def test_rows_hand_worked_shuffled():
    """Sampled rows in shuffled order: column i is output row row_ids[i].
    W [5 x 4] and x [2 x 4] are small integers (exact in bf16); the outputs
    are worked by hand:
      row 4 = [1, 0, -2, 3]:  x0 = [1, 2, 3, 4] -> 1 - 6 + 12 = 7
                              x1 = [-1, 0, 2, 1] -> -1 - 4 + 3 = -2
      row 0 = [2, -1, 0, 1]:  x0 -> 2 - 2 + 4 = 4;   x1 -> -2 + 1 = -1
      row 2 = [0, 3, 1, -1]:  x0 -> 6 + 3 - 4 = 5;   x1 -> 2 - 1 = 1"""
    W = bf(np.array([[2, -1, 0, 1], [5, 5, 5, 5], [0, 3, 1, -1], [9, 9, 9, 9],
                     [1, 0, -2, 3]]))
    x = bf(np.array([[1, 2, 3, 4], [-1, 0, 2, 1]]))
    rows = np.array([4, 0, 2])
    y = og.gemv_rows_f64(W[rows], rows, x)
    assert y.tolist() == [[7.0, 4.0, 5.0], [-2.0, -1.0, 1.0]]
    # the same columns of the full product
    assert og.gemv_f64(W, x)[:, rows].tolist() == y.tolist()
    with pytest.raises(ValueError):
        og.gemv_rows_f64(W[rows], rows[:2], x)


def test_rows_equal_brute_force_columns():
    """Random rows (shuffled, repeated) against a plain double loop over the
    full W: a row shift, a transposed W or a dropped batch row fails."""
    rng = np.random.default_rng(9)
    n, k, B = 37, 72, 3
    w = synth.normal_bf16(rng, (n, k), 0.02)
    x = synth.normal_bf16(rng, (B, k), 1.0)
    rows = rng.permutation(n)[:11]
    rows = np.concatenate([rows, rows[:2]])
    y = og.gemv_rows_f64(w[rows], rows, x)
    wf = og.bf16_to_f32(w).astype(np.float64)
    xf = og.bf16_to_f32(x).astype(np.float64)
    for b in range(B):
        for i, r in enumerate(rows):
            ref = sum(wf[r, c] * xf[b, c] for c in range(k))
            assert abs(y[b, i] - ref) <= 1e-12 * max(1.0, abs(ref))
