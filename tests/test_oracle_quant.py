"""Pins of the oracle's block-scaled 8-bit quantiser (CPU only): a block worked out
by hand, ties, a scale that must round to half precision, the zero block, the
bounds every block satisfies, and the scalar-loop form against the vectorised one."""

from __future__ import annotations

import numpy as np
import pytest

from oracle import dequantize_q8, quantize_q8, quantize_q8_loops


def test_hand_block_with_exact_scale():
    # amax = 127 * 2^-7, so the scale is exactly 2^-7 and w = k * 2^-7 maps to k
    k = np.array([127, -127, 0, 1, -1, 64, -100, 3] + [5] * 24, np.float32)
    w = (k * np.float32(2.0 ** -7))[None, :]
    q, d = quantize_q8(w)
    assert d.dtype == np.float16 and float(d[0, 0]) == 2.0 ** -7
    assert q.tolist()[0] == k.astype(int).tolist()
    assert np.array_equal(dequantize_q8(q, d), w.astype(np.float64))


def test_ties_round_to_even():
    base = [127.0] + [0.0] * 31                     # fixes the scale at 2^-7
    for val, code in [(2.5, 2), (3.5, 4), (-2.5, -2), (-3.5, -4), (0.5, 0), (1.5, 2)]:
        row = np.array(base, np.float32)
        row[1] = val
        q, _ = quantize_q8((row * np.float32(2.0 ** -7))[None, :])
        assert q[0, 1] == code, (val, q[0, 1])


def test_scale_rounds_to_half_precision():
    # amax = 1: s = 1/127 in float32; the nearest half (ulp 2^-17 there) is 1032 * 2^-17
    w = np.zeros((1, 32), np.float32)
    w[0, 0] = 1.0
    w[0, 1] = -0.5
    q, d = quantize_q8(w)
    assert float(d[0, 0]) == 1032 * 2.0 ** -17
    # 1 / d = 127.0078 -> 127;  0.5 / d = 63.50 -> 64 (63.5039 rounds up)
    assert q[0, 0] == 127 and q[0, 1] == -64


def test_zero_block_and_tiny_block():
    w = np.zeros((2, 64), np.float32)
    w[1, 40] = 1e-9                                 # s = 7.9e-12 rounds to a zero half
    q, d = quantize_q8(w)
    assert not q.any() and not d.astype(np.float32).any()


def test_bounds_on_random_rows():
    rng = np.random.default_rng(5)
    w = (rng.standard_normal((64, 512)) * 0.02).astype(np.float32)
    w[3, :32] *= 50.0                               # one block with large weights
    q, d = quantize_q8(w)
    d32 = d.astype(np.float32)
    assert np.abs(q.astype(int)).max() <= 127
    # the largest weight of every block lands on +-127
    qb = np.abs(q.astype(int)).reshape(64, 16, 32).max(axis=2)
    assert np.all(qb == 127)
    # every weight within half a quantum of its code (plus float32 rounding of w/d)
    err = np.abs(dequantize_q8(q, d) - w.astype(np.float64))
    bound = np.repeat(d32.astype(np.float64), 32, axis=1) * (0.5 + 1e-6)
    assert np.all(err <= bound)
    # the scale is the half-precision rounding of amax / 127 (relative 2^-11)
    amax = np.abs(w).reshape(64, 16, 32).max(axis=2).astype(np.float64)
    assert np.all(np.abs(d32 - amax / 127) <= amax / 127 * 2.0 ** -11 * 1.0001)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_scalar_loops_match_vectorised(seed):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((4, 96)) * 0.05).astype(np.float32)
    w[0, :32] = 0.0                                 # zero block
    w[1, 32:64] *= 1e-5                             # half-precision subnormal scale
    w[2, 64:96] = np.round(w[2, 64:96] * 1000) / 1000
    q1, d1 = quantize_q8(w)
    q2, d2 = quantize_q8_loops(w)
    assert np.array_equal(q1, q2)
    assert np.array_equal(d1.view(np.uint16), d2.view(np.uint16))


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        quantize_q8(np.zeros((1, 33), np.float32))
    w = np.zeros((1, 32), np.float32)
    w[0, 3] = np.inf
    with pytest.raises(ValueError):
        quantize_q8(w)
