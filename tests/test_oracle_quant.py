"""Pins for the INT8 codec oracle (App. E.1, Eq. 10), CPU only."""

import numpy as np

from oracle import quant as Q

F32 = np.float32


def test_error_bound_and_range():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal((50, 128)) * rng.uniform(1e-6, 10, size=(50, 1))).astype(F32)
    q, s = Q.quantize_rows(x)
    assert q.dtype == np.int8 and s.dtype == F32
    assert np.all(np.abs(q.astype(int)) <= 127)
    # every row's largest magnitude maps to +-127
    np.testing.assert_array_equal(np.abs(q).max(axis=1), 127)
    err = np.abs(Q.dequantize_rows(q, s) - x)
    assert np.all(err <= s[:, None] * (0.5 + 1e-5))


def test_exact_multiples_round_trip():
    rng = np.random.default_rng(1)
    q0 = rng.integers(-127, 128, size=(7, 64)).astype(np.int8)
    q0[:, 0] = 127                                  # row max magnitude 127
    step = F32(2.0 ** -7)                           # a = 127 * 2^-7 -> s = 2^-7 exactly
    x = q0.astype(F32) * step
    q, s = Q.quantize_rows(x)
    np.testing.assert_array_equal(s, step)
    np.testing.assert_array_equal(q, q0)
    np.testing.assert_array_equal(Q.dequantize_rows(q, s), x)


def test_round_half_to_even_and_symmetry():
    step = F32(2.0 ** -7)
    x = np.zeros((1, 8), dtype=F32)
    x[0, 0] = 127 * step
    x[0, 1:5] = np.array([2.5, 3.5, -2.5, 0.5], dtype=F32) * step
    q, _ = Q.quantize_rows(x)
    np.testing.assert_array_equal(q[0, 1:5], [2, 4, -2, 0])
    qn, sn = Q.quantize_rows(-x)
    np.testing.assert_array_equal(qn, -q)


def test_zero_row():
    q, s = Q.quantize_rows(np.zeros((2, 16), dtype=F32))
    assert np.all(q == 0)
    np.testing.assert_array_equal(s, np.maximum(F32(0), F32(1e-8)) / F32(127))
    np.testing.assert_array_equal(Q.dequantize_rows(q, s), 0)


def test_pack_restore_q8_matches_rowwise_codec():
    rng = np.random.default_rng(2)
    states = rng.standard_normal((3, 20, 16)).astype(F32)
    unit_row = np.array([1, 4, 5, 9, 19])
    q, s = Q.pack_q8(states, [2, 0], unit_row)
    q2, s2 = Q.quantize_rows(states[[2, 0]][:, unit_row])
    np.testing.assert_array_equal(q, q2)
    np.testing.assert_array_equal(s, s2)
    out = Q.restore_q8(q, s, unit_row, 20)
    mask = np.zeros(20, bool)
    mask[unit_row] = True
    assert np.all(out[:, ~mask] == 0)
    assert np.all(np.abs(out[:, mask] - states[[2, 0]][:, mask]) <= s[..., None] * 0.5001)
