"""Pins of the oracle's 4-bit dequantisation (GPTQ-style symmetric groups,
w = s (q - 8); the paper's INT4 targets, §4.1)."""

import numpy as np
import pytest

from oracle import quant


def test_nibble_order_hand_worked():
    # byte 0x21: input 0 -> code 1 (low nibble), input 1 -> code 2
    assert quant.unpack_codes(np.array([[0x21, 0xF0]], dtype=np.uint8)).tolist() == [[1, 2, 0, 15]]


def test_dequantize_hand_worked():
    # two rows, four inputs, groups of two: scales per (row, group)
    codes = np.array([[8, 9, 0, 15], [7, 8, 12, 4]])
    scales = np.array([[0.5, 2.0], [0.25, -1.0]])
    want = np.array([[0.0, 0.5, -16.0, 14.0], [-0.25, 0.0, -4.0, 4.0]])
    np.testing.assert_array_equal(quant.dequantize(codes, scales, 2), want)


def test_closed_forms_and_invariants():
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 16, size=(6, 256))
    scales = rng.uniform(0.5, 2.0, size=(6, 2))
    w = quant.dequantize(codes, scales, 128)
    # the zero point is 8: code 8 stands for 0 whatever the scale
    assert np.all(w[codes == 8] == 0.0)
    # codes mirrored about the zero point give the negated weight
    mirrored = np.where(codes > 0, 16 - codes, codes)
    wm = quant.dequantize(mirrored, scales, 128)
    on = codes > 0
    np.testing.assert_array_equal(wm[on], -w[on])
    # linear in the scales, and a scale reaches exactly its own group
    s2 = scales.copy()
    s2[3, 1] *= 3.0
    w2 = quant.dequantize(codes, s2, 128)
    changed = np.nonzero(w2 != w)
    assert set(changed[0].tolist()) <= {3} and set(changed[1].tolist()) <= set(range(128, 256))
    np.testing.assert_allclose(w2[3, 128:], 3.0 * w[3, 128:], rtol=0, atol=0)
    # the largest magnitude a code reaches is 8 s (code 0), the largest positive 7 s (code 15)
    assert quant.dequantize(np.zeros((1, 128), int), np.array([[0.25]]), 128).min() == -2.0
    assert quant.dequantize(np.full((1, 128), 15), np.array([[0.25]]), 128).max() == 1.75


def test_round_trip_of_bytes():
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 16, size=(4, 64))
    packed = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    np.testing.assert_array_equal(quant.unpack_codes(packed), codes)


def test_shape_mismatch_is_refused():
    with pytest.raises(ValueError):
        quant.dequantize(np.zeros((2, 100), int), np.ones((2, 1)), 128)
