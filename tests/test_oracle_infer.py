"""Pins of the oracle's packed-code and dequantized-product functions
(``oracle/infer.py``) against hand-worked values and plain definitions."""

import numpy as np
import pytest

from oracle import infer as oi


def test_pack_hand_worked_3bit():
    # codes 0..7 at 3 bits each: the word is sum_i i * 8^i = 0xFAC688
    p = oi.pack_codes(np.arange(8, dtype=np.uint8)[None, :], 3)
    assert p.shape == (1, 1) and int(p[0, 0]) == 0xFAC688
    # an eleventh code of value 7 straddles bits 30..32: two top bits of word
    # 0 and the lowest bit of word 1
    c = np.zeros((1, 11), dtype=np.uint8)
    c[0, 10] = 7
    p = oi.pack_codes(c, 3)
    assert p.shape == (1, 2) and int(p[0, 0]) == 0xC0000000 and int(p[0, 1]) == 1


@pytest.mark.parametrize("bits", range(1, 9))
def test_pack_round_trip(bits):
    rng = np.random.default_rng(bits)
    codes = rng.integers(0, 1 << bits, size=(5, 37), dtype=np.uint8)
    p = oi.pack_codes(codes, bits)
    assert p.shape == (5, oi.packed_words(37, bits))
    assert np.array_equal(oi.unpack_codes(p, 37, bits), codes)
    # bits past the last code are zero
    tail = 32 * p.shape[1] - 37 * bits
    if tail:
        assert np.all(p[:, -1] >> np.uint32(32 - tail) == 0)


def test_dequantize_rounds_to_nearest_even():
    s = np.float32(1.0 + 2.0 ** -11)       # exact in float32
    S = np.array([[s]], dtype=np.float32)
    Z = np.array([[4.0]], dtype=np.float32)
    w = oi.dequantize_fp16(np.array([[5, 7]], dtype=np.uint8), S, Z, 128)
    # 1 + 2^-11 is halfway between fp16 neighbours 1 and 1 + 2^-10: to even, 1
    assert w[0, 0] == np.float16(1.0)
    # 3 (1 + 2^-11) = 3 + 3 2^-11 lies nearer 3 + 2^-9 than 3
    assert w[0, 1] == np.float16(3.0 + 2.0 ** -9)


def test_dequant_matmul_is_the_plain_sum():
    rng = np.random.default_rng(3)
    W16 = rng.standard_normal((3, 5)).astype(np.float16)
    X16 = rng.standard_normal((5, 4)).astype(np.float16)
    Y = oi.dequant_matmul(W16, X16)
    for j in range(3):
        for t in range(4):
            ref = sum(float(W16[j, i]) * float(X16[i, t]) for i in range(5))
            assert abs(Y[j, t] - ref) <= 1e-15 * max(1.0, abs(ref))
    assert np.all(oi.summation_bound(W16, X16) >= 0)
