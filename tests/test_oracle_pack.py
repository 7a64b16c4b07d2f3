"""Pins of the message layout (push of p-hat, Algorithm 2): sign plane and
4/8-bit level planes, LSB-first."""
import numpy as np
import pytest


def test_sign_bit_positions(oracle_mod):
    f = np.zeros(70, np.uint16)
    f[[0, 5, 31, 33, 69]] = 1
    w = oracle_mod.pack_bits(f, 1, 3)
    assert int(w[0]) == (1 << 0) | (1 << 5) | (1 << 31)
    assert int(w[1]) == (1 << 1)
    assert int(w[2]) == (1 << 5)


def test_level_positions(oracle_mod):
    f = np.array([1, 2, 3, 4, 5, 6, 7, 15, 9], np.uint16)
    w4 = oracle_mod.pack_bits(f, 4, 2)
    assert int(w4[0]) == 0xF7654321
    assert int(w4[1]) == 0x9
    f8 = np.array([0x11, 0xFF, 0x00, 0x80, 0x7F], np.uint16)
    w8 = oracle_mod.pack_bits(f8, 8, 2)
    assert int(w8[0]) == 0x8000FF11
    assert int(w8[1]) == 0x7F


@pytest.mark.parametrize("b", [1, 4, 8])
def test_roundtrip(oracle_mod, b):
    rng = np.random.default_rng(b)
    for n in (1, 31, 32, 33, 1000, 4096 + 3):
        f = rng.integers(0, 1 << b, n).astype(np.uint16)
        nw = (n * b + 31) // 32 + 2
        w = oracle_mod.pack_bits(f, b, nw)
        np.testing.assert_array_equal(oracle_mod.unpack_bits(w, b, n), f)
        # bits beyond the last element are zero
        assert int(w[-1]) == 0 and int(w[-2]) == 0
