"""Pins of the scaled-sign compressor with error feedback (Section 2.4;
Definition 1; Algorithm 2)."""
import numpy as np
import pytest

from conftest import load_golden


def test_worked_example(oracle_mod):
    g = load_golden("sign_worked_example.txt")
    x = np.array(g["x"], np.float32)
    s = oracle_mod.scale(x, "l1")
    assert s == np.float32(g["scale"][0])
    bits, phat, e = oracle_mod.sign_encode(x, s)
    np.testing.assert_array_equal(phat, np.array(g["phat"], np.float32))
    np.testing.assert_array_equal(e, np.array(g["e"], np.float32))
    w = oracle_mod.pack_bits(bits, 1, 1)
    assert int(w[0]) == int(g["word"][0], 16)
    assert float((e.astype(np.float64) ** 2).sum()) == float(g["err2"][0])


@pytest.mark.parametrize("n", [1, 2, 7, 64, 1000, 4097])
def test_closed_form_error(oracle_mod, n):
    """||Q(x) - x||^2 = ||x||^2 - ||x||_1^2 / n for the mean-magnitude scale
    (so delta(x) = ||x||_1^2 / (n ||x||_2^2) in Definition 1)."""
    rng = np.random.default_rng(n)
    x = (rng.standard_normal(n) * rng.uniform(0.1, 10, n)).astype(np.float32)
    s = oracle_mod.scale(x, "l1")
    bits, phat, e = oracle_mod.sign_encode(x, s)
    x64 = x.astype(np.float64)
    lhs = ((x64 - phat.astype(np.float64)) ** 2).sum()
    rhs = (x64 ** 2).sum() - np.abs(x64).sum() ** 2 / n
    assert abs(lhs - rhs) <= 1e-9 * (x64 ** 2).sum() + 1e-30
    delta = np.abs(x64).sum() ** 2 / (n * (x64 ** 2).sum())
    assert 1.0 / n - 1e-12 <= delta <= 1.0 + 1e-12
    assert lhs <= (1 - delta) * (x64 ** 2).sum() * (1 + 1e-9) + 1e-30


def test_scale_is_mean_magnitude_in_double(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.standard_normal(100_000).astype(np.float32)
    s = oracle_mod.scale(x, "l1")
    ref = np.float32(np.abs(x.astype(np.float64)).sum() / x.size)
    assert s == ref


def test_constant_magnitude_is_exact(oracle_mod):
    x = np.array([0.75, -0.75, 0.75, 0.75, -0.75], np.float32)
    s = oracle_mod.scale(x, "l1")
    bits, phat, e = oracle_mod.sign_encode(x, s)
    np.testing.assert_array_equal(phat, x)
    assert np.all(e == 0)


def test_signed_zero_reading(oracle_mod):
    x = np.array([0.0, -0.0, 1.0, -1.0], np.float32)
    bits, phat, e = oracle_mod.sign_encode(x, np.float32(0.5))
    np.testing.assert_array_equal(bits, [0, 1, 0, 1])
    np.testing.assert_array_equal(phat, np.array([0.5, -0.5, 0.5, -0.5], np.float32))


def test_error_feedback_identity(oracle_mod):
    """e + p-hat reproduces p up to one rounding (Algorithm 2: e = p - p-hat)."""
    rng = np.random.default_rng(11)
    p = (rng.standard_normal(5000) * 1e-3).astype(np.float32)
    s = oracle_mod.scale(p, "l1")
    _, phat, e = oracle_mod.sign_encode(p, s)
    back = (e + phat).astype(np.float32)
    ulp = np.spacing(np.maximum(np.abs(p), np.abs(phat)))
    assert np.all(np.abs(back - p) <= ulp)
