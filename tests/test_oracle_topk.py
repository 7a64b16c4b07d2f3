"""Pins of the top-k sparsifier (Section 2.4; Theorem 1 and its proof)."""
import itertools

import numpy as np
import pytest

from conftest import load_golden


def test_worked_example(oracle_mod):
    g = load_golden("topk_worked_example.txt")
    x = np.array(g["x"], np.float32)
    for k in (3, 4):
        idx, val, phat, e = oracle_mod.topk(x, k)
        np.testing.assert_array_equal(idx, np.array(g["k%d_idx" % k], np.uint32))
        np.testing.assert_array_equal(val, np.array(g["k%d_val" % k], np.float32))
        np.testing.assert_array_equal(e, np.array(g["k%d_e" % k], np.float32))


def _brute(x, k):
    order = sorted(range(len(x)), key=lambda i: (-abs(float(x[i])), i))
    return sorted(order[:k])


def test_brute_force_with_ties(oracle_mod):
    rng = np.random.default_rng(0)
    vocab = np.array([0.0, 1.0, -1.0, 2.5, -2.5, 0.5], np.float32)
    for d in range(1, 65):
        for _ in range(4):
            x = vocab[rng.integers(0, vocab.size, d)]
            k = int(rng.integers(1, d + 1))
            idx, val, phat, e = oracle_mod.topk(x, k)
            assert list(idx) == _brute(x, k)
            np.testing.assert_array_equal(val, x[idx])
            sel = np.zeros(d, bool)
            sel[idx] = True
            assert np.all(e[sel] == 0) and np.array_equal(e[~sel], x[~sel])
            np.testing.assert_array_equal(phat[sel], x[sel])
            assert np.all(phat[~sel] == 0)


@pytest.mark.parametrize("d,k", [(10, 1), (1000, 10), (4096, 4096), (5000, 1234)])
def test_contraction(oracle_mod, d, k):
    """Theorem 1: ||x - topk(x)||^2 <= (1 - k/d) ||x||^2, deterministically."""
    rng = np.random.default_rng(d + k)
    x = (rng.standard_normal(d) * np.exp(rng.uniform(-5, 0, d))).astype(np.float32)
    idx, val, phat, e = oracle_mod.topk(x, k)
    x64 = x.astype(np.float64)
    lhs = ((x64 - phat) ** 2).sum()
    assert lhs <= (1 - k / d) * (x64 ** 2).sum() * (1 + 1e-12)
    assert np.all(np.diff(idx.astype(np.int64)) > 0)


def test_all_permutations_small(oracle_mod):
    base = np.array([3.0, -3.0, 1.0, 0.0, -1.0], np.float32)
    for perm in itertools.permutations(range(5)):
        x = base[list(perm)]
        for k in range(1, 6):
            idx, *_ = oracle_mod.topk(x, k)
            assert list(idx) == _brute(x, k)
