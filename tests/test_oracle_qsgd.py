"""Pins of the s-level stochastic quantizer (equation qsgd; Hou et al.'s
infinity-norm variant; unbiasedness and variance from the proof of Theorem 2
in Appendix A)."""
import numpy as np
import pytest

from conftest import load_golden


def _mc(oracle_mod, v, s, norm, N, seed=7):
    sigma = oracle_mod.scale(v, norm)
    acc = np.zeros(v.size, np.float64)
    acc2 = np.zeros(v.size, np.float64)
    err = np.zeros(N, np.float64)
    v64 = v.astype(np.float64)
    for t in range(N):
        _, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, s, seed, 3, t)
        q = phat.astype(np.float64)
        acc += q
        acc2 += q * q
        err[t] = ((q - v64) ** 2).sum()
    return sigma, acc / N, err


def _bin_variance(v, sigma, s):
    """(a - C_r)(C_{r+1} - a) with C_r = r sigma / s: the variance of Q(v_i)
    (Appendix A, with B_r = r/s)."""
    a = np.abs(v.astype(np.float64))
    step = float(sigma) / s
    r = np.minimum(np.floor(a / step), s)
    lo, hi = r * step, np.minimum(r + 1, s) * step
    return (a - lo) * (hi - a)


@pytest.mark.parametrize("s,norm", [(15, "l2"), (255, "l2"), (15, "linf"), (7, "linf"), (127, "linf")])
def test_unbiased_and_exact_variance(oracle_mod, s, norm):
    rng = np.random.default_rng(s)
    d = 600
    v = (rng.standard_normal(d) * np.exp(rng.uniform(-3, 0, d))).astype(np.float32)
    N = 4000
    sigma, mean, err = _mc(oracle_mod, v, s, norm, N)
    var = _bin_variance(v, sigma, s)
    v64 = v.astype(np.float64)
    bias_tol = 2.0 ** -20 * float(sigma)
    z = np.abs(mean - v64) - bias_tol
    assert np.all(z <= 6 * np.sqrt(var / N) + 1e-30)
    mask = var > 0
    chi2 = (((mean - v64)[mask]) ** 2 / (var[mask] / N)).sum()
    k = mask.sum()
    assert chi2 < k + 6 * np.sqrt(2 * k)
    # E||Q(v) - v||^2 = sum of the per-element bin variances
    expect = var.sum()
    assert abs(err.mean() - expect) <= 6 * err.std() / np.sqrt(N) + 1e-6 * expect


def test_delta_bound_under_sufficient_condition(oracle_mod):
    """With n < 4 s^2 every bin variance is at most (sigma/s)^2 / 4, so
    E||Q(v)-v||^2 <= n/(4 s^2) ||v||^2 and Definition 1 holds with
    delta = 1 - n/(4 s^2)."""
    s, n = 15, 500
    rng = np.random.default_rng(1)
    v = rng.standard_normal(n).astype(np.float32)
    N = 2000
    sigma, mean, err = _mc(oracle_mod, v, s, "l2", N)
    bound = n / (4 * s * s) * float((v.astype(np.float64) ** 2).sum())
    assert err.mean() <= bound


def test_zero_bin_breaks_per_element_inequality(oracle_mod):
    """Reading recorded in the design notes: in the r = 0 bin the per-element
    error a (C_1 - a) exceeds a^2 when 0 < a < C_1 / 2, so the per-element
    step of Theorem 2's proof cannot hold there.  Element 0 below sits at
    C_1 / 8."""
    s = 15
    v = np.array([15.0 / 8 / 15 * 1.0, 14.9], np.float32)  # a = C_1/8 with sigma ~ 14.9
    sigma = oracle_mod.scale(v, "l2")
    var = _bin_variance(v, sigma, s)
    assert var[0] > float(v[0]) ** 2


def test_exact_grid_is_deterministic(oracle_mod):
    g = load_golden("qsgd_exact_grid.txt")
    for key_v, key_l, s in (("s15_v", "s15_levels", 15), ("s255_v", "s255_levels", 255)):
        v = np.array(g[key_v], np.float32)
        sigma = oracle_mod.scale(v, "l2")
        for t in range(50):
            bits, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, s, 1, 0, t)
            np.testing.assert_array_equal(lv, np.array(g[key_l], np.uint16))
            np.testing.assert_array_equal(phat, v)
            assert np.all(e == 0)
            np.testing.assert_array_equal(bits, (v < 0).astype(np.uint8))
    v = np.array(g["linf_v"], np.float32)
    sigma = oracle_mod.scale(v, "linf")
    assert sigma == np.float32(g["linf_scale"][0])
    seen = set()
    for t in range(200):
        _, lv, phat, _ = oracle_mod.qsgd_encode(v, sigma, 15, 1, 0, t)
        assert lv[1] == int(g["linf_level2"][0]) and phat[1] == v[1]
        seen.add(int(lv[0]))
    assert seen == {11, 12}


def test_zero_segment_and_levels_in_range(oracle_mod):
    z = np.array([0.0, -0.0, 0.0], np.float32)
    bits, lv, phat, e = oracle_mod.qsgd_encode(z, np.float32(0.0), 15, 1, 0, 0)
    assert np.all(lv == 0)
    np.testing.assert_array_equal(e, z)
    np.testing.assert_array_equal(bits, [0, 1, 0])
    rng = np.random.default_rng(3)
    v = rng.standard_normal(4000).astype(np.float32)
    for s in (15, 255):
        for norm in ("l2", "linf"):
            sigma = oracle_mod.scale(v, norm)
            bits, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, s, 9, 1, 2)
            assert lv.max() <= s
            np.testing.assert_array_equal(bits, np.signbit(v).astype(np.uint8))
            back = (e + phat).astype(np.float32)
            assert np.all(np.abs(back - v) <= np.spacing(np.maximum(np.abs(v), np.abs(phat))))


def test_element_offset_selects_counter(oracle_mod):
    """Quantizing a segment that starts at row index i0 draws the uniforms of
    elements i0, i0+1, ... (the counter is the element's row index)."""
    rng = np.random.default_rng(8)
    v = rng.standard_normal(64).astype(np.float32)
    sigma = oracle_mod.scale(v, "l2")
    full = np.concatenate([np.zeros(37, np.float32), v])
    _, lv_a, _, _ = oracle_mod.qsgd_encode(v, sigma, 15, 5, 2, 9, i0=37)
    # element by element from the uniforms
    inv = np.float32(15) / sigma
    for j in range(64):
        r = np.float32(abs(v[j]) * inv)
        l = min(np.floor(r), 15)
        frac = 0.0 if l == 15 else r - l
        u = oracle_mod.uniform(5, 37 + j, 2, 9)
        assert lv_a[j] == min(int(l) + (1 if u < frac else 0), 15)
