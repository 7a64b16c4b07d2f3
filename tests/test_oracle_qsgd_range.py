"""Pins of the s-level quantizer (equation qsgd) over the whole binary32
range of the segment norm.

Equation (qsgd) depends on v only through r_i = |v_i| s / ||v||, which does
not change when v is multiplied by a positive constant: Q(c v) = c Q(v) for
the same random draws.  A binary32 evaluation of fl(s / sigma) overflows
once sigma < s / FLT_MAX (about 4.4e-38 for s = 15), and fl(sigma / s) loses
significand bits once it is subnormal, so these pins put segments there:
exact-grid vectors whose levels and decoded values are fixed for every
draw, homogeneity against the same vector at a normal scale, levels that
bracket the exact r, and unbiasedness (the proof of Theorem 2, Appendix A)
on a segment of subnormal values.  A segment norm that binary32 cannot hold
(+inf) cannot be sent as the message's scale: the reading is that such a
segment sends level 0 everywhere and keeps p in its residual.
"""
import numpy as np
import pytest

TWO = np.float64(2.0)


def _exact_grid_cases():
    # (vector, norm, s, levels): |v_i| s / ||v|| is an integer for every i
    return [
        ([3.0, -4.0], "l2", 15, [9, 12]),
        ([3.0, -4.0], "l2", 255, [153, 204]),
        ([1.0, 3.0, -5.0], "linf", 15, [3, 9, 15]),
        ([1.0, 3.0, -5.0], "linf", 255, [51, 153, 255]),
    ]


@pytest.mark.parametrize("e2", [0, -60, -70, -100, -120, -126, -130, -140, -146])
def test_exact_grid_at_every_scale(oracle_mod, e2):
    """v = (3, -4) 2^e2 has ||v||_2 = 5 * 2^e2 exactly, levels (9, 12) for
    s = 15 and (153, 204) for s = 255, and Q(v) = v for every draw; likewise
    (1, 3, -5) 2^e2 under the max norm.  2^-146 puts v and sigma among the
    subnormals."""
    for base, norm, s, levels in _exact_grid_cases():
        v = (np.array(base) * TWO ** e2).astype(np.float32)
        assert np.array_equal(v.astype(np.float64), np.array(base) * TWO ** e2)  # exact
        sigma = oracle_mod.scale(v, norm)
        expect_sigma = (5.0 * TWO ** e2)
        assert float(sigma) == expect_sigma
        for t in range(12):
            bits, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, s, 77, 1, t)
            np.testing.assert_array_equal(lv, np.array(levels, np.uint16))
            np.testing.assert_array_equal(phat.view(np.uint32), v.view(np.uint32))
            assert np.all(e == 0)
            np.testing.assert_array_equal(bits, np.signbit(v).astype(np.uint8))
        # the server's decode of the same message
        dec = oracle_mod.decode_segment("qsgd", np.signbit(v).astype(np.uint16), np.array(levels), sigma, s)
        np.testing.assert_array_equal(dec.view(np.uint32), v.view(np.uint32))


def _short_vector(rng, n):
    """Values with 10 significant bits and magnitudes in [2^-5, 1): scaled by
    a power of two so that the norm is normal and at least 2^-126, every one
    of them stays exact."""
    mant = rng.integers(512, 1024, n).astype(np.float64) / 1024.0
    ex = rng.integers(-4, 0, n).astype(np.float64)
    sgn = np.where(rng.random(n) < 0.5, -1.0, 1.0)
    return (sgn * mant * TWO ** ex).astype(np.float32)


@pytest.mark.parametrize("s,norm", [(15, "l2"), (255, "l2"), (15, "linf"), (255, "linf"), (7, "linf")])
@pytest.mark.parametrize("target", [-126, -125, -110, -90, -70])
def test_homogeneous_in_the_scale(oracle_mod, s, norm, target):
    """Q(2^-k v) has the levels of Q(v) and decodes to fl(2^-k Q(v)), with
    2^-k sigma anywhere in the normal range: in particular where
    fl(s / sigma) overflows (2^-k sigma in [2^-126, 2^-125), s >= 15)."""
    rng = np.random.default_rng(1000 + s + 7 * abs(target))
    v = _short_vector(rng, 700)
    sigma = oracle_mod.scale(v, norm)
    k = int(np.floor(np.log2(float(sigma)))) - target
    vc = (v.astype(np.float64) * TWO ** -k).astype(np.float32)
    assert np.array_equal(vc.astype(np.float64), v.astype(np.float64) * TWO ** -k)
    sigma_c = oracle_mod.scale(vc, norm)
    assert float(sigma_c) == float(sigma) * TWO ** -k  # the norm scales exactly
    if target == -126 and s >= 15:
        assert float(s) / float(sigma_c) > 3.4028234663852886e38  # fl(s / sigma) overflows
    for t in range(4):
        _, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, s, 5, 3, t)
        _, lvc, phatc, ec = oracle_mod.qsgd_encode(vc, sigma_c, s, 5, 3, t)
        np.testing.assert_array_equal(lvc, lv)
        want = (phat.astype(np.float64) * TWO ** -k).astype(np.float32)
        np.testing.assert_array_equal(phatc.view(np.uint32), want.view(np.uint32))


def _subnormal_vector(rng, n):
    return (rng.standard_normal(n) * 1e-41).astype(np.float32)


@pytest.mark.parametrize("s,norm", [(15, "l2"), (255, "l2"), (15, "linf"), (127, "linf")])
def test_subnormal_segment_levels_bracket_exact_r(oracle_mod, s, norm):
    """Every level is floor(r) or floor(r) + 1 for the exact
    r = |v_i| s / sigma (computed in binary64 from the binary32 inputs)."""
    rng = np.random.default_rng(s)
    v = _subnormal_vector(rng, 2000)
    sigma = oracle_mod.scale(v, norm)
    assert 0.0 < float(sigma) < 2.0 ** -64
    r = np.abs(v.astype(np.float64)) * s / float(sigma)
    lo = np.floor(r * (1 - 2.0 ** -20))
    hi = np.minimum(np.floor(r * (1 + 2.0 ** -20)) + 1, s)
    seen_up = False
    for t in range(6):
        _, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, s, 11, 0, t)
        lvf = lv.astype(np.float64)
        assert np.all(lvf >= lo) and np.all(lvf <= hi)
        seen_up |= bool(np.any(lvf > np.floor(r)))
        # decoded magnitude: level * sigma / s, one subnormal ulp apart at most
        mag = lvf * float(sigma) / s
        assert np.all(np.abs(np.abs(phat.astype(np.float64)) - mag) <= 2.0 ** -149)
        # error feedback identity: p-hat + e = p exactly in this range
        assert np.array_equal((phat.astype(np.float64) + e.astype(np.float64)), v.astype(np.float64))
    assert seen_up


@pytest.mark.parametrize("s,norm", [(15, "l2"), (255, "l2"), (7, "linf")])
def test_subnormal_segment_unbiased(oracle_mod, s, norm):
    """E[Q(v)] = v (Appendix A, proof of Theorem 2) on a segment of
    subnormal values; the tolerance adds one subnormal ulp of rounding of the
    decoded value to six standard errors of the exact bin variance."""
    rng = np.random.default_rng(40 + s)
    v = _subnormal_vector(rng, 300)
    sigma = oracle_mod.scale(v, norm)
    N = 3000
    acc = np.zeros(v.size)
    for t in range(N):
        _, _, phat, _ = oracle_mod.qsgd_encode(v, sigma, s, 21, 2, t)
        acc += phat.astype(np.float64)
    mean = acc / N
    a = np.abs(v.astype(np.float64))
    step = float(sigma) / s
    rr = np.minimum(np.floor(a / step), s)
    var = (a - rr * step) * (np.minimum(rr + 1, s) * step - a)
    assert np.all(np.abs(mean - v.astype(np.float64)) <= 6 * np.sqrt(var / N) + 2.0 ** -149)
    assert abs(mean.sum() - v.astype(np.float64).sum()) <= 6 * np.sqrt(var.sum() / N) + v.size * 2.0 ** -149


def test_infinite_norm_sends_nothing(oracle_mod):
    """||v||_2 above FLT_MAX (finite elements): the scale is +inf, every
    level is 0, p-hat is a zero with the sign of p, and e = p;
    the server decodes the message to the same signed zeros."""
    v = np.array([1e38] * 16 + [-2e38, 0.0, -0.0, 3.0], np.float32)
    sigma = oracle_mod.scale(v, "l2")
    assert np.isinf(sigma) and sigma > 0
    for s in (15, 255, 7):
        bits, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, s, 3, 0, 1)
        assert np.all(lv == 0)
        np.testing.assert_array_equal(phat.view(np.uint32), (np.signbit(v).astype(np.uint32) << 31))
        # e = fl(p - (+-0)): p itself (a -0 element gives -0 - -0 = +0)
        np.testing.assert_array_equal(e, v)
        nz = v != 0
        np.testing.assert_array_equal(e[nz].view(np.uint32), v[nz].view(np.uint32))
        dec = oracle_mod.decode_segment("qsgd", bits.astype(np.uint16), lv, sigma, s)
        np.testing.assert_array_equal(dec.view(np.uint32), phat.view(np.uint32))


def test_infinite_norm_in_the_iteration(oracle_mod):
    """The same reading inside one whole iteration (Algorithm 2): the
    segment with the overflowing norm contributes zeros to the average, the
    other segment is quantized as usual, and every output is finite."""
    d, M = 40, 2
    ld = 1024
    G = np.zeros((M, ld), np.float32)
    G[:, :20] = 1e38
    G[:, 20:d] = np.linspace(-1, 1, 20, dtype=np.float32)
    E = np.zeros((M, ld), np.float32)
    W = np.zeros(ld, np.float32)
    cfg = dict(d=d, ld=ld, M=M, seg_offsets=[0, 20, d], kind="qsgd", norm="l2", levels=15, seed=9)
    out = oracle_mod.step(cfg, np.float32(1.0), 1, G, E, W)
    assert np.isinf(out["scale"][:, 0]).all() and np.isfinite(out["scale"][:, 1]).all()
    assert np.all(out["qhat"][:20] == 0)
    np.testing.assert_array_equal(out["E"][:, :20], G[:, :20])
    assert np.all(np.isfinite(out["qhat"])) and np.all(np.isfinite(out["WX"][:, :d]))
    assert np.any(out["qhat"][20:d] != 0)
