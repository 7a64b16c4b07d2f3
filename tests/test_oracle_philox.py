"""Pins of the oracle's counter-based generator (Philox4x32-10, Salmon et al.
SC'11) and of the uniforms the stochastic quantizer draws from it."""
import random

import numpy as np

from oracle import philox_ref


def test_reference_structure_matches_numpy_philox4x64():
    """The pure-Python Philox is generic over the word width.  Its 64-bit
    instance must reproduce numpy's Philox4x64-10 bit generator exactly: this
    pins the round function, the key schedule and the output order
    independently of any code in this repository."""
    for key in ([0, 0], [123456789, 987654321], [2**64 - 1, 2**63 + 5]):
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64))
        raw = [int(x) for x in bg.random_raw(16)]
        ctr = [0, 0, 0, 0]
        mine = []
        for _ in range(4):
            ctr[0] += 1  # numpy advances the counter before each block
            mine += philox_ref.philox4(ctr, key, width=64, rounds=10)
        assert mine == raw


def test_c_oracle_matches_reference_4x32(oracle_mod):
    rng = random.Random(1234)
    for _ in range(5000):
        c = [rng.getrandbits(32) for _ in range(4)]
        k = [rng.getrandbits(32) for _ in range(2)]
        assert oracle_mod.philox4x32_10(c, k) == philox_ref.philox4(c, k, 32, 10)
    # edge counters and keys
    for c in ([0, 0, 0, 0], [0xFFFFFFFF] * 4, [1, 0, 0, 0], [0, 0, 0, 1]):
        for k in ([0, 0], [0xFFFFFFFF, 0xFFFFFFFF]):
            assert oracle_mod.philox4x32_10(c, k) == philox_ref.philox4(c, k, 32, 10)


def test_uniform_counter_layout(oracle_mod):
    rng = random.Random(99)
    for _ in range(3000):
        seed = rng.getrandbits(64)
        i = rng.getrandbits(36)
        m = rng.randrange(0, 128)
        t = rng.getrandbits(32)
        u = oracle_mod.uniform(seed, i, m, t)
        assert u == philox_ref.uniform(seed, i, m, t)
        assert 0.0 <= u < 1.0


def test_uniforms_statistics(oracle_mod):
    """Mean, a 256-bin chi-square and the lag-1 correlation of 2^16 uniforms
    of consecutive elements (the draw order of one row)."""
    n = 1 << 16
    seed = 3 | (2 << 32)
    u = np.array([oracle_mod.uniform(seed, i, 5, 7) for i in range(n)], dtype=np.float64)
    assert abs(u.mean() - 0.5) < 6 * np.sqrt(1 / 12 / n)
    counts = np.bincount((u * 256).astype(int), minlength=256)
    exp = n / 256
    chi2 = ((counts - exp) ** 2 / exp).sum()
    # 255 degrees of freedom: mean 255, sd ~22.6; 6 sd bound
    assert chi2 < 255 + 6 * 22.6
    c = np.corrcoef(u[:-1], u[1:])[0, 1]
    assert abs(c) < 6 / np.sqrt(n)
    # 24-bit grid
    assert np.all(u * (1 << 24) == np.floor(u * (1 << 24)))
