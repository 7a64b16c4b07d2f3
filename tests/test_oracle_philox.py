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


_ROCRAND_PROBE = r"""
#include <cstdio>
#include <rocrand/rocrand_kernel.h>
// rocRAND's Philox4x32-10 block function (host-callable), made public
struct Engine : rocrand_device::philox4x32_10_engine {
    using rocrand_device::philox4x32_10_engine::ten_rounds;
};
int main() {
    Engine eng;
    unsigned c0, c1, c2, c3, k0, k1;
    while (std::scanf("%u %u %u %u %u %u", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        uint4 c; c.x = c0; c.y = c1; c.z = c2; c.w = c3;
        uint2 k; k.x = k0; k.y = k1;
        const uint4 r = eng.ten_rounds(c, k);
        std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
    }
    return 0;
}
"""


def test_c_oracle_matches_rocrand_philox4x32(oracle_mod, tmp_path):
    """The oracle's 32-bit instance against an implementation outside this
    repository: rocRAND's Philox4x32-10 block function (its multipliers,
    Weyl key increments and round order), run on the host."""
    import os
    import subprocess
    import pytest
    hipcc = "/opt/rocm/bin/hipcc"
    if not (os.path.exists(hipcc) and os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h")):
        pytest.skip("hipcc or rocRAND headers not installed")
    src = tmp_path / "rocrand_philox.cpp"
    exe = tmp_path / "rocrand_philox"
    src.write_text(_ROCRAND_PROBE)
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-o", str(exe), str(src)], check=True,
                   capture_output=True, timeout=300)
    rng = random.Random(4321)
    cases = [([rng.getrandbits(32) for _ in range(4)], [rng.getrandbits(32) for _ in range(2)]) for _ in range(3000)]
    for c in ([0, 0, 0, 0], [0xFFFFFFFF] * 4, [1, 0, 0, 0], [0, 0, 0, 1]):
        for k in ([0, 0], [0xFFFFFFFF, 0xFFFFFFFF], [0x9E3779B9, 0]):
            cases.append((c, k))
    stdin = "".join("%d %d %d %d %d %d\n" % (*c, *k) for c, k in cases)
    out = subprocess.run([str(exe)], input=stdin, capture_output=True, text=True, check=True, timeout=120).stdout
    got = [list(map(int, line.split())) for line in out.strip().splitlines()]
    assert len(got) == len(cases)
    for (c, k), r in zip(cases, got):
        assert oracle_mod.philox4x32_10(c, k) == r, (c, k)
