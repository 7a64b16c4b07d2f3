"""Seeded random shapes through the C ABI against the oracle (teacher-forced,
bit-exact): every compressor, worker counts 1..140 (every launch shape of the fused
kernel), lengths 1..60000 with ragged tails, random segment layouts down to
one-element segments, random step sizes and residual magnitudes."""
import numpy as np
import pytest

from gpu_common import GpuState, compare_step
from synth.configs import custom

pytestmark = pytest.mark.gpu

KINDS = [("sign", {}), ("qsgd", {"levels": 15}), ("qsgd", {"levels": 255}), ("qsgd", {"levels": 15, "norm": "linf"}),
         ("qsgd", {"levels": 255, "norm": "linf"}), ("mbit", {"levels": 8, "norm": "linf"}),
         ("mbit", {"levels": 4, "norm": "l2"}), ("topk", {}), ("identity", {})]


def _random_case(seed):
    rng = np.random.default_rng(1000 + seed)
    kind, extra = KINDS[seed % len(KINDS)]
    extra = dict(extra)
    d = int(rng.integers(1, 60001)) if seed % 3 else int(rng.integers(1, 300))
    M = int(rng.choice([1, 2, 3, 4, 7, 8, 16, 17, 31, 32, 33, 64, 70, 100, 140]))
    if kind == "topk":
        M = min(M, 64)
        extra["k"] = int(rng.integers(1, d + 1)) if seed % 4 else max(1, d // 100)
        offs = [0, d]
    else:
        nseg = int(rng.integers(1, min(d, 12) + 1))
        cuts = sorted(set(int(x) for x in rng.integers(1, d, size=nseg - 1))) if d > 1 else []
        offs = [0] + cuts + [d]
    eta = float(10 ** rng.uniform(-4, -1))
    w = custom(d=d, M=M, kind=kind, seg_offsets=offs, eta=eta, seed=seed, law="laplace" if seed % 2 else "normal",
               **extra)
    return w, float(10 ** rng.uniform(-6, -2))


@pytest.mark.parametrize("seed", range(27))
def test_random_shape_matches_oracle(seed):
    from gpu_common import inputs
    from oracle import oracle as orc
    w, e_scale = _random_case(seed)
    print("seed", seed, w.kind, "d", w.d, "M", w.M, "segs", w.n_seg, "k", w.k, flush=True)
    G, E, W = inputs(w, t=1, e_scale=e_scale, seed=seed)
    s = GpuState(w, G, E, W)
    s.fused(3)
    gpu = s.host()
    s.close()
    scales = gpu.get("scale") if w.kind in ("sign", "qsgd", "mbit") else None
    ref = orc.step(w.as_dict(), np.float32(w.eta), 3, G, E.copy(), W.copy(), scales_in=scales)
    if scales is not None:
        own = orc.step(w.as_dict(), np.float32(w.eta), 3, G, E.copy(), W.copy())
        np.testing.assert_allclose(scales, own["scale"], rtol=1e-5, atol=0)
    compare_step(w, gpu, ref)
