"""Message planes larger than the Infinity Cache (256 MiB): the fused pass
writes them with gathered 128-bit streaming stores, smaller ones with
cache-allocating stores (every other parity test).  One shape per packed
field width, M = 16 (two rows per wave), each with a plane past the
threshold: the s = 255 and s = 15 quantizers and the 8-bit and 4-bit
sign-magnitude codes.

The iteration is checked against the oracle, teacher-forced with the GPU's
segment scales, on windows at the start of the row, across a segment
boundary, in the middle and at the ragged end; the scales of the sampled
segments against the oracle's own within 1e-5.  Inputs are drawn on the
device; only windows are copied to the host.
"""
import numpy as np
import pytest

from gpu_common import assert_same
from synth.configs import custom

pytestmark = pytest.mark.gpu

CASES = [
    # kind, levels (QSGD s / MBIT m), norm, d: message bytes 16 * ld * bits / 8 > 256 MiB
    ("qsgd", 255, "l2", 20_000_003),   # 9 bits per element: 360 MB
    ("qsgd", 15, "l2", 30_000_001),    # 5 bits: 300 MB
    ("mbit", 8, "linf", 20_000_005),   # 8 bits: 320 MB
    ("mbit", 4, "l2", 40_000_007),     # 4 bits: 320 MB
]


@pytest.fixture(autouse=True)
def _release_memory():
    yield
    import gc
    import torch
    gc.collect()
    torch.cuda.empty_cache()


def _words(plane_row, a, b, bits):
    """The words that hold elements [a, b) (a is a multiple of 32)."""
    per = 32 // bits
    return plane_row[a // per:(b + per - 1) // per].cpu().numpy().view(np.uint32)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s%d" % (c[0], c[1]))
def test_streamed_plane_windows(case):
    import torch
    from oracle import oracle as orc
    from paper_2010_13359_amd import dqgan
    kind, levels, norm, d = case
    M = 16
    offs = [0, 4_000_003, d - 50_000, d]
    w = custom(d=d, M=M, kind=kind, levels=levels, norm=norm, seg_offsets=offs, eta=1e-3, seed=41)
    bits = (9 if levels == 255 else 5) if kind == "qsgd" else levels
    assert M * w.ld * bits / 8 > 256 * 2 ** 20
    print("streamed plane %s %d: d=%d" % (kind, levels, d), flush=True)
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(41)
    G = torch.zeros((M, w.ld), dtype=torch.float32, device=dev)
    E = torch.zeros_like(G)
    W = torch.zeros(w.ld, dtype=torch.float32, device=dev)
    G[:, :d].normal_(0.0, 1.0, generator=gen)
    E[:, :d].normal_(0.0, 1e-3, generator=gen)
    W[:d].normal_(0.0, 0.02, generator=gen)
    E0, W0 = E.clone(), W.clone()
    plan = dqgan.Plan.from_workload(w)
    WX = torch.empty_like(G)
    wire = plan.new_wire(dev)
    t = 3
    dqgan.step_fused(plan, w.eta, t, G, E, W, WX, wire)
    torch.cuda.synchronize()
    scales = wire.scale.view(M, w.n_seg).cpu().numpy()
    mbit = kind == "mbit"
    k_levels = (1 << (levels - 1)) - 1 if mbit else levels
    sign_rows = None if mbit else wire.sign.view(M, -1)
    level_rows = wire.level.view(M, -1)
    eta = np.float32(w.eta)
    # the sampled segments' scales against the oracle's own
    for j in (0, 2):
        a, b = offs[j], offs[j + 1]
        for m in (0, M - 1):
            p = orc.ef_accumulate(eta, G[m, a:b].cpu().numpy(), E0[m, a:b].cpu().numpy())
            own = float(orc.scale(p, w.norm))
            assert abs(float(scales[m, j]) - own) <= 1e-5 * own, (j, m, float(scales[m, j]), own)
    windows = [(0, 8192), (offs[1] // 32 * 32 - 4096, offs[1] // 32 * 32 + 4096), (d // 2 // 32 * 32, d // 2 // 32 * 32 + 8192),
               (d // 32 * 32 - 8192, d)]
    for a, b in windows:
        n = b - a
        Gs = G[:, a:b].cpu().numpy()
        Es = E0[:, a:b].cpu().numpy()
        Ws = W0[a:b].cpu().numpy()
        phat = np.empty((M, n), np.float32)
        enew = np.empty((M, n), np.float32)
        for m in range(M):
            p = orc.ef_accumulate(eta, Gs[m], Es[m])
            # the window may straddle a segment boundary: encode each part with its scale
            for j in range(w.n_seg):
                lo, hi = max(a, offs[j]), min(b, offs[j + 1])
                if lo >= hi:
                    continue
                sb, lv, ph, e = orc.qsgd_encode(p[lo - a:hi - a], scales[m, j], k_levels, w.quant_seed, m, t, i0=lo)
                phat[m, lo - a:hi - a], enew[m, lo - a:hi - a] = ph, e
                if mbit:
                    codes = orc.unpack_bits(_words(level_rows[m], a, b, levels), levels, b - a)[lo - a:hi - a]
                    assert_same("codes [%d,%d) row %d" % (lo, hi, m), codes, orc.mbit_fields(sb, lv, levels))
                else:
                    gs = orc.unpack_bits(_words(sign_rows[m], a, b, 1), 1, b - a)[lo - a:hi - a]
                    gl = orc.unpack_bits(_words(level_rows[m], a, b, 8 if levels == 255 else 4),
                                         8 if levels == 255 else 4, b - a)[lo - a:hi - a]
                    assert_same("sign bits [%d,%d) row %d" % (lo, hi, m), gs, sb.astype(np.uint16))
                    assert_same("levels [%d,%d) row %d" % (lo, hi, m), gl, lv)
        assert_same("e_t [%d,%d)" % (a, b), E[:, a:b].cpu().numpy(), enew)
        q = orc.aggregate(phat, n)
        wt = orc.omd_update(q, Ws)
        assert_same("w_t [%d,%d)" % (a, b), W[a:b].cpu().numpy(), wt)
        wx = np.stack([orc.extrapolate(eta, wt, Gs[m], enew[m]) for m in range(M)])
        assert_same("WX [%d,%d)" % (a, b), WX[:, a:b].cpu().numpy(), wx)
    plan.close()
