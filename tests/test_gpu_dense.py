"""GPU parity of the dense compressors (scaled sign, s-level quantizer,
identity) through the C ABI, against the oracle on the same inputs.

Teacher-forced: the oracle recomputes the iteration from the same pre-step
state with the GPU's segment scales; every message bit and every binary32
output must be identical.  The scales themselves must agree with the
oracle's own within 1e-5 relative."""
import numpy as np
import pytest

from gpu_common import GpuState, assert_same, compare_step, inputs, to_dev, u32
import synth
from synth.configs import custom

pytestmark = pytest.mark.gpu

CASES = {
    # name: workload
    "sign_2seg_m4": lambda: custom(d=5000, M=4, kind="sign", seg_offsets=[0, 1234, 5000], eta=1e-2, seed=1),
    "sign_tiny_segs_m2": lambda: custom(d=100, M=2, kind="sign", seg_offsets=[0, 1, 2, 3, 50, 99, 100], eta=1e-2,
                                        seed=2),
    "sign_d1_m1": lambda: custom(d=1, M=1, kind="sign", eta=1e-2, seed=3),
    "sign_d33_m3": lambda: custom(d=33, M=3, kind="sign", seg_offsets=[0, 31, 33], eta=1e-2, seed=4),
    "sign_c0": lambda: synth.get(0),
    "qsgd15_l2_m4": lambda: custom(d=5000, M=4, kind="qsgd", levels=15, seg_offsets=[0, 1234, 5000], eta=1e-2,
                                   seed=5),
    "qsgd15_l2_m32_many": lambda: custom(d=70001, M=32, kind="qsgd", levels=15,
                                         seg_offsets=[0, 64, 65, 1000, 4097, 30000, 65536, 70001], eta=1e-2, seed=6),
    "qsgd15_l2_m5_generic": lambda: custom(d=9000, M=5, kind="qsgd", levels=15, seg_offsets=[0, 4500, 9000],
                                           eta=1e-2, seed=7),
    "qsgd15_linf_m8": lambda: custom(d=20000, M=8, kind="qsgd", levels=15, norm="linf",
                                     seg_offsets=[0, 7, 19999, 20000], eta=1e-2, seed=8),
    "qsgd255_l2_m8": lambda: custom(d=3001, M=8, kind="qsgd", levels=255, seg_offsets=[0, 3001], eta=1e-2, seed=9),
    "qsgd255_linf_m16": lambda: custom(d=40000, M=16, kind="qsgd", levels=255, norm="linf",
                                       seg_offsets=[0, 100, 40000], eta=1e-2, seed=10),
    "qsgd255_m64_generic": lambda: custom(d=2048, M=64, kind="qsgd", levels=255, eta=1e-2, seed=11),
    "qsgd15_m17_masked": lambda: custom(d=6000, M=17, kind="qsgd", levels=15, seg_offsets=[0, 2999, 6000],
                                        eta=1e-2, seed=16),
    "sign_m33_masked": lambda: custom(d=4100, M=33, kind="sign", seg_offsets=[0, 64, 4100], eta=1e-2, seed=17),
    # 8 waves x 2 rows: an odd worker count leaves the last wave half empty and
    # the waves beyond it idle
    "qsgd255_m9_masked": lambda: custom(d=5000, M=9, kind="qsgd", levels=255, seg_offsets=[0, 1000, 5000],
                                        eta=1e-2, seed=23),
    "mbit8_m13_masked": lambda: custom(d=3333, M=13, kind="mbit", levels=8, norm="linf", seg_offsets=[0, 3333],
                                       eta=1e-2, seed=24),
    "topk_m11_masked": lambda: custom(d=7000, M=11, kind="topk", k=300, eta=1e-2, seed=25),
    "qsgd15_m65_split8": lambda: custom(d=3000, M=65, kind="qsgd", levels=15, eta=1e-2, seed=18),
    "sign_m128_split8": lambda: custom(d=2100, M=128, kind="sign", seg_offsets=[0, 100, 2100], eta=1e-2, seed=26),
    "mbit4_m100_split8": lambda: custom(d=1500, M=100, kind="mbit", levels=4, norm="linf", eta=1e-2, seed=27),
    # the largest worker count the library takes
    "sign_m1024_max": lambda: custom(d=1100, M=1024, kind="sign", seg_offsets=[0, 37, 1100], eta=1e-2, seed=29),
    "mbit4_m1024_d1": lambda: custom(d=1, M=1024, kind="mbit", levels=4, norm="linf", eta=1e-2, seed=30),
    "qsgd255_m130_one_lane": lambda: custom(d=1800, M=130, kind="qsgd", levels=255, seg_offsets=[0, 901, 1800],
                                            eta=1e-2, seed=28),
    "mbit8_linf_m4": lambda: custom(d=5000, M=4, kind="mbit", levels=8, norm="linf", seg_offsets=[0, 1234, 5000],
                                    eta=1e-2, seed=19),
    "mbit8_linf_m32_many": lambda: custom(d=70001, M=32, kind="mbit", levels=8, norm="linf",
                                          seg_offsets=[0, 64, 65, 1000, 4097, 30000, 65536, 70001], eta=1e-2, seed=20),
    "mbit4_l2_m16": lambda: custom(d=20000, M=16, kind="mbit", levels=4, norm="l2", seg_offsets=[0, 7, 19999, 20000],
                                   eta=1e-2, seed=21),
    "mbit4_linf_m5_generic": lambda: custom(d=9000, M=5, kind="mbit", levels=4, norm="linf", eta=1e-2, seed=22),
    "identity_m2": lambda: custom(d=4097, M=2, kind="identity", eta=1e-2, seed=12),
    "identity_m1": lambda: custom(d=1500, M=1, kind="identity", eta=1e-2, seed=13),
}


def _oracle(w, G, E, W, scales_in=None, t=1):
    from oracle import oracle as orc
    return orc.step(w.as_dict(), np.float32(w.eta), t, G, E.copy(), W.copy(), scales_in=scales_in)


@pytest.mark.parametrize("name", sorted(CASES))
def test_fused_step_teacher_forced(name):
    w = CASES[name]()
    G, E, W = inputs(w)
    print("case", name, "d", w.d, "M", w.M, flush=True)
    s = GpuState(w, G, E, W)
    s.fused(1)
    gpu = s.host()
    s.close()
    scales = gpu.get("scale")
    own = _oracle(w, G, E, W)
    if scales is not None:
        np.testing.assert_allclose(scales, own["scale"], rtol=1e-5, atol=0)
    ref = _oracle(w, G, E, W, scales_in=scales)
    compare_step(w, gpu, ref)
    # padding of E and W is preserved
    assert np.array_equal(gpu["E"][:, w.d:], E[:, w.d:]) and np.array_equal(gpu["W"][w.d:], W[w.d:])


@pytest.mark.parametrize("name", sorted(CASES))
def test_unfused_equals_fused(name):
    """dqgan_compress_ef + dqgan_aggregate + dqgan_omd_step give the fused
    step's results bit for bit."""
    w = CASES[name]()
    G, E, W = inputs(w)
    a = GpuState(w, G, E, W)
    a.fused(2)
    fa = a.host()
    a.close()
    b = GpuState(w, G, E, W)
    b.unfused(2)
    fb = b.host()
    b.close()
    compare_step(w, fa, fb)


@pytest.mark.parametrize("name", ["sign_2seg_m4", "qsgd15_l2_m4", "qsgd255_l2_m8", "qsgd15_l2_m32_many",
                                  "identity_m2", "sign_tiny_segs_m2", "mbit8_linf_m32_many", "mbit4_l2_m16"])
def test_unpack_matches_oracle_decode(name):
    """The server's decode of the message (dqgan_unpack) equals the oracle's
    decode of the same message planes."""
    w = CASES[name]()
    G, E, W = inputs(w)
    _unpack_vs_oracle(w, G, E, W)


def _unpack_vs_oracle(w, G, E, W):
    import torch
    from oracle import oracle as orc
    s = GpuState(w, G, E, W)
    s.dq.compress_ef(s.plan, w.eta, 3, s.G, s.E, None, s.wire)
    Ph = torch.full((w.M, w.ld), float("nan"), dtype=torch.float32, device=s.G.device)
    s.dq.unpack(s.plan, s.wire, Ph)
    torch.cuda.synchronize()
    got = Ph.cpu().numpy()
    out = s.host()
    s.close()
    b = {255: 8, 15: 4}.get(w.levels, 0)
    for m in range(w.M):
        if w.kind == "identity":
            exp = out["val"][m, :w.d]
        elif w.kind == "mbit":
            k = (1 << (w.levels - 1)) - 1
            signs, levels = orc.mbit_split(orc.unpack_bits(out["level"][m], w.levels, w.d), w.levels)
            exp = np.empty(w.d, np.float32)
            for j in range(w.n_seg):
                a0, a1 = w.seg_offsets[j], w.seg_offsets[j + 1]
                exp[a0:a1] = orc.decode_segment("qsgd", signs[a0:a1], levels[a0:a1], out["scale"][m, j], k)
        else:
            signs = orc.unpack_bits(out["sign"][m], 1, w.d)
            levels = orc.unpack_bits(out["level"][m], b, w.d) if b else np.zeros(w.d, np.uint16)
            exp = np.empty(w.d, np.float32)
            for j in range(w.n_seg):
                a0, a1 = w.seg_offsets[j], w.seg_offsets[j + 1]
                exp[a0:a1] = orc.decode_segment(w.kind, signs[a0:a1], levels[a0:a1], out["scale"][m, j], w.levels)
        assert_same("phat row %d" % m, got[m, :w.d], exp)
        assert np.all(got[m, w.d:] == 0)


@pytest.mark.parametrize("kind,levels", [("sign", 0), ("qsgd", 15), ("qsgd", 255), ("mbit", 8), ("mbit", 4)])
def test_pack_matches_oracle(kind, levels):
    import torch
    from oracle import oracle as orc
    w = custom(d=10007, M=3, kind=kind, levels=levels, seg_offsets=[0, 5000, 10007], seed=14)
    rng = np.random.default_rng(1)
    smax = ((1 << (levels - 1)) - 1) if kind == "mbit" else (levels if levels else 0)
    lv = rng.integers(0, smax + 1, (w.M, w.ld)).astype(np.uint16)
    sg = rng.integers(0, 2, (w.M, w.ld)).astype(np.uint16)
    codes = (sg << 15) | lv
    scales = rng.uniform(0.1, 1, (w.M, w.n_seg)).astype(np.float32)
    G, E, W = inputs(w)
    s = GpuState(w, G, E, W)
    ct = torch.from_numpy(codes.view(np.int16)).to(s.G.device)
    st = to_dev(scales)
    s.dq.pack(s.plan, ct, st, s.wire)
    torch.cuda.synchronize()
    out = s.host()
    s.close()
    b = {255: 8, 15: 4}.get(levels, 0)
    for m in range(w.M):
        if kind == "mbit":
            codes = orc.mbit_fields(sg[m, :w.d].astype(np.uint8), lv[m, :w.d], levels)
            assert_same("code words", out["level"][m], orc.pack_bits(codes, levels, w.ld * levels // 32))
            continue
        exp_s = orc.pack_bits(sg[m, :w.d], 1, w.ld // 32)
        assert_same("sign words", out["sign"][m], exp_s)
        if b:
            exp_l = orc.pack_bits(lv[m, :w.d], b, w.ld * b // 32)
            assert_same("level words", out["level"][m], exp_l)
    assert_same("scales", out["scale"], scales)


def test_zero_segment_quantizes_to_zero():
    """A segment whose p is identically zero has sigma = 0: every level is 0,
    p-hat = 0 and e = p (the oracle's reading of the undefined case)."""
    w = custom(d=3000, M=4, kind="qsgd", levels=15, seg_offsets=[0, 1000, 3000], eta=1e-2, seed=15)
    G, E, W = inputs(w)
    G[:, :1000] = 0.0
    E[:, :1000] = 0.0
    E[1, 5] = -0.0
    s = GpuState(w, G, E, W)
    s.fused(1)
    gpu = s.host()
    s.close()
    assert np.all(gpu["scale"][:, 0] == 0)
    ref = _oracle(w, G, E, W, scales_in=gpu["scale"])
    compare_step(w, gpu, ref)


def test_deterministic():
    w = CASES["qsgd15_l2_m32_many"]()
    G, E, W = inputs(w)
    outs = []
    for _ in range(2):
        s = GpuState(w, G, E, W)
        s.fused(4)
        outs.append(s.host())
        s.close()
    for k in outs[0]:
        assert np.array_equal(outs[0][k].view(np.uint32), outs[1][k].view(np.uint32)), k


PAD_CASES = {
    "sign_m20": lambda: custom(d=4001, M=20, kind="sign", seg_offsets=[0, 77, 4001], eta=1e-2, seed=51,
                               ld=4096 + 2048),
    "qsgd15_m3": lambda: custom(d=3000, M=3, kind="qsgd", levels=15, seg_offsets=[0, 1500, 3000], eta=1e-2,
                                seed=52, ld=3072 + 4096),
    "mbit8_m9": lambda: custom(d=2050, M=9, kind="mbit", levels=8, norm="linf", eta=1e-2, seed=53, ld=3072 + 1024),
    "topk_m3": lambda: custom(d=5000, M=3, kind="topk", k=100, eta=1e-2, seed=54, ld=5120 + 3072),
    "identity_m2": lambda: custom(d=999, M=2, kind="identity", eta=1e-2, seed=55, ld=1024 + 1024),
}


@pytest.mark.parametrize("name", sorted(PAD_CASES))
def test_padding_is_never_read(name):
    """Row strides with whole padding tiles beyond d, NaN in the padding of
    the gradients and sentinels in that of e and w: results on [0, d) equal
    the oracle's, the padding of E and W is untouched, that of WX and q-hat
    is written as 0."""
    w = PAD_CASES[name]()
    assert w.ld >= (w.d + 1023) // 1024 * 1024 + 1024
    G, E, W = inputs(w)
    G[:, w.d:] = np.nan
    E[:, w.d:] = 7.0
    W[w.d:] = -3.0
    print("case", name, "d", w.d, "ld", w.ld, "M", w.M, flush=True)
    s = GpuState(w, G, E, W)
    s.fused(1)
    gpu = s.host()
    s.close()
    ref = _oracle(w, G, E, W, scales_in=gpu.get("scale"))
    compare_step(w, gpu, ref)
    assert np.all(gpu["E"][:, w.d:] == 7.0) and np.all(gpu["W"][w.d:] == -3.0)


@pytest.mark.parametrize("kind,extra", [("sign", {}), ("qsgd", {"levels": 15}), ("qsgd", {"levels": 255, "norm": "linf"}),
                                        ("mbit", {"levels": 8, "norm": "linf"}), ("mbit", {"levels": 4, "norm": "l2"})])
def test_denormal_segment(kind, extra):
    """A segment whose p is subnormal (|p| ~ 1e-41, so s / sigma overflows
    binary32 for the quantizers and the 2^64-scaled evaluation of equation
    (qsgd) applies) next to a normal one: bit-exact against the oracle,
    subnormals kept."""
    w = custom(d=3000, M=4, kind=kind, seg_offsets=[0, 1000, 3000], eta=1.0, seed=61, group_scale=[1e-41, 1e-3],
               **extra)
    G, E, W = inputs(w, e_scale=0.0)
    assert np.abs(G[:, :1000]).max() < 1.2e-38 and np.count_nonzero(G[:, :1000]) > 3000
    print("case", kind, extra, flush=True)
    s = GpuState(w, G, E, W)
    s.fused(1)
    gpu = s.host()
    s.close()
    own = _oracle(w, G, E, W)
    np.testing.assert_allclose(gpu["scale"], own["scale"], rtol=1e-5, atol=0)
    ref = _oracle(w, G, E, W, scales_in=gpu["scale"])
    compare_step(w, gpu, ref)


# Segment scales across the binary32 range: subnormal p (sigma subnormal or
# tiny), sigma just above and below s / FLT_MAX (where fl(s / sigma)
# overflows), around 2^-64 (where the scaled evaluation starts), a normal
# segment, and one whose 2-norm exceeds FLT_MAX with finite elements (+inf
# scale: level 0, p-hat = +-0, e = p).
RANGE_SCALES = [1e-41, 3e-39, 2e-38, 1e-37, 1e-30, 5e-20, 1e-3, 2e37]
RANGE_OFFSETS = [0, 600, 1200, 1800, 2400, 3000, 3600, 4200, 5000]


@pytest.mark.parametrize("kind,extra", [("sign", {}), ("qsgd", {"levels": 15}), ("qsgd", {"levels": 255}),
                                        ("qsgd", {"levels": 255, "norm": "linf"}),
                                        ("mbit", {"levels": 8, "norm": "linf"}), ("mbit", {"levels": 4, "norm": "l2"})])
def test_norm_range_segments(kind, extra):
    """Fused step bit-exact against the oracle (teacher-forced), the separate
    worker and server calls equal to it, and the server's decode of the
    message equal to the oracle's."""
    w = custom(d=5000, M=4, kind=kind, seg_offsets=RANGE_OFFSETS, eta=1.0, seed=62, group_scale=RANGE_SCALES,
               **extra)
    G, E, W = inputs(w, e_scale=0.0)
    print("case", kind, extra, flush=True)
    a = GpuState(w, G, E, W)
    a.fused(1)
    gpu = a.host()
    a.close()
    own = _oracle(w, G, E, W)
    np.testing.assert_allclose(gpu["scale"], own["scale"], rtol=1e-5, atol=0)
    if w.norm == "l2":
        assert np.all(np.isinf(gpu["scale"][:, -1]))
    ref = _oracle(w, G, E, W, scales_in=gpu["scale"])
    compare_step(w, gpu, ref)
    assert np.all(np.isfinite(gpu["WX"][:, :w.d])) and np.all(np.isfinite(gpu["qhat"][:w.d]))
    b = GpuState(w, G, E, W)
    b.unfused(1)
    fb = b.host()
    b.close()
    compare_step(w, gpu, fb)
    _unpack_vs_oracle(w, G, E, W)
