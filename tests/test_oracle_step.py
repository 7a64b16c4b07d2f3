"""Pins of one full iteration of Algorithm 2 in the oracle: the OMD special
case (equation omd), the error-corrected sequence (Appendix B, equation
tilde), Lemma 1's per-step contraction, the server average's order."""
import numpy as np
import pytest

from conftest import load_golden
import synth
from synth.configs import custom


def _state(w, seed=0):
    W = synth.init_params_np(w)
    E = np.zeros((w.M, w.ld), np.float32)
    return W, E


def test_aggregate_order_golden(oracle_mod):
    g = load_golden("aggregate_order_example.txt")
    for ex in ("a", "b"):
        ph = np.array(g[ex + "_phat"], np.float32).reshape(4, 1)
        q = oracle_mod.aggregate(ph, 1)
        assert q[0] == np.float32(g[ex + "_qhat"][0])
        # the full iteration's server sum follows the same order: identity
        # compressor, zero error, eta = 1, one parameter
        w = custom(d=1, M=4, kind="identity", eta=1.0, seed=0, ld=1024)
        G = np.zeros((4, w.ld), np.float32)
        G[:, 0] = ph[:, 0]
        W = np.zeros(w.ld, np.float32)
        E = np.zeros((4, w.ld), np.float32)
        out = oracle_mod.step(w.as_dict(), np.float32(1.0), 1, G, E, W)
        assert out["qhat"][0] == np.float32(g[ex + "_qhat"][0])


def test_aggregate_divides_once_golden(oracle_mod):
    """M = 3: the average is the ascending sum divided once by M; the
    hand-derived value differs from the sum times the rounded 1/M."""
    g = load_golden("aggregate_mean_example.txt")
    ph = np.array(g["c_phat"], np.float32).reshape(3, 1)
    want = np.float32(g["c_qhat"][0])
    assert want != np.float32(g["c_reciprocal_qhat"][0])
    assert oracle_mod.aggregate(ph, 1)[0] == want
    w = custom(d=1, M=3, kind="identity", eta=1.0, seed=0, ld=1024)
    G = np.zeros((3, w.ld), np.float32)
    G[:, 0] = ph[:, 0]
    out = oracle_mod.step(w.as_dict(), np.float32(1.0), 1, G, np.zeros((3, w.ld), np.float32),
                          np.zeros(w.ld, np.float32))
    assert out["qhat"][0] == want


def test_step_quantizer_uses_row_index_counter(oracle_mod):
    """In the full iteration, element i of worker m (in whichever segment)
    rounds with the uniform of counter (i, m, t), drawn here from the
    pure-Python Philox reference (itself pinned to numpy's Philox), and the
    level follows equation (qsgd)'s rule in binary32."""
    from oracle import philox_ref
    seed, t = (7 | (2 << 32)), 3
    w = custom(d=300, M=2, kind="qsgd", levels=15, seg_offsets=[0, 100, 300], eta=1.0, seed=seed, ld=1024)
    rng = np.random.default_rng(31)
    G = np.zeros((2, w.ld), np.float32)
    G[:, :300] = rng.standard_normal((2, 300)).astype(np.float32)
    out = oracle_mod.step(w.as_dict(), np.float32(1.0), t, G, np.zeros((2, w.ld), np.float32),
                          np.zeros(w.ld, np.float32))
    s = np.float32(15)
    for m in range(2):
        words = out["level"][m]
        for j, (lo, hi) in enumerate(((0, 100), (100, 300))):
            inv = s / out["scale"][m, j]
            for i in range(lo, hi):
                lev = (int(words[i // 8]) >> (4 * (i % 8))) & 15   # 4-bit fields, low to high
                r = np.float32(abs(G[m, i]) * inv)  # p = fl(fl(1 * g) + 0) = g
                l = min(np.floor(r), s)
                frac = np.float32(0) if l == s else np.float32(r - l)
                u = philox_ref.uniform(seed, i, m, t)
                assert lev == min(int(l) + (1 if u < frac else 0), 15), (m, i)


@pytest.mark.parametrize("kind,norm,levels", [("sign", "l1", 0), ("qsgd", "l2", 15), ("qsgd", "linf", 15),
                                              ("qsgd", "l2", 255), ("mbit", "linf", 8), ("mbit", "l2", 4)])
def test_step_scales_follow_norm(oracle_mod, kind, norm, levels):
    """Each segment's scale in the full iteration is the norm the compressor
    names (equation qsgd's L2, the max norm of Section 2.4 / Appendix A, the
    mean magnitude of the scaled sign), checked with numpy's norms: the max
    exactly, the others to binary32 rounding of the binary64 value."""
    w = custom(d=500, M=3, kind=kind, levels=levels, norm=norm, seg_offsets=[0, 37, 300, 500], eta=1.0, seed=5,
               ld=1024)
    rng = np.random.default_rng(41)
    G = np.zeros((3, w.ld), np.float32)
    G[:, :500] = (rng.standard_normal((3, 500)) * np.exp(rng.uniform(-4, 0, (3, 500)))).astype(np.float32)
    out = oracle_mod.step(w.as_dict(), np.float32(1.0), 1, G, np.zeros((3, w.ld), np.float32),
                          np.zeros(w.ld, np.float32))
    for m in range(3):
        for j, (lo, hi) in enumerate(((0, 37), (37, 300), (300, 500))):
            p = G[m, lo:hi].astype(np.float64)  # p = fl(fl(1 * g) + 0) = g
            if norm == "linf":
                assert out["scale"][m, j] == np.float32(np.abs(p).max())
            elif norm == "l2":
                np.testing.assert_allclose(out["scale"][m, j], np.linalg.norm(p), rtol=1.2e-7)
            else:
                np.testing.assert_allclose(out["scale"][m, j], np.abs(p).mean(), rtol=1.2e-7)


def test_ef_accumulate_two_roundings(oracle_mod):
    """Reading of Algorithm 2's p = eta F + e: two binary32 roundings (the
    product, then the sum), no fused multiply-add.  numpy's binary32 ufuncs
    round each operation; the fused value, rounded once from double, differs
    on a sizeable fraction of random inputs."""
    rng = np.random.default_rng(21)
    g = rng.standard_normal(20000).astype(np.float32)
    e = (rng.standard_normal(20000) * 1e-3).astype(np.float32)
    eta = np.float32(1e-3)
    p = oracle_mod.ef_accumulate(eta, g, e)
    two = np.add(np.multiply(eta, g, dtype=np.float32), e, dtype=np.float32)
    np.testing.assert_array_equal(p, two)
    fused = (np.float64(eta) * g.astype(np.float64) + e.astype(np.float64)).astype(np.float32)
    assert np.count_nonzero(fused != p) > 100


def test_aggregate_close_to_exact_mean(oracle_mod):
    rng = np.random.default_rng(2)
    M, d = 16, 5000
    ph = rng.standard_normal((M, d)).astype(np.float32)
    q = oracle_mod.aggregate(ph, d)
    q64 = ph.astype(np.float64).mean(0)
    bound = M * 2.0 ** -24 * np.abs(ph.astype(np.float64)).mean(0)
    assert np.all(np.abs(q - q64) <= bound)


def test_identity_single_worker_is_omd(oracle_mod):
    """With Q = id (delta = 1) and M = 1 the evaluation points satisfy the one
    line OMD recurrence w_{t+1/2} = w_{t-1/2} - 2 eta F_t + eta F_{t-1}, and
    e stays 0 (Lemma 1 with delta = 1)."""
    w = custom(d=3000, M=1, kind="identity", eta=1e-2, seed=4)
    cfg = w.as_dict()
    W, E = _state(w)
    eta = np.float32(w.eta)
    g_prev = synth.gradients_np(w, 0)
    WX_prev = oracle_mod.extrapolate(eta, W[:w.d], g_prev[0, :w.d], E[0, :w.d])
    for t in range(1, 8):
        G = synth.gradients_np(w, t)
        out = oracle_mod.step(cfg, eta, t, G, E, W)
        assert np.all(out["E"] == 0)
        WX = out["WX"][0, :w.d].astype(np.float64)
        pred = WX_prev.astype(np.float64) - 2 * float(eta) * G[0, :w.d] + float(eta) * g_prev[0, :w.d]
        mag = np.maximum(np.abs(WX), np.abs(WX_prev)) + 2 * float(eta) * np.abs(G[0, :w.d])
        assert np.all(np.abs(WX - pred) <= 8 * 2.0 ** -24 * mag)
        WX_prev, g_prev = out["WX"][0, :w.d].copy(), G


@pytest.mark.parametrize("kind,extra", [("sign", {}), ("qsgd", {"levels": 15}), ("qsgd", {"levels": 255}),
                                        ("qsgd", {"levels": 15, "norm": "linf"}), ("topk", {"k": 97}),
                                        ("mbit", {"levels": 8, "norm": "linf"}), ("mbit", {"levels": 4, "norm": "l2"})])
def test_error_corrected_sequence(oracle_mod, kind, extra):
    """Appendix B, equation tilde: w~_t = w_t - (1/M) sum_m e_t^(m) obeys
    w~_t = w~_{t-1} - (eta/M) sum_m g_t^(m) for any compressor.  Checked in
    double against the oracle's binary32 state; the tolerance is the
    accumulated rounding of the binary32 operations."""
    d = 2053
    offs = [0, 700, 701, 2053] if kind != "topk" else [0, d]
    w = custom(d=d, M=4, kind=kind, seg_offsets=offs, eta=1e-2, seed=6, **extra)
    cfg = w.as_dict()
    W, E = _state(w)
    eta = float(np.float32(w.eta))
    wt = W[:d].astype(np.float64) - E[:, :d].astype(np.float64).mean(0)
    tol = np.zeros(d)
    u = 2.0 ** -24
    for t in range(1, 7):
        G = synth.gradients_np(w, t)
        P = np.abs(np.float32(w.eta) * G[:, :d]).astype(np.float64) + np.abs(E[:, :d])
        out = oracle_mod.step(cfg, np.float32(w.eta), t, G, E, W)
        wt = wt - eta * G[:, :d].astype(np.float64).mean(0)
        got = W[:d].astype(np.float64) - E[:, :d].astype(np.float64).mean(0)
        tol += 4 * u * (np.abs(W[:d]) + w.M * np.abs(out["qhat"]) + 4 * P.mean(0) + np.abs(E[:, :d]).mean(0))
        assert np.all(np.abs(got - wt) <= tol + 1e-30), (t, np.max(np.abs(got - wt) - tol))
        # the evaluation points w_{t+1/2}^(m) = w_t - (eta g_t + e_t) average
        # to the error-corrected point minus the mean step: w~_t - eta g_bar
        wx_mean = out["WX"][:, :d].astype(np.float64).mean(0)
        pred = wt - eta * G[:, :d].astype(np.float64).mean(0)
        wx_tol = tol + 4 * u * (np.abs(out["WX"][:, :d]).mean(0) + 2 * P.mean(0))
        assert np.all(np.abs(wx_mean - pred) <= wx_tol + 1e-30)


def test_lemma1_per_step_contraction(oracle_mod):
    """First line of Lemma 1's proof: ||e_t||^2 <= (1 - delta) ||p_t||^2, with
    delta = ||p||_1^2/(n ||p||_2^2) per segment for the scaled sign and
    delta = k/d for top-k."""
    d = 4000
    for kind, extra, offs in (("sign", {}, [0, 1500, 4000]), ("topk", {"k": 40}, [0, d])):
        w = custom(d=d, M=3, kind=kind, seg_offsets=offs, eta=1e-2, seed=8, **extra)
        cfg = w.as_dict()
        W, E = _state(w)
        for t in range(1, 5):
            G = synth.gradients_np(w, t)
            P = np.stack([oracle_mod.ef_accumulate(np.float32(w.eta), G[m, :d], E[m, :d]) for m in range(w.M)])
            oracle_mod.step(cfg, np.float32(w.eta), t, G, E, W)
            for m in range(w.M):
                for a, b in zip(offs[:-1], offs[1:]) if kind == "sign" else [(0, d)]:
                    p = P[m, a:b].astype(np.float64)
                    e2 = (E[m, a:b].astype(np.float64) ** 2).sum()
                    delta = (np.abs(p).sum() ** 2 / ((b - a) * (p ** 2).sum())) if kind == "sign" else 40 / d
                    assert e2 <= (1 - delta) * (p ** 2).sum() * (1 + 1e-6)


def test_teacher_forced_scales_reproduce(oracle_mod):
    w = custom(d=5000, M=4, kind="qsgd", levels=15, seg_offsets=[0, 1000, 5000], eta=1e-2, seed=9)
    cfg = w.as_dict()
    G = synth.gradients_np(w, 1)
    W1, E1 = _state(w)
    W2, E2 = W1.copy(), E1.copy()
    a = oracle_mod.step(cfg, np.float32(w.eta), 1, G, E1, W1)
    b = oracle_mod.step(cfg, np.float32(w.eta), 1, G, E2, W2, scales_in=a["scale"])
    for key in ("E", "W", "WX", "qhat", "sign", "level", "scale"):
        np.testing.assert_array_equal(a[key], b[key])


def test_bilinear_game_omd_contracts(oracle_mod):
    """Qualitative: on f(x, y) = x y (F = (y, -x)) plain gradient steps spiral
    out (Section 2.2), while the iteration of Algorithm 2 with Q = id and the
    gradient taken at the extrapolated point spirals in."""
    eta = np.float32(0.1)
    w = custom(d=2, M=1, kind="identity", eta=float(eta), seed=0, ld=1024)
    cfg = w.as_dict()
    W = np.zeros(w.ld, np.float32)
    W[:2] = [1.0, 1.0]
    E = np.zeros((1, w.ld), np.float32)
    F = lambda z: np.array([z[1], -z[0]], np.float32)
    G = np.zeros((1, w.ld), np.float32)
    G[0, :2] = F(W[:2])
    WX = oracle_mod.extrapolate(eta, W[:2], G[0, :2], E[0, :2])
    for t in range(1, 300):
        G = np.zeros((1, w.ld), np.float32)
        G[0, :2] = F(WX)
        out = oracle_mod.step(cfg, eta, t, G, E, W)
        WX = out["WX"][0, :2].copy()
    z = np.array([1.0, 1.0])
    for t in range(300):
        z = z - float(eta) * np.array([z[1], -z[0]])
    assert np.linalg.norm(W[:2]) < 0.5 * np.sqrt(2)
    assert np.linalg.norm(z) > 2 * np.sqrt(2)
