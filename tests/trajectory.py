"""Helpers of the full-trajectory GPU parity tests.

`encode_rows` runs the oracle's worker side (EF accumulate, segment scale,
compressor) over whole rows: every (segment, worker) pair is independent, so
the pairs run in threads (the oracle's C functions release the interpreter
lock), each on its own slice of the same arrays.  `server_side` then takes the
oracle's server average, update and extrapolation.

`StepCheck` checks, on the device and in binary64, what Algorithm 2 fixes for
any compressor (Appendix B, eq. (tilde)): w~_t = w_t - (1/M) sum_m e_t^(m)
follows w~_t = w~_{t-1} - (eta/M) sum_m g_t^(m), up to the binary32 roundings
of one iteration.  It also reports, per worker, ||e_t|| and the contraction
||e_t||^2 / ||p_t||^2 of Lemma 1 (delta_eff = 1 - that ratio), and checks
it where the paper fixes it: the scaled sign's closed form per segment
(||Q(x) - x||^2 = ||x||^2 - ||x||_1^2 / n) and Theorem 1's 1 - k/d for top-k.
"""
import concurrent.futures
import json
import os

import numpy as np

from oracle import oracle as orc

THREADS = max(1, min(16, os.cpu_count() or 1))
EPS32 = 2.0 ** -24


def levels_of(w):
    return (1 << (w.levels - 1)) - 1 if w.kind == "mbit" else w.levels


def encode_rows(w, G, E_prev, t, scales=None):
    """The oracle's worker side of iteration t for every worker and segment.

    G, E_prev: host [M][ld] float32.  scales: None (the oracle's own segment
    scales) or [M][S] (teacher-forced).  Returns own scales [M][S], sign bits
    uint8 [M][d], levels uint16 [M][d], p-hat and e_t float32 [M][ld] (zero
    padding)."""
    M, d, ld = w.M, w.d, w.ld
    offs = w.seg_offsets
    S = len(offs) - 1
    eta = np.float32(w.eta)
    own = np.zeros((M, S), np.float32)
    bits = np.zeros((M, d), np.uint8)
    lv = np.zeros((M, d), np.uint16)
    phat = np.zeros((M, ld), np.float32)
    enew = np.zeros((M, ld), np.float32)
    k = levels_of(w)

    def task(jm):
        j, m = jm
        a, b = offs[j], offs[j + 1]
        p = orc.ef_accumulate(eta, G[m, a:b], E_prev[m, a:b])
        own[m, j] = orc.scale(p, w.norm)
        sc = own[m, j] if scales is None else scales[m, j]
        if w.kind == "sign":
            bt, ph, e = orc.sign_encode(p, sc)
        else:
            bt, l, ph, e = orc.qsgd_encode(p, sc, k, w.quant_seed, m, t, i0=a)
            lv[m, a:b] = l
        bits[m, a:b] = bt
        phat[m, a:b] = ph
        enew[m, a:b] = e

    with concurrent.futures.ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(task, [(j, m) for j in range(S) for m in range(M)]))
    return own, bits, lv, phat, enew


def pack_rows(w, bits, lv):
    """The oracle's message planes of every row: sign plane and level plane
    (or the m-bit code plane)."""
    M, d, ld = w.M, w.d, w.ld
    sign = np.zeros((M, ld // 32), np.uint32) if w.kind in ("sign", "qsgd") else None
    b = w.levels if w.kind == "mbit" else {255: 8, 15: 4}.get(w.levels, 0)
    level = np.zeros((M, ld * b // 32), np.uint32) if b else None

    def task(m):
        if sign is not None:
            sign[m] = orc.pack_bits(bits[m].astype(np.uint16), 1, ld // 32)
        if level is not None:
            f = orc.mbit_fields(bits[m], lv[m], w.levels) if w.kind == "mbit" else lv[m]
            level[m] = orc.pack_bits(f, b, ld * b // 32)

    with concurrent.futures.ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(task, range(M)))
    return sign, level


def server_side(w, G, phat, enew, W_prev):
    """The oracle's server average of p-hat, the update w_t and every
    worker's next evaluation point.  Returns q-hat [d], w_t [d], WX [M][d]."""
    d = w.d
    eta = np.float32(w.eta)
    q = orc.aggregate(phat, d)
    wt = orc.omd_update(q, W_prev[:d])
    wx = np.empty((w.M, d), np.float32)

    def task(m):
        wx[m] = orc.extrapolate(eta, wt, G[m, :d], enew[m, :d])

    with concurrent.futures.ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(task, range(w.M)))
    return q, wt, wx


class StepCheck:
    """Device-side binary64 checks around one iteration (see the module
    docstring).  Call before() with the pre-step state, run the iteration,
    then after() with the results; after() returns the per-step report."""

    def __init__(self, w):
        self.w = w

    def before(self, G, E, W):
        import torch
        w = self.w
        d = w.d
        eta = torch.tensor(w.eta, dtype=torch.float32, device=G.device)
        f64 = dict(dtype=torch.float64, device=G.device)
        self.W_prev = W[:d].double()
        self.sum_e = torch.zeros(d, **f64)
        self.sum_g = torch.zeros(d, **f64)
        self.sum_abs = torch.zeros(d, **f64)
        self.p2 = torch.zeros(w.M, **f64)
        self.l1_term = torch.zeros(w.M, **f64)  # sum over segments of ||p_j||_1^2 / n_j
        offs = torch.tensor(w.seg_offsets, dtype=torch.int64, device=G.device)
        for m in range(w.M):
            eg = G[m, :d] * eta
            p = eg + E[m, :d]
            pd = p.double()
            self.sum_e += E[m, :d].double()
            self.sum_g += G[m, :d].double()
            self.sum_abs += eg.double().abs() + pd.abs()
            self.p2[m] = (pd * pd).sum()
            if w.kind == "sign":
                c = torch.cat([torch.zeros(1, **f64), pd.abs().cumsum(0)])
                l1 = c[offs[1:]] - c[offs[:-1]]
                self.l1_term[m] = (l1 * l1 / (offs[1:] - offs[:-1]).double()).sum()

    def after(self, E, W, Q):
        import torch
        w = self.w
        d = w.d
        e2 = torch.zeros(w.M, dtype=torch.float64, device=E.device)
        sum_e_t = torch.zeros(d, dtype=torch.float64, device=E.device)
        sum_abs_e = torch.zeros(d, dtype=torch.float64, device=E.device)
        for m in range(w.M):
            ed = E[m, :d].double()
            e2[m] = (ed * ed).sum()
            sum_e_t += ed
            sum_abs_e += ed.abs()
        eta = float(np.float32(w.eta))
        Wd = W[:d].double()
        tilde = Wd - sum_e_t / w.M
        expect = (self.W_prev - self.sum_e / w.M) - eta * self.sum_g / w.M
        resid = (tilde - expect).abs()
        tol = 2 * EPS32 * (Wd.abs() + self.W_prev.abs() + Q[:d].double().abs() + self.sum_abs + sum_abs_e)
        worst = float((resid / torch.clamp(tol, min=1e-300)).max())
        assert bool((resid <= tol).all()), "Appendix B eq. (tilde): residual above the rounding bound (%.3g)" % worst
        ratio = (e2 / torch.clamp(self.p2, min=1e-300)).cpu().numpy()
        if w.kind == "sign":
            # per segment ||Q(x) - x||^2 = ||x||^2 - ||x||_1^2 / n, summed over segments
            closed = (self.p2 - self.l1_term).cpu().numpy()
            np.testing.assert_allclose(e2.cpu().numpy(), closed, rtol=1e-5, atol=1e-30)
        if w.kind == "topk":
            assert np.all(ratio <= 1.0 - w.k / w.d + 1e-12), ratio.max()
        assert np.all(np.isfinite(ratio))
        enorm = np.sqrt(e2.cpu().numpy())
        return {"appB_resid_over_bound": worst,
                "e_norm_min": float(enorm.min()), "e_norm_max": float(enorm.max()),
                "e_norm_mean": float(enorm.mean()),
                "delta_eff_min": float(1 - ratio.max()), "delta_eff_mean": float(1 - ratio.mean()),
                "delta_eff_max": float(1 - ratio.min())}


def log_report(name, t, rep):
    """One line per iteration in the test output (pytest -s shows it)."""
    print("REPORT " + json.dumps(dict(workload=name, t=t, **rep)), flush=True)
