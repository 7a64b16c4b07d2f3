"""GPU parity of every benchmark workload over its whole stated trajectory,
in the launch configuration bench.py times (gradients drawn on the device
with the bench's generator), through the C ABI.

* C0 (T = 10), C1 (T = 100), C2 and C5 (T = 50): free-running at full size,
  each side on its own state and its own scales, every output of every
  iteration against the oracle: scales within 1e-5 relative, e_t, w_t, q-hat
  and WX identical.  The two sides sum a segment's binary64 norm in
  different orders; where the rounded scale differs in its last bit, that
  (worker, segment) pair takes the GPU's scale (counted and reported).
* C3 and C6: one teacher-forced iteration over all 64 segments and all 32
  workers (every message bit and every binary32 output identical, scales
  within 1e-5); then the 20-iteration free run on sampled segments.
* C4 (T = 5): every iteration, every one of the 64 rows on the device: the
  exact top-k property of (value, index) against the row's p (ties to the
  lower index), e_t exact, and q-hat, w_t and WX over all 10^8 columns from
  the ascending-worker sum of the messages.

Every iteration of every workload also checks Appendix B's eq. (tilde) in
binary64 on the GPU's own state and reports ||e_t|| per worker and delta_eff
(tests/trajectory.py), with Lemma 1's contraction checked for the scaled
sign (closed form) and top-k (Theorem 1).
"""
import numpy as np
import pytest

from gpu_common import assert_same, rel_close
from trajectory import StepCheck, encode_rows, levels_of, log_report, pack_rows, server_side

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _release_memory():
    yield
    import gc
    import torch
    gc.collect()
    torch.cuda.empty_cache()


def _device_state(w):
    import torch
    import synth
    from paper_2010_13359_amd import dqgan
    dev = torch.device("cuda:0")
    plan = dqgan.Plan.from_workload(w)
    E = torch.zeros((w.M, w.ld), dtype=torch.float32, device=dev)
    W = synth.init_params(w, device=dev)
    WX = torch.empty((w.M, w.ld), dtype=torch.float32, device=dev)
    Q = torch.empty(w.ld, dtype=torch.float32, device=dev)
    return plan, E, W, WX, Q, plan.new_wire(dev)


def _step(plan, w, t, G, E, W, WX, wire, Q):
    import torch
    from paper_2010_13359_amd import dqgan
    dqgan.step_scales(plan, w.eta, G, E, wire)
    dqgan.step_apply(plan, w.eta, t, G, E, W, WX, wire, Q)
    torch.cuda.synchronize()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("index", [0, 1, 2, 5])
def test_free_running_whole_trajectory(index):
    import synth
    w = synth.get(index)
    d = w.d
    print("C%d free-running, %d iterations" % (index, w.T), flush=True)
    plan, E, W, WX, Q, wire = _device_state(w)
    check = StepCheck(w)
    E_r = np.zeros((w.M, w.ld), np.float32)
    W_r = W.cpu().numpy()
    G = None
    forced = 0
    for t in range(1, w.T + 1):
        G = synth.gradients(w, t, device=E.device, out=G)
        check.before(G, E, W)
        _step(plan, w, t, G, E, W, WX, wire, Q)
        rep = check.after(E, W, Q)
        Gh = G.cpu().numpy()
        own, _, _, phat, enew = encode_rows(w, Gh, E_r, t)
        scales = wire.scale.view(w.M, w.n_seg).cpu().numpy()
        rel_close("scale t=%d" % t, scales, own, tau=1e-30)
        differ = scales != own
        if differ.any():
            # binary64 sums in another order rounded to the other neighbour:
            # those (worker, segment) pairs take the GPU's scale
            _, _, _, phat, enew = encode_rows(w, Gh, E_r, t, scales=np.where(differ, scales, own))
            forced += int(differ.sum())
        q, wt, wx = server_side(w, Gh, phat, enew, W_r)
        assert_same("e_t t=%d" % t, E[:, :d].cpu().numpy(), enew[:, :d])
        assert_same("qhat t=%d" % t, Q[:d].cpu().numpy(), q)
        assert_same("w_t t=%d" % t, W[:d].cpu().numpy(), wt)
        assert_same("WX t=%d" % t, WX[:, :d].cpu().numpy(), wx)
        E_r, W_r[:d] = enew, wt
        log_report("C%d" % index, t, dict(rep, scales_forced=int(differ.sum())))
    plan.close()
    print("C%d: %d iterations identical; %d of %d scales taken from the GPU (last-bit differences)"
          % (index, w.T, forced, w.T * w.M * w.n_seg), flush=True)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("index", [3, 6])
def test_c3_c6_teacher_forced_every_segment(index):
    """Iteration t = 2 (from e_1 of the first iteration), all 64 segments and
    all 32 workers, teacher-forced with the GPU's scales: the sign and level
    (or code) planes word for word, e_t, q-hat, w_t and WX identical; every
    GPU scale within 1e-5 of the oracle's own."""
    import synth
    w = synth.get(index)
    d = w.d
    print("C%d teacher-forced, every segment" % index, flush=True)
    plan, E, W, WX, Q, wire = _device_state(w)
    G = None
    for t in (1, 2):
        G = synth.gradients(w, t, device=E.device, out=G)
        if t == 2:
            E_pre, W_pre = E.cpu().numpy(), W.cpu().numpy()
        _step(plan, w, t, G, E, W, WX, wire, Q)
    Gh = G.cpu().numpy()
    scales = wire.scale.view(w.M, w.n_seg).cpu().numpy()
    own, bits, lv, phat, enew = encode_rows(w, Gh, E_pre, 2, scales=scales)
    print("oracle worker side done", flush=True)
    rel_close("scale", scales, own, tau=1e-30)
    sign, level = pack_rows(w, bits, lv)
    if sign is not None:
        assert_same("sign plane", wire.sign.view(w.M, -1).cpu().numpy().view(np.uint32), sign)
    assert_same("level plane", wire.level.view(w.M, -1).cpu().numpy().view(np.uint32), level)
    assert_same("e_t", E[:, :d].cpu().numpy(), enew[:, :d])
    del bits, lv
    q, wt, wx = server_side(w, Gh, phat, enew, W_pre)
    assert_same("qhat", Q[:d].cpu().numpy(), q)
    assert_same("w_t", W[:d].cpu().numpy(), wt)
    assert_same("WX", WX[:, :d].cpu().numpy(), wx)
    plan.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("index", [3, 6])
def test_c3_c6_free_running_sampled_segments(index):
    """The whole 20-iteration trajectory at full size, each side on its own
    state.  Every quantity of an iteration is a function of the columns of
    whole segments, so the oracle follows the sampled segments (the smallest,
    a middle one, the largest) of all workers on its own, with the global
    element index for the generator counter.  Scales within 1e-5 (a pair
    whose scale differs in its last bit takes the GPU's); e_t, w_t and WX
    identical."""
    import synth
    from oracle import oracle as orc
    w = synth.get(index)
    print("C%d free-running, sampled segments, %d iterations" % (index, w.T), flush=True)
    sizes = np.diff(w.seg_offsets)
    picks = sorted({int(np.argmin(sizes)), int(np.argsort(sizes)[len(sizes) // 2]), int(np.argmax(sizes))})
    plan, E, W, WX, Q, wire = _device_state(w)
    check = StepCheck(w)
    eta = np.float32(w.eta)
    k = levels_of(w)
    seg = {j: (w.seg_offsets[j], w.seg_offsets[j + 1]) for j in picks}
    E_r = {j: np.zeros((w.M, b - a), np.float32) for j, (a, b) in seg.items()}
    W_r = {j: W[a:b].cpu().numpy() for j, (a, b) in seg.items()}
    G = None
    forced = 0
    for t in range(1, w.T + 1):
        G = synth.gradients(w, t, device=E.device, out=G)
        check.before(G, E, W)
        _step(plan, w, t, G, E, W, WX, wire, Q)
        rep = check.after(E, W, Q)
        scales = wire.scale.view(w.M, w.n_seg).cpu().numpy()
        for j, (a, b) in seg.items():
            n = b - a
            Gs = G[:, a:b].cpu().numpy()
            own = np.empty(w.M, np.float32)
            phat = np.empty((w.M, n), np.float32)
            enew = np.empty((w.M, n), np.float32)
            for m in range(w.M):
                p = orc.ef_accumulate(eta, Gs[m], E_r[j][m])
                own[m] = orc.scale(p, w.norm)
                sc = own[m]
                if scales[m, j] != own[m]:
                    # a last-bit difference of the binary64 sums' rounding:
                    # the GPU's scale for this (worker, segment)
                    assert abs(float(scales[m, j]) - float(own[m])) <= 1e-5 * float(own[m]), (j, m, t)
                    sc = scales[m, j]
                    forced += 1
                _, _, phat[m], enew[m] = orc.qsgd_encode(p, sc, k, w.quant_seed, m, t, i0=a)
            rel_close("scale seg %d t=%d" % (j, t), scales[:, j], own, tau=1e-30)
            wt = orc.omd_update(orc.aggregate(phat, n), W_r[j])
            wx = np.stack([orc.extrapolate(eta, wt, Gs[m], enew[m]) for m in range(w.M)])
            assert_same("e_t seg %d t=%d" % (j, t), E[:, a:b].cpu().numpy(), enew)
            assert_same("w_t seg %d t=%d" % (j, t), W[a:b].cpu().numpy(), wt)
            assert_same("WX seg %d t=%d" % (j, t), WX[:, a:b].cpu().numpy(), wx)
            E_r[j], W_r[j] = enew, wt
        log_report("C%d" % index, t, dict(rep, scales_forced=forced))
    plan.close()
    print("C%d: %d iterations identical on the sampled segments; %d scales taken from the GPU" % (index, w.T, forced),
          flush=True)


@pytest.mark.timeout(900)
def test_c4_every_row_every_iteration():
    """Top-k, d = 10^8, M = 64, k = 10^6, the 5 iterations of the workload.
    On the device (torch, each binary32 operation a separate rounding, sums
    in ascending worker order): for every row, the message is the exact
    top-k of |p| (ties to the lower index) in ascending index order with the
    values of p; e_t = 0 on it and p elsewhere; then q-hat, w_t and WX over
    all columns."""
    import torch
    import synth
    w = synth.get(4)
    d, M, k = w.d, w.M, w.k
    print("C4 every row, %d iterations" % w.T, flush=True)
    plan, E, W, WX, Q, wire = _device_state(w)
    check = StepCheck(w)
    eta = torch.tensor(w.eta, dtype=torch.float32, device=E.device)
    idx_all = wire.idx.view(M, k)
    val_all = wire.val.view(M, k)
    G = None
    for t in range(1, w.T + 1):
        G = synth.gradients(w, t, device=E.device, out=G)
        E_prev = E.clone()
        W_prev = W[:d].clone()
        check.before(G, E, W)
        _step(plan, w, t, G, E, W, WX, wire, Q)
        rep = check.after(E, W, Q)
        S = None
        for m in range(M):
            p = G[m, :d] * eta + E_prev[m, :d]
            key = p.abs().view(torch.int32)
            idx = idx_all[m].long()
            val = val_all[m]
            assert bool((idx[1:] > idx[:-1]).all()) and int(idx[0]) >= 0 and int(idx[-1]) < d, (t, m)
            assert torch.equal(val.view(torch.int32), p[idx].view(torch.int32)), (t, m)
            sel = torch.zeros(d, dtype=torch.bool, device=p.device)
            sel[idx] = True
            T = key[idx].min()
            rest = ~sel
            assert int(key[rest].max()) <= int(T), (t, m)
            tie_rest = torch.nonzero(rest & (key == T)).view(-1)
            if tie_rest.numel():
                tie_sel = torch.nonzero(sel & (key == T)).view(-1)
                assert int(tie_sel.max()) < int(tie_rest.min()), (t, m)
            e_t = E[m, :d]
            assert bool((e_t[sel] == 0).all()), (t, m)
            assert torch.equal(e_t[rest].view(torch.int32), p[rest].view(torch.int32)), (t, m)
            ph = torch.zeros(d, dtype=torch.float32, device=p.device)
            ph[idx] = val
            S = ph if S is None else S + ph
            del p, key, sel, rest, ph
        q = S / M
        wt = W_prev - q
        assert bool((Q[:d] == q).all()), t
        assert bool((W[:d] == wt).all()), t
        for m in range(M):
            x = G[m, :d] * eta + E[m, :d]
            assert bool((WX[m, :d] == wt - x).all()), (t, m)
        del E_prev, W_prev, S, q, wt
        log_report("C4", t, rep)
        print("C4 iteration %d checked" % t, flush=True)
    plan.close()
