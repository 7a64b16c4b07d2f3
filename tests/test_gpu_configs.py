"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times (dqgan_step_scales then dqgan_step_apply), on the gradient
batches bench.py draws: one teacher-forced iteration.

C2 (d = 6.3M, M = 16, s = 255) and C5 (the same shape, 8-bit Appendix A
codes, infinity norm): every output against the oracle.
C4 (d = 1e8, M = 64, top-k k = 1e6): sampled workers checked for the exact
top-k property (ties to the lower index) from their p, residuals exact, and
the server average / OMD outputs on sampled column windows against the
oracle, fed the messages of all workers.

The whole trajectories of every workload (C3 and C6 teacher-forced over
every segment, C4 over every row and iteration) are in
test_gpu_trajectories.py."""
import numpy as np
import pytest

from gpu_common import assert_same

pytestmark = pytest.mark.gpu


def _run(w, t_steps=2):
    """Run t_steps iterations from e_0 = 0; return host snapshots of the
    pre-step state of the last iteration and the device outputs."""
    import torch
    import synth
    from paper_2010_13359_amd import dqgan
    dev = torch.device("cuda:0")
    plan = dqgan.Plan.from_workload(w)
    E = torch.zeros((w.M, w.ld), dtype=torch.float32, device=dev)
    W = synth.init_params(w, device=dev)
    WX = torch.empty((w.M, w.ld), dtype=torch.float32, device=dev)
    wire = plan.new_wire(dev)
    G = None
    for t in range(1, t_steps + 1):
        G = synth.gradients(w, t, device=dev, out=G)
        if t == t_steps:
            torch.cuda.synchronize()
            pre = {"E": E, "W": W.clone()}
            pre["E"] = E.clone()
        dqgan.step_scales(plan, w.eta, G, E, wire)
        dqgan.step_apply(plan, w.eta, t, G, E, W, WX, wire)
    torch.cuda.synchronize()
    return plan, G, pre, E, W, WX, wire


@pytest.fixture(autouse=True)
def _release_memory():
    yield
    import gc
    import torch
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.timeout(300)
@pytest.mark.parametrize("index", [2, 5])
def test_c2_c5_full_teacher_forced(index):
    """C2: 8-bit s-level quantizer, L2; C5: the same shape with the paper's
    8-bit sign-magnitude codes and the infinity-norm scale.  Every output."""
    from oracle import oracle as orc
    import synth
    from gpu_common import compare_step
    w = synth.get(index)
    print("C%d full" % index, flush=True)
    plan, G, pre, E, W, WX, wire = _run(w)
    t = 2
    gpu = {"E": E.cpu().numpy(), "W": W.cpu().numpy(), "WX": WX.cpu().numpy(),
           "scale": wire.scale.view(w.M, w.n_seg).cpu().numpy(),
           "level": wire.level.view(w.M, -1).cpu().numpy().view(np.uint32)}
    if wire.sign is not None:
        gpu["sign"] = wire.sign.view(w.M, -1).cpu().numpy().view(np.uint32)
    Gh, Eh, Wh = G.cpu().numpy(), pre["E"].cpu().numpy(), pre["W"].cpu().numpy()
    plan.close()
    ref = orc.step(w.as_dict(), np.float32(w.eta), t, Gh, Eh.copy(), Wh.copy(), scales_in=gpu["scale"])
    gpu["qhat"] = ref["qhat"]  # not requested from the GPU here; W and WX carry it
    compare_step(w, gpu, ref, check_padding=False)
    own = orc.step(w.as_dict(), np.float32(w.eta), t, Gh, Eh.copy(), Wh.copy())
    np.testing.assert_allclose(gpu["scale"], own["scale"], rtol=1e-5, atol=0)


@pytest.mark.timeout(300)
def test_c4_sampled_rows_and_windows():
    from oracle import oracle as orc
    import synth
    w = synth.get(4)
    print("C4 sampled", flush=True)
    plan, G, pre, E, W, WX, wire = _run(w)
    eta = np.float32(w.eta)
    k = w.k
    idx = wire.idx.view(w.M, k)
    val = wire.val.view(w.M, k)
    for m in (0, w.M - 1):
        p = orc.ef_accumulate(eta, G[m, :w.d].cpu().numpy(), pre["E"][m, :w.d].cpu().numpy())
        ii = idx[m].cpu().numpy().view(np.uint32).astype(np.int64)
        vv = val[m].cpu().numpy()
        assert np.all(np.diff(ii) > 0) and ii[0] >= 0 and ii[-1] < w.d
        assert_same("values row %d" % m, vv, p[ii])
        key = np.abs(p).view(np.uint32)
        sel = np.zeros(w.d, bool)
        sel[ii] = True
        T = key[ii].min()
        assert key[~sel].max() <= T
        # ties at T: the selected ones are the lowest indices among them
        tie_sel = np.flatnonzero(sel & (key == T))
        tie_rest = np.flatnonzero(~sel & (key == T))
        if tie_rest.size:
            assert tie_sel.max() < tie_rest.min()
        e_t = E[m, :w.d].cpu().numpy()
        assert np.all(e_t[sel] == 0) and np.array_equal(e_t[~sel], p[~sel])
    # server average, update and extrapolation on windows, from all messages
    all_idx = idx.cpu().numpy().view(np.uint32).astype(np.int64)
    all_val = val.cpu().numpy()
    for a in (0, 50_000_000 - 4096, w.d - 8192):
        b = a + 8192
        ph = np.zeros((w.M, b - a), np.float32)
        for m in range(w.M):
            lo_, hi_ = np.searchsorted(all_idx[m], [a, b])
            ph[m, all_idx[m, lo_:hi_] - a] = all_val[m, lo_:hi_]
        q = orc.aggregate(ph, b - a)
        wt = orc.omd_update(q, pre["W"][a:b].cpu().numpy())
        assert_same("w_t window %d" % a, W[a:b].cpu().numpy(), wt)
        Gs = G[:, a:b].cpu().numpy()
        Es = E[:, a:b].cpu().numpy()
        wx = np.stack([orc.extrapolate(eta, wt, Gs[m], Es[m]) for m in range(w.M)])
        assert_same("WX window %d" % a, WX[:, a:b].cpu().numpy(), wx)
    plan.close()
