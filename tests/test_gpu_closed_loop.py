"""Closed loop on the GPU: Algorithm 2 on the bilinear game with each worker's
gradient evaluated at its own extrapolated point (qualitative, Section 2.2:
the optimistic iteration converges where plain gradient steps diverge), and
a teacher-forced parity check of an iteration in the middle of the loop."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

COMPRESSORS = [("identity", {}), ("sign", {}), ("qsgd", {"levels": 15}), ("topk", {"k": 64}),
               ("mbit", {"levels": 8, "norm": "linf"})]


@pytest.mark.parametrize("kind,extra", COMPRESSORS)
def test_bilinear_converges_with_compression(kind, extra):
    from paper_2010_13359_amd import closed_loop
    checked = []

    def check(t, st):
        if t != 300:
            return
        import torch
        from oracle import oracle as orc
        plan = st["plan"]
        G, E, W = st["G"].cpu().numpy(), st["E"].cpu().numpy(), st["W"].cpu().numpy()
        cfg = {"d": plan.d, "ld": plan.ld, "M": plan.M, "seg_offsets": [0, plan.d], "kind": kind,
               "norm": extra.get("norm", {"sign": "l1", "qsgd": "l2"}.get(kind, "l1")),
               "levels": extra.get("levels", 0), "k": extra.get("k", 0), "seed": plan.seed}
        # run this iteration on a copy and compare with the oracle
        Gd, Ed, Wd = torch.from_numpy(G).cuda(), torch.from_numpy(E).cuda(), torch.from_numpy(W).cuda()
        WXd = torch.empty_like(Ed)
        wire = plan.new_wire("cuda")
        from paper_2010_13359_amd import dqgan
        dqgan.step_fused(plan, 0.2, t, Gd, Ed, Wd, WXd, wire)
        torch.cuda.synchronize()
        scales = wire.scale.view(plan.M, 1).cpu().numpy() if wire.scale is not None else None
        ref = orc.step(cfg, np.float32(0.2), t, G, E.copy(), W.copy(), scales_in=scales)
        d = plan.d
        assert np.array_equal(Ed.cpu().numpy()[:, :d], ref["E"][:, :d])
        assert np.array_equal(Wd.cpu().numpy()[:d], ref["W"][:d])
        assert np.array_equal(WXd.cpu().numpy()[:, :d], ref["WX"][:, :d])
        checked.append(t)

    hist = closed_loop.run_bilinear(kind, n=512, M=4, T=800, eta=0.2, noise=0.05, seed=0, on_step=check,
                                    **extra)
    print(kind, ["%.3f" % h for h in hist])
    assert checked == [300]
    assert hist[-1] < 0.5 and hist[-1] < hist[0]


def test_plain_gradient_steps_diverge():
    from paper_2010_13359_amd import closed_loop
    r = closed_loop.run_gradient_descent(n=512, T=800, eta=0.2, seed=0)
    assert not np.isfinite(r) or r > 10
