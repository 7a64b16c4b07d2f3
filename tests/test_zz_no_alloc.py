"""dqgan_step_fused_noalloc (the fused iteration with no plan and no
allocation, its scratch in a static device array) against dqgan_step_fused
through the C ABI: every output identical, on two calls in a row, the second
with a smaller workload, so that the shared scratch holds the first call's
tables when the second starts."""
import numpy as np
import pytest

import synth
from gpu_common import GpuState, compare_step, inputs
from synth.configs import custom

pytestmark = pytest.mark.gpu

PAIRS = {
    # (first call, second call: smaller)
    "qsgd255_c2_then_small": (lambda: synth.get(2),
                              lambda: custom(d=5000, M=4, kind="qsgd", levels=15, seg_offsets=[0, 1234, 5000],
                                             eta=1e-2, seed=5)),
    "qsgd15_segs_then_sign": (lambda: custom(d=70001, M=32, kind="qsgd", levels=15,
                                             seg_offsets=[0, 64, 65, 1000, 4097, 30000, 65536, 70001], eta=1e-2,
                                             seed=6),
                              lambda: custom(d=100, M=2, kind="sign", seg_offsets=[0, 1, 2, 3, 50, 99, 100],
                                             eta=1e-2, seed=2)),
    "mbit8_then_mbit4": (lambda: custom(d=40000, M=16, kind="mbit", levels=8, norm="linf",
                                        seg_offsets=[0, 7, 19999, 40000], eta=1e-2, seed=21),
                         lambda: custom(d=1500, M=100, kind="mbit", levels=4, norm="l2", eta=1e-2, seed=27)),
    "sign_c1_then_identity": (lambda: synth.get(1),
                              lambda: custom(d=4097, M=2, kind="identity", eta=1e-2, seed=12)),
    "tiny_norms_then_m1024": (lambda: custom(d=5000, M=4, kind="qsgd", levels=255,
                                             seg_offsets=[0, 600, 1200, 1800, 2400, 3000, 3600, 4200, 5000],
                                             eta=1.0, seed=62,
                                             group_scale=[1e-41, 3e-39, 2e-38, 1e-37, 1e-30, 5e-20, 1e-3, 2e37]),
                              lambda: custom(d=1, M=1024, kind="mbit", levels=4, norm="linf", eta=1e-2, seed=30)),
}


@pytest.mark.parametrize("name", sorted(PAIRS))
def test_noalloc_equals_plan_step(name):
    import torch
    for i, make in enumerate(PAIRS[name]):
        w = make()
        e_scale = 0.0 if w.eta == 1.0 else 1e-3
        G, E, W = inputs(w, t=2 + i, e_scale=e_scale)
        print("case", name, "call", i, "d", w.d, "M", w.M, w.kind, flush=True)
        a = GpuState(w, G, E, W)
        a.fused(3 + i)
        ref = a.host()
        a.close()
        b = GpuState(w, G, E, W)
        b.dq.step_fused_noalloc(b.plan, w.eta, 3 + i, b.G, b.E, b.W, b.WX, b.wire, b.Q)
        torch.cuda.synchronize()
        got = b.host()
        b.close()
        compare_step(w, got, ref)
        for k in got:
            assert np.array_equal(got[k].view(np.uint32), ref[k].view(np.uint32)), k
