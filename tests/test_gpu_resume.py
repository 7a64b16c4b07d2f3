"""Checkpoint and resume.  The state of Algorithm 2 between iterations is
w_t, every worker's e_t and the iteration number t (with the workload's
seeds); the plan keeps nothing between iterations that a result depends on.
So T iterations in one run must equal k iterations, a checkpoint of W and E
to files, and the remaining T - k iterations on a fresh plan with fresh
device buffers loaded from those files: e_T, w_T, the evaluation points and
the last message, bit for bit."""
import numpy as np
import pytest

import synth
from synth.configs import custom

pytestmark = pytest.mark.gpu

CASES = {
    "sign": lambda: custom(d=70001, M=8, kind="sign", seg_offsets=[0, 5000, 70001], eta=1e-2, seed=81),
    "qsgd15": lambda: custom(d=70001, M=16, kind="qsgd", levels=15, seg_offsets=[0, 64, 4097, 30000, 70001],
                             eta=1e-2, seed=82),
    "mbit8_linf": lambda: custom(d=50000, M=5, kind="mbit", levels=8, norm="linf", seg_offsets=[0, 777, 50000],
                                 eta=1e-2, seed=83),
    "topk": lambda: custom(d=200000, M=8, kind="topk", k=2000, eta=1e-2, seed=84),
}
T, K = 6, 3


def _iterate(w, E_host, W_host, t_from, t_to):
    """A fresh plan and fresh device buffers, loaded with (E, W); iterations
    t_from .. t_to; returns the host state and the last message."""
    import torch
    from paper_2010_13359_amd import dqgan
    dev = torch.device("cuda:0")
    plan = dqgan.Plan.from_workload(w)
    E = torch.from_numpy(E_host).to(dev)
    W = torch.from_numpy(W_host).to(dev)
    WX = torch.full((w.M, w.ld), float("nan"), dtype=torch.float32, device=dev)
    wire = plan.new_wire(dev)
    for t in range(t_from, t_to + 1):
        G = synth.gradients(w, t, device=dev)
        dqgan.step_fused(plan, w.eta, t, G, E, W, WX, wire)
    torch.cuda.synchronize()
    out = {"E": E.cpu().numpy(), "W": W.cpu().numpy(), "WX": WX.cpu().numpy()}
    for name in ("sign", "level", "scale", "val", "idx"):
        x = getattr(wire, name)
        if x is not None:
            out[name] = x.cpu().numpy()
    plan.close()
    return out


@pytest.mark.parametrize("name", sorted(CASES))
def test_resume_from_checkpoint_is_bit_identical(name, tmp_path):
    w = CASES[name]()
    print("case", name, "d", w.d, "M", w.M, flush=True)
    E0 = np.zeros((w.M, w.ld), np.float32)
    W0 = synth.init_params_np(w)
    straight = _iterate(w, E0, W0, 1, T)
    first = _iterate(w, E0, W0, 1, K)
    np.save(tmp_path / "E.npy", first["E"])
    np.save(tmp_path / "W.npy", first["W"])
    resumed = _iterate(w, np.load(tmp_path / "E.npy", allow_pickle=False),
                       np.load(tmp_path / "W.npy", allow_pickle=False), K + 1, T)
    for key in straight:
        assert np.array_equal(straight[key].view(np.uint32), resumed[key].view(np.uint32)), key
    # and the checkpoint is not a no-op: the state moved between k and T
    assert not np.array_equal(first["W"], straight["W"])
