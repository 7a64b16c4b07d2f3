"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
(via the binding) and the oracle on the very same inputs."""
import numpy as np

import synth


def device():
    import torch
    return torch.device("cuda:0")


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(device())


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def inputs(w, t=1, e_scale=1e-3, seed=7):
    """Host inputs of one iteration: gradients g_t, a non-zero e_{t-1} (so the
    error feedback is exercised), w_{t-1}."""
    G = synth.gradients_np(w, t)
    rng = np.random.default_rng(seed)
    E = np.zeros((w.M, w.ld), np.float32)
    E[:, :w.d] = (rng.standard_normal((w.M, w.d)) * e_scale).astype(np.float32)
    W = synth.init_params_np(w)
    return G, E, W


class GpuState:
    """Device copies of one iteration's state plus the plan and message."""

    def __init__(self, w, G, E, W):
        import torch
        from paper_2010_13359_amd import dqgan
        self.w = w
        self.dq = dqgan
        self.plan = dqgan.Plan.from_workload(w)
        self.G, self.E, self.W = to_dev(G), to_dev(E), to_dev(W)
        self.WX = torch.full((w.M, w.ld), float("nan"), dtype=torch.float32, device=device())
        self.Q = torch.full((w.ld,), float("nan"), dtype=torch.float32, device=device())
        self.wire = self.plan.new_wire(device())

    def fused(self, t, eta=None):
        import torch
        self.dq.step_fused(self.plan, self.w.eta if eta is None else eta, t, self.G, self.E, self.W, self.WX,
                           self.wire, self.Q)
        torch.cuda.synchronize()

    def unfused(self, t, scales_in=None):
        import torch
        w = self.w
        self.dq.compress_ef(self.plan, w.eta, t, self.G, self.E, scales_in, self.wire)
        self.dq.aggregate(self.plan, self.wire, self.Q)
        self.dq.omd_step(self.plan, w.eta, self.Q, self.W, self.G, self.E, self.WX)
        torch.cuda.synchronize()

    def host(self):
        w = self.w
        out = {"E": self.E.cpu().numpy(), "W": self.W.cpu().numpy(), "WX": self.WX.cpu().numpy(),
               "qhat": self.Q.cpu().numpy()}
        if self.wire.scale is not None:
            out["scale"] = self.wire.scale.view(w.M, w.n_seg).cpu().numpy()
        if self.wire.sign is not None:
            out["sign"] = u32(self.wire.sign.view(w.M, -1))
        if self.wire.level is not None:
            out["level"] = u32(self.wire.level.view(w.M, -1))
        if self.wire.val is not None:
            out["val"] = self.wire.val.view(w.M, -1).cpu().numpy()
        if self.wire.idx is not None:
            out["idx"] = u32(self.wire.idx.view(w.M, -1))
        return out

    def close(self):
        self.plan.close()


def assert_same(name, got, exp):
    """Element-by-element equality (binary32 values; +0 and -0 compare
    equal), reporting the first differences."""
    got = np.asarray(got)
    exp = np.asarray(exp)
    assert got.shape == exp.shape, (name, got.shape, exp.shape)
    bad = np.flatnonzero(~((got == exp) | (np.isnan(got) & np.isnan(exp)) if got.dtype.kind == "f" else got == exp))
    if bad.size:
        i = bad[:5]
        raise AssertionError("%s: %d of %d elements differ; first at %s: got %s expected %s" % (
            name, bad.size, got.size, i.tolist(), got.ravel()[i].tolist(), exp.ravel()[i].tolist()))


def compare_step(w, gpu, ref, check_padding=True):
    d = w.d
    assert_same("E", gpu["E"][:, :d], ref["E"][:, :d])
    assert_same("W", gpu["W"][:d], ref["W"][:d])
    assert_same("WX", gpu["WX"][:, :d], ref["WX"][:, :d])
    assert_same("qhat", gpu["qhat"][:d], ref["qhat"][:d])
    if w.kind in ("sign", "qsgd"):
        assert_same("sign plane", gpu["sign"], ref["sign"])
    if w.kind in ("sign", "qsgd", "mbit"):
        assert_same("scale", gpu["scale"], ref["scale"])
    if w.kind in ("qsgd", "mbit"):
        assert_same("level plane", gpu["level"], ref["level"])
    if w.kind == "topk":
        assert_same("idx", gpu["idx"], ref["idx"])
        assert_same("val", gpu["val"], ref["val"])
    if check_padding and w.ld > d:
        assert np.all(gpu["WX"][:, d:] == 0) and np.all(gpu["qhat"][d:] == 0)


def rel_close(name, got, exp, tau, rtol=1e-5):
    """max_i |got_i - exp_i| / max(|exp_i|, tau_i) <= rtol."""
    err = np.abs(got.astype(np.float64) - exp.astype(np.float64)) / np.maximum(np.abs(exp.astype(np.float64)), tau)
    worst = float(err.max()) if err.size else 0.0
    assert worst <= rtol, "%s: max relative error %.3g > %.1g" % (name, worst, rtol)
    return worst
