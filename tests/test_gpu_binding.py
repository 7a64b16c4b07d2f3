"""The Python binding rejects tensors the C ABI cannot check (plain pointers):
wrong dtype, too few bytes, host memory, non-contiguous views, missing
message planes.  Every rejection happens on the host, before anything is
enqueued; a correct call afterwards still matches the oracle's message."""
import numpy as np
import pytest

from gpu_common import GpuState, inputs
from synth.configs import custom

pytestmark = pytest.mark.gpu


def _state():
    w = custom(d=5000, M=3, kind="qsgd", levels=15, seg_offsets=[0, 1234, 5000], eta=1e-2, seed=41)
    G, E, W = inputs(w)
    return w, GpuState(w, G, E, W)


def test_rejects_bad_tensors():
    import torch
    from paper_2010_13359_amd import dqgan
    w, s = _state()
    dev = s.G.device
    bad = {
        "too small": s.G.view(-1)[:-1],
        "float64": s.G.double(),
        "host memory": s.G.cpu(),
        "not contiguous": s.G.t(),
    }
    for why, G in bad.items():
        with pytest.raises((TypeError, ValueError)):
            dqgan.step_fused(s.plan, w.eta, 1, G, s.E, s.W, s.WX, s.wire)
        print("rejected G:", why, flush=True)
    with pytest.raises(ValueError):
        dqgan.step_fused(s.plan, w.eta, 1, s.G, s.E, s.W[:-1], s.WX, s.wire)
    with pytest.raises(ValueError):
        dqgan.step_fused(s.plan, w.eta, 1, s.G, s.E, s.W, s.WX, s.wire, Qhat=s.Q[: w.d])
    # message planes: missing, too small, wrong dtype
    for plane, repl in (("sign", None), ("level", s.wire.level[:-1]), ("scale", s.wire.scale.to(torch.float64))):
        wire = dqgan.Wire(s.wire.sign, s.wire.level, s.wire.scale, s.wire.val, s.wire.idx)
        setattr(wire, plane, repl)
        with pytest.raises((TypeError, ValueError)):
            dqgan.step_fused(s.plan, w.eta, 1, s.G, s.E, s.W, s.WX, wire)
    # codes of dqgan_pack must be 16-bit
    codes32 = torch.zeros((w.M, w.ld), dtype=torch.int32, device=dev)
    with pytest.raises(TypeError):
        dqgan.pack(s.plan, codes32, s.wire.scale, s.wire)
    # nothing ran: the state is untouched, and a correct call works
    torch.cuda.synchronize()
    s.fused(1)
    gpu = s.host()
    s.close()
    from oracle import oracle as orc
    G0, E0, W0 = inputs(w)
    ref = orc.step(w.as_dict(), np.float32(w.eta), 1, G0, E0.copy(), W0.copy(), scales_in=gpu["scale"])
    assert np.array_equal(gpu["level"], ref["level"]) and np.array_equal(gpu["sign"], ref["sign"])
    assert np.array_equal(gpu["E"].view(np.uint32), ref["E"].view(np.uint32))
