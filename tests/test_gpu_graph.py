"""Iterations of Algorithm 2, and the server side as separate calls,
captured in a HIP graph and replayed.

The two passes (dqgan_step_scales, dqgan_step_apply) issue kernel launches
only (no memset, no host synchronisation), so a caller can capture several
iterations into one graph.  Each replay here starts from the same state,
reset by eager copies and a device synchronisation between replays, and must
reproduce the eager run bit for bit: e_t, w_t, the evaluation points and
every message plane.
"""
import numpy as np
import pytest

import synth
from gpu_common import GpuState, inputs, to_dev
from synth.configs import custom

pytestmark = pytest.mark.gpu

CASES = {
    "sign_c0": lambda: synth.get(0),
    "qsgd15_m32_segs": lambda: custom(d=70001, M=32, kind="qsgd", levels=15, seg_offsets=[0, 64, 4097, 30000, 70001],
                                      eta=1e-2, seed=6),
    "mbit8_linf_m13": lambda: custom(d=3333, M=13, kind="mbit", levels=8, norm="linf", seg_offsets=[0, 1000, 3333],
                                     eta=1e-2, seed=24),
    "topk_m11": lambda: custom(d=7000, M=11, kind="topk", k=300, eta=1e-2, seed=25),
}

STEPS = 3
REPLAYS = 3


def _steps(s, G2):
    """STEPS iterations t = 1..STEPS, the gradient buffers alternating."""
    for t in range(1, STEPS + 1):
        G = s.G if t % 2 else G2
        s.dq.step_scales(s.plan, s.w.eta, G, s.E, s.wire)
        s.dq.step_apply(s.plan, s.w.eta, t, G, s.E, s.W, s.WX, s.wire)


def _scramble(s):
    """Overwrite every output so that a replay must write all of it again."""
    s.WX.fill_(float("nan"))
    for t in (s.wire.sign, s.wire.level, s.wire.scale, s.wire.val, s.wire.idx):
        if t is not None:
            t.fill_(float("nan") if t.dtype.is_floating_point else -1)


@pytest.mark.parametrize("name", sorted(CASES))
def test_graph_replay_equals_eager(name):
    import torch
    w = CASES[name]()
    print("case", name, "d", w.d, "M", w.M, flush=True)
    G, E, W = inputs(w)
    s = GpuState(w, G, E, W)
    G2 = to_dev(synth.gradients_np(w, 2))
    E0, W0 = s.E.clone(), s.W.clone()
    _steps(s, G2)
    torch.cuda.synchronize()
    ref = s.host()

    s.E.copy_(E0)
    s.W.copy_(W0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _steps(s, G2)
    torch.cuda.synchronize()
    for rep in range(REPLAYS):
        s.E.copy_(E0)
        s.W.copy_(W0)
        _scramble(s)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = s.host()
        for key, want in ref.items():
            a, b = np.ascontiguousarray(got[key]), np.ascontiguousarray(want)
            assert a.shape == b.shape, (rep, key)
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "replay %d differs in %s" % (rep, key)
    del graph
    s.close()


SERVER_CASES = {
    "qsgd15_m32_segs": CASES["qsgd15_m32_segs"],
    "mbit8_linf_m13": CASES["mbit8_linf_m13"],
    "topk_m11": CASES["topk_m11"],
    # several column tiles of the top-k average, dense and sparse ones
    "topk_m64_tiles": lambda: custom(d=50001, M=64, kind="topk", k=3000, eta=1e-2, seed=26),
}


@pytest.mark.parametrize("name", sorted(SERVER_CASES))
def test_graph_replay_server_calls_equal_eager(name):
    """The server side as separate calls (dqgan_aggregate, then
    dqgan_unpack) captured in a graph: every replay, after the outputs are
    overwritten, reproduces the eager results bit for bit."""
    import torch
    w = SERVER_CASES[name]()
    print("case", name, "d", w.d, "M", w.M, flush=True)
    G, E, W = inputs(w)
    s = GpuState(w, G, E, W)
    s.fused(1)  # a message to average
    Ph = torch.full((w.M, w.ld), float("nan"), dtype=torch.float32, device=s.Q.device)
    s.dq.aggregate(s.plan, s.wire, s.Q)
    s.dq.unpack(s.plan, s.wire, Ph)
    torch.cuda.synchronize()
    q_ref, ph_ref = s.Q.cpu().numpy(), Ph.cpu().numpy()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        s.dq.aggregate(s.plan, s.wire, s.Q)
        s.dq.unpack(s.plan, s.wire, Ph)
    torch.cuda.synchronize()
    for rep in range(REPLAYS):
        s.Q.fill_(float("nan"))
        Ph.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(s.Q.cpu().numpy().view(np.uint32), q_ref.view(np.uint32)), "replay %d: q-hat" % rep
        assert np.array_equal(Ph.cpu().numpy().view(np.uint32), ph_ref.view(np.uint32)), "replay %d: p-hat" % rep
    del graph
