"""Distinct plans are independent, and every call runs on the stream it is
given.

Three plans (the 4-bit quantizer over seven segments twice, with the same
descriptor, and top-k) iterate at the same time on three non-default
streams, their launches interleaved call by call.  Each must reproduce, bit
for bit, the same iterations run one plan at a time on the default stream:
e_t, w_t, the evaluation points, q-hat and every message plane.  Plans with
one descriptor share no scratch (the top-k selection state and the segment
partials live in the plan).
"""
import numpy as np
import pytest

import synth
from gpu_common import GpuState, assert_same, inputs, to_dev
from synth.configs import custom

pytestmark = pytest.mark.gpu

STEPS = 3


def _workloads():
    q = lambda: custom(d=70001, M=32, kind="qsgd", levels=15,
                       seg_offsets=[0, 64, 65, 1000, 4097, 30000, 65536, 70001], eta=1e-2, seed=6)
    return [q(), q(), custom(d=7000, M=11, kind="topk", k=300, eta=1e-2, seed=25)]


def _states():
    states = []
    for n, w in enumerate(_workloads()):
        G, E, W = inputs(w, seed=7 + n)
        s = GpuState(w, G, E, W)
        s.G2 = to_dev(synth.gradients_np(w, 2 + n))
        states.append(s)
    return states


def _iteration(s, t, stream=None):
    G = s.G if t % 2 else s.G2
    s.dq.step_scales(s.plan, s.w.eta, G, s.E, s.wire, stream=stream)
    s.dq.step_apply(s.plan, s.w.eta, t, G, s.E, s.W, s.WX, s.wire, s.Q, stream=stream)


def test_plans_on_separate_streams_match_sequential():
    import torch
    print("three plans, %d iterations each, sequential then on three streams" % STEPS, flush=True)
    seq = _states()
    for s in seq:
        for t in range(1, STEPS + 1):
            _iteration(s, t)
    torch.cuda.synchronize()
    want = [s.host() for s in seq]
    for s in seq:
        s.close()

    par = _states()
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in par]
    for t in range(1, STEPS + 1):
        # scales of every plan, then the apply passes: the calls of different
        # plans alternate on the host while each stream keeps its own order
        for s, st in zip(par, streams):
            G = s.G if t % 2 else s.G2
            s.dq.step_scales(s.plan, s.w.eta, G, s.E, s.wire, stream=st)
        for s, st in zip(par, streams):
            G = s.G if t % 2 else s.G2
            s.dq.step_apply(s.plan, s.w.eta, t, G, s.E, s.W, s.WX, s.wire, s.Q, stream=st)
    torch.cuda.synchronize()
    for n, (s, ref) in enumerate(zip(par, want)):
        got = s.host()
        assert sorted(got) == sorted(ref)
        for key in ref:
            a, b = np.ascontiguousarray(got[key]), np.ascontiguousarray(ref[key])
            assert_same("plan %d %s" % (n, key), a.view(np.uint32), b.view(np.uint32))
        s.close()
