"""GPU parity of the top-k server average (dqgan_aggregate for TOPK) on
messages built on the host, against the oracle's average of the decoded
messages (the sum in ascending worker order, one division by M), bit for bit
including the sign of zero.

The messages mix the kinds of column tiles the kernel tells apart: tiles no
worker sends anything for, tiles with fewer entries than workers, sparse
tiles, and dense bands where every worker sends a large share of the columns (as the layer-wise gradient
scales of the large workloads make them).  Values span sixteen decades with
both signs, so that a sum taken in another order differs.  Worker counts
cover one, partial rounds of four, one and several groups of 64, and
messages that hold every column (k = d).  Special
columns: every worker sends -0 (the average is -0), every worker but one
sends -0 (+0), and one worker alone sends -0 (+0).  The full-size check
compares the server average of the 64 x 1e6 top-k messages of the largest
workload with the fused step's, which the parity tests of that workload tie
to the oracle.  Lists with runs of empty tiles of every length between a
worker's entries check the start of every tile.  Two checks cover messages
outside the format: sorted lists
ending in indices at or beyond d (skipped, so the average is the oracle's
over the rest), and unsorted, repeated and out-of-range indices (undefined
values, but the calls complete, their outputs are finite and the same plan
then averages a well-formed message exactly)."""
import numpy as np
import pytest

from synth.configs import custom

pytestmark = pytest.mark.gpu

ALL_NEG0, ALL_BUT_ONE_NEG0, ONE_NEG0 = 17, 18, 19  # special columns (inside every case's d)


def _messages(d, M, k, seed, dense_band=None, empty_band=None, dense_share=0.7):
    """Sorted distinct indices and values of M workers.  A share of each
    worker's k entries falls in dense_band, none in empty_band."""
    rng = np.random.default_rng(seed)
    idx = np.zeros((M, k), np.uint32)
    val = np.zeros((M, k), np.float32)
    pool = np.ones(d, bool)
    if empty_band is not None:
        pool[empty_band[0]:empty_band[1]] = False
    pool[[ALL_NEG0, ALL_BUT_ONE_NEG0, ONE_NEG0]] = False
    for m in range(M):
        if k == d:  # every worker sends every column: the special columns carry +0 instead
            idx[m] = np.arange(d, dtype=np.uint32)
            val[m] = (rng.standard_normal(k) * 10.0 ** rng.uniform(-8, 8, k)).astype(np.float32)
            val[m, ALL_NEG0] = -0.0
            val[m, ALL_BUT_ONE_NEG0] = 0.0 if m == 1 else -0.0
            val[m, ONE_NEG0] = -0.0 if m == 2 else 0.0
            continue
        special = [ALL_NEG0] + ([ALL_BUT_ONE_NEG0] if m != 1 else []) + ([ONE_NEG0] if m == 2 else [])
        n_free = k - len(special)
        if dense_band is not None:
            a, b = dense_band
            band_pool = np.setdiff1d(np.arange(a, b), [ALL_NEG0, ALL_BUT_ONE_NEG0, ONE_NEG0])
            nd = min(int(dense_share * n_free), band_pool.size)
            band = rng.choice(band_pool, size=nd, replace=False)
            rest_pool = pool.copy()
            rest_pool[a:b] = False
            rest = rng.choice(np.flatnonzero(rest_pool), size=n_free - nd, replace=False)
            chosen = np.concatenate([band, rest])
        else:
            chosen = rng.choice(np.flatnonzero(pool), size=n_free, replace=False)
        chosen = np.sort(np.concatenate([chosen, special]))
        v = (rng.standard_normal(k) * 10.0 ** rng.uniform(-8, 8, k)).astype(np.float32)
        for c in special:
            v[np.searchsorted(chosen, c)] = np.float32(-0.0)
        idx[m] = chosen.astype(np.uint32)
        val[m] = v
    return idx, val


def _oracle_average(w, idx, val):
    from oracle import oracle as orc
    ph = np.zeros((w.M, w.ld), np.float32)
    for m in range(w.M):
        ph[m, idx[m].astype(np.int64)] = val[m]
    q = np.zeros(w.ld, np.float32)
    q[:w.d] = orc.aggregate(ph, w.d)
    return q


def _gpu_average(w, idx, val):
    import torch
    from paper_2010_13359_amd import dqgan
    dev = torch.device("cuda:0")
    plan = dqgan.Plan.from_workload(w)
    wire = plan.new_wire(dev)
    wire.idx.copy_(torch.from_numpy(idx.reshape(-1).view(np.int32)).to(dev))
    wire.val.copy_(torch.from_numpy(val.reshape(-1)).to(dev))
    Q = torch.full((w.ld,), float("nan"), dtype=torch.float32, device=dev)
    dqgan.aggregate(plan, wire, Q)
    torch.cuda.synchronize()
    out = Q.cpu().numpy()
    plan.close()
    return out


CASES = {
    # d, M, k, dense band, empty band
    "m64_mixed": (1_000_000, 64, 10_000, (200_000, 230_000), (600_000, 700_000)),
    "m1_band": (100_000, 1, 20_000, (10_000, 30_000), (50_000, 90_000)),
    "m3_kd": (3001, 3, 3001, None, None),
    "m4_kd": (5000, 4, 5000, None, None),
    "m7_mixed": (300_000, 7, 6_000, (40_000, 46_000), (100_000, 200_000)),
    "m65_mixed": (200_000, 65, 3_000, (20_000, 26_000), (100_000, 150_000)),
    "m130_mixed": (100_000, 130, 1_500, (8_000, 12_000), (50_000, 60_000)),
    "m64_sparse": (300_000, 64, 1_000, None, None),
    # fewer entries per tile than workers (the direct path), next to tiles
    # that take the other routes
    "m64_few": (2_000_000, 64, 100, (1_000_000, 1_004_000), None),
    "m130_few": (1_000_000, 130, 50, (500_000, 502_000), None),
    # many groups of 64 workers: 16 sparse groups per tile; five dense groups
    "m1024_sparse": (20_000, 1024, 20, None, None),
    "m300_dense": (30_000, 300, 10_000, (0, 20_000), None),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_topk_average_matches_oracle(name):
    d, M, k, band, empty = CASES[name]
    print("case", name, "d", d, "M", M, "k", k, flush=True)
    w = custom(d=d, M=M, kind="topk", k=k, eta=1e-2, seed=61)
    idx, val = _messages(d, M, k, seed=sorted(CASES).index(name), dense_band=band, empty_band=empty)
    got = _gpu_average(w, idx, val)
    exp = _oracle_average(w, idx, val)
    bad = np.flatnonzero(got.view(np.uint32) != exp.view(np.uint32))
    assert bad.size == 0, "%d of %d differ; first at %s: got %s expected %s" % (
        bad.size, got.size, bad[:5].tolist(), got[bad[:5]].tolist(), exp[bad[:5]].tolist())
    assert np.signbit(got[ALL_NEG0]) and got[ALL_NEG0] == 0
    if M >= 3:
        assert not np.signbit(got[ALL_BUT_ONE_NEG0]) and not np.signbit(got[ONE_NEG0])


def _gap_messages(M, k, seed):
    """Sorted lists whose consecutive entries lie 0, 1, 2, 7, 8, 9, 10, 40 or
    120 column tiles (2048 columns) apart, at most four in one tile: the
    tiles between two entries have no entry of that worker, and a run of
    four entries starts anything from none to hundreds of tiles."""
    rng = np.random.default_rng(seed)
    gaps = np.array([0, 0, 1, 2, 7, 8, 9, 10, 40, 120])
    cols = []
    for m in range(M):
        g = rng.choice(gaps, size=k)
        g[0] = rng.integers(0, 3)
        run = 0
        for j in range(1, k):  # at most four entries per tile
            run = run + 1 if g[j] == 0 else 0
            if run == 4:
                g[j], run = 1, 0
        T = np.cumsum(g)
        off = np.empty(k, np.int64)
        for t in np.unique(T):
            sel = np.flatnonzero(T == t)
            off[sel] = np.sort(rng.choice(2048, size=sel.size, replace=False))
        cols.append(T * 2048 + off)
    d = int(max(c[-1] for c in cols)) + 1 + int(rng.integers(0, 5000))
    idx = np.stack(cols).astype(np.uint32)
    val = (rng.standard_normal((M, k)) * 10.0 ** rng.uniform(-8, 8, (M, k))).astype(np.float32)
    return d, idx, val


@pytest.mark.parametrize("M,k", [(6, 300), (66, 40)])
def test_topk_average_runs_of_empty_tiles(M, k):
    """Runs of empty tiles of every length between a worker's entries, so
    that the starts of each tile are written both by the lane whose entry
    follows the run and, for long runs, by the whole wave."""
    d, idx, val = _gap_messages(M, k, seed=M)
    print("gaps M", M, "k", k, "d", d, flush=True)
    w = custom(d=d, M=M, kind="topk", k=k, eta=1e-2, seed=64)
    got = _gpu_average(w, idx, val)
    exp = _oracle_average(w, idx, val)
    bad = np.flatnonzero(got.view(np.uint32) != exp.view(np.uint32))
    assert bad.size == 0, "%d of %d differ; first at %s" % (bad.size, got.size, bad[:5].tolist())


@pytest.mark.timeout(300)
def test_topk_average_full_size_equals_fused_step():
    """The largest workload's server average (d = 1e8, M = 64, k = 1e6) from
    dqgan_aggregate equals the one the fused step computes, bit for bit."""
    import torch
    import synth
    from paper_2010_13359_amd import dqgan
    w = synth.get(4)
    print("C4 average", flush=True)
    dev = torch.device("cuda:0")
    plan = dqgan.Plan.from_workload(w)
    E = torch.zeros((w.M, w.ld), dtype=torch.float32, device=dev)
    W = synth.init_params(w, device=dev)
    WX = torch.empty((w.M, w.ld), dtype=torch.float32, device=dev)
    wire = plan.new_wire(dev)
    Qf = torch.empty(w.ld, dtype=torch.float32, device=dev)
    G = synth.gradients(w, 1, device=dev)
    dqgan.step_scales(plan, w.eta, G, E, wire)
    dqgan.step_apply(plan, w.eta, 1, G, E, W, WX, wire, Qf)
    del G, E, WX
    Qa = torch.full((w.ld,), float("nan"), dtype=torch.float32, device=dev)
    dqgan.aggregate(plan, wire, Qa)
    torch.cuda.synchronize()
    same = torch.equal(Qa.view(torch.int32), Qf.view(torch.int32))
    n_bad = int((Qa.view(torch.int32) != Qf.view(torch.int32)).sum())
    plan.close()
    assert same, "%d columns differ" % n_bad


def test_topk_average_skips_indices_beyond_d():
    """Sorted lists whose last entries lie at or beyond d (in the padding
    [d, ld) and past ld) average as if those entries were not sent."""
    d, M, k = 100_001, 9, 3_000
    w = custom(d=d, M=M, kind="topk", k=k, eta=1e-2, seed=62)
    idx, val = _messages(d, M, k, seed=71, dense_band=(40_000, 44_000))
    tail = np.array([d, d + 5, w.ld - 1, w.ld, w.ld + 70_000, 2 ** 32 - 1], np.uint32)
    for m in range(M):
        # the last len(tail) entries of each list move past d (still ascending)
        idx[m, -len(tail):] = tail
    got = _gpu_average(w, idx, val)
    keep = idx.astype(np.int64) < d
    ph = np.zeros((M, w.ld), np.float32)
    for m in range(M):
        ph[m, idx[m][keep[m]].astype(np.int64)] = val[m][keep[m]]
    from oracle import oracle as orc
    exp = np.zeros(w.ld, np.float32)
    exp[:d] = orc.aggregate(ph, d)
    assert np.array_equal(got.view(np.uint32), exp.view(np.uint32))


def test_topk_malformed_messages_complete_and_leave_the_plan_usable():
    """Unsorted lists, repeated indices and indices far beyond d give
    undefined values (the header's contract) but complete without touching
    memory outside the buffers; the same plan then averages a well-formed
    message exactly."""
    import torch
    from paper_2010_13359_amd import dqgan
    d, M, k = 50_000, 5, 4_000
    w = custom(d=d, M=M, kind="topk", k=k, eta=1e-2, seed=63)
    rng = np.random.default_rng(72)
    bad_idx = rng.integers(0, 2 ** 32, size=(M, k), dtype=np.uint64).astype(np.uint32)
    bad_idx[:, ::3] = rng.integers(0, d, size=(M, (k + 2) // 3)).astype(np.uint32)  # in range, unsorted
    bad_idx[:, 1::7] = 1234  # repeated
    bad_val = rng.standard_normal((M, k)).astype(np.float32)
    good_idx, good_val = _messages(d, M, k, seed=73, dense_band=(10_000, 20_000))
    dev = torch.device("cuda:0")
    plan = dqgan.Plan.from_workload(w)
    wire = plan.new_wire(dev)
    Q = torch.full((w.ld,), float("nan"), dtype=torch.float32, device=dev)
    Ph = torch.full((M, w.ld), float("nan"), dtype=torch.float32, device=dev)
    wire.idx.copy_(torch.from_numpy(bad_idx.reshape(-1).view(np.int32)).to(dev))
    wire.val.copy_(torch.from_numpy(bad_val.reshape(-1)).to(dev))
    dqgan.aggregate(plan, wire, Q)
    dqgan.unpack(plan, wire, Ph)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(Q).all()) and bool(torch.isfinite(Ph).all())
    wire.idx.copy_(torch.from_numpy(good_idx.reshape(-1).view(np.int32)).to(dev))
    wire.val.copy_(torch.from_numpy(good_val.reshape(-1)).to(dev))
    dqgan.aggregate(plan, wire, Q)
    torch.cuda.synchronize()
    got = Q.cpu().numpy()
    plan.close()
    exp = _oracle_average(w, good_idx, good_val)
    assert np.array_equal(got.view(np.uint32), exp.view(np.uint32))
