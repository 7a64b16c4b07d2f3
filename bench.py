"""Benchmark of the fused DQGAN iteration (Algorithm 2 of arXiv:2010.13359)
on one MI355X.

One step = one full iteration over all M workers: EF accumulate, compress,
pack, EF residual, server average, OMD update and the M extrapolated points,
as the two passes of the library (dqgan_step_scales, dqgan_step_apply).
Inputs (gradients, residuals, parameters) are resident in HBM before the timed
region; two gradient batches alternate between steps.

Prints one JSON line.  `value` is gradient GB/s = M * d * 4 bytes / step time
of the headline workload (C3 unless --config says otherwise); by default
`also_measured` carries the same record for C4 (top-k, 64 x 10^8), timed
in the same process after it.
`roofline` is the dominant kernel (the apply pass) against the 8 TB/s HBM
peak, with its algorithmic bytes per launch; `step_roofline` is the same for
the whole step, plus the HBM bytes the rocprofv3 counters measured for the
step's two main kernels (profiles/traffic.json) over the step time.  `cpu_baseline` is the oracle (single-threaded C) on a
bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3] [--also 4|none] [--graph]
"""
import argparse
import hashlib
import glob
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "GB/s of gradient processed per fused compress+EF+aggregate+OMD step; % HBM peak"


KERNEL_SOURCES = {
    "dense": ("dense.hip", "device.hpp", "plan.hpp"),
    "topk": ("topk.hip", "device.hpp", "plan.hpp"),
}


def _code_only(text):
    """Source text without comments and blank lines: comment edits do not
    change what the counters measured."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = (re.sub(r"//.*$", "", line).rstrip() for line in text.splitlines())
    return "\n".join(line for line in lines if line.strip())


def source_hash(group="dense"):
    """Hash of the code a kernel family is built from (the counters in
    profiles/traffic.json are valid only for the code they were taken on)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[group]:
        p = os.path.join(ROOT, "paper_2010_13359_amd", "csrc", name)
        with open(p, encoding="utf-8") as f:
            h.update(os.path.basename(p).encode())
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def wire_bits(w):
    if w.kind == "sign":
        return 1.0
    if w.kind == "qsgd":
        return 1.0 + (8 if w.levels == 255 else 4)
    if w.kind == "mbit":
        return float(w.levels)
    if w.kind == "topk":
        return 64.0 * w.k / w.d
    return 32.0


def algorithmic_bytes(w):
    """Bytes the iteration must move at minimum: per (worker, element) read g,
    read and write e, write the evaluation point, write the message; per
    element read and write w; per (worker, segment) the scale."""
    per_mi = 16.0 + wire_bits(w) / 8.0
    scales = 4.0 * w.M * w.n_seg if w.kind in ("sign", "qsgd", "mbit") else 0.0
    return w.M * w.d * per_mi + 8.0 * w.d + scales


def workload_label(w):
    if w.kind == "sign":
        comp = "scaled sign (L1 mean)"
    elif w.kind == "qsgd":
        comp = "s-level quantizer s=%d %s" % (w.levels, w.norm.upper())
    elif w.kind == "mbit":
        comp = "%d-bit sign-magnitude quantizer (k=%d) %s" % (w.levels, (1 << (w.levels - 1)) - 1, w.norm.upper())
    elif w.kind == "topk":
        comp = "top-k k=%d" % w.k
    else:
        comp = "identity"
    scope = "per row" if w.kind == "topk" else "%d segments" % w.n_seg
    return "C%d %s: d=%d, M=%d workers, %s, %s, eta=%g" % (w.index, w.name, w.d, w.M, comp, scope, w.eta)


def separate_calls(plan, w, G, E, W, WX, wire, dev, reps=5):
    """The worker and server sides as separate calls (what a multi-process
    deployment would run): dqgan_compress_ef (both passes), dqgan_aggregate
    and dqgan_omd_step, each timed with HIP events after the step's timed
    region, with the algorithmic bytes of each call's one pass."""
    import torch
    from paper_2010_13359_amd import dqgan
    Q = torch.empty(w.ld, dtype=torch.float32, device=dev)
    msg = w.M * w.d * wire_bits(w) / 8.0
    scales = 4.0 * w.M * w.n_seg if w.kind in ("sign", "qsgd", "mbit") else 0.0
    calls = {
        "compress_ef": (lambda: dqgan.compress_ef(plan, w.eta, 1, G, E, None, wire),
                        12.0 * w.M * w.d + msg + scales),
        "aggregate": (lambda: dqgan.aggregate(plan, wire, Q), msg + scales + 4.0 * w.d),
        "omd_step": (lambda: dqgan.omd_step(plan, w.eta, Q, W, G, E, WX), 12.0 * w.M * w.d + 12.0 * w.d),
    }
    res = {}
    for name, (fn, alg) in calls.items():
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        res[name] = {"ms": round(ms, 4), "algorithmic_GB/s": round(alg / (ms * 1e-3) / 1e9, 1)}
    del Q
    return res


def traffic_record(kernel_key, group):
    """HBM bytes per launch from the committed rocprofv3 counter summary,
    if it was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            rec = json.load(f).get(kernel_key)
    except (ValueError, OSError):
        return None
    if not rec or rec.get("source_hash") != source_hash(group):
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(w, target_elems=4_000_000):
    """The oracle on the first segments of the workload (all M workers),
    timed on this host; single thread."""
    import numpy as np
    import synth
    from synth.configs import custom
    from oracle import oracle as orc
    offs = [o for o in w.seg_offsets if o <= target_elems]
    if len(offs) < 2:
        offs = [0, min(w.d, target_elems)]
    n = offs[-1]
    nseg = len(offs) - 1
    sub = custom(d=n, M=w.M, kind=w.kind, levels=w.levels, k=max(1, w.k * n // w.d) if w.k else 0,
                 seg_offsets=offs if w.kind != "topk" else None, norm=w.norm if w.kind in ("sign", "qsgd", "mbit") else None,
                 eta=w.eta, seed=w.seed, law=w.law, group_scale=w.group_scale[:nseg])
    G = synth.gradients_np(sub, 1)
    E = np.zeros((sub.M, sub.ld), np.float32)
    W = synth.init_params_np(sub)
    orc.lib()
    t0 = time.perf_counter()
    orc.step(sub.as_dict(), np.float32(sub.eta), 1, G, E, W)
    dt = time.perf_counter() - t0
    gbs = sub.M * sub.d * 4 / dt / 1e9
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": "one full iteration over the first %d segments (d=%d of %d, all %d workers), "
                      "%.1f s, single-threaded C oracle; host reports %d CPUs" % (nseg, sub.d, w.d, w.M, dt,
                                                                                 os.cpu_count() or 0)}


def measure(w, steps, warmup, graph_mode=False, copy_calibration=False, extras=True):
    """Time `steps` iterations of workload `w` (after `warmup` untimed ones)
    on cuda:0 and return the record: step time, gradient GB/s, the apply
    pass against the HBM peak (`roofline`), the whole step (`step_roofline`)
    and, with `extras`, the reference streams and the separate calls."""
    import torch
    import synth
    from paper_2010_13359_amd import dqgan

    dev = torch.device("cuda:0")
    print("bench: workload %s" % workload_label(w), file=sys.stderr, flush=True)
    plan = dqgan.Plan.from_workload(w)
    Gs = [synth.gradients(w, t, device=dev) for t in (1, 2)]
    E = torch.zeros((w.M, w.ld), dtype=torch.float32, device=dev)
    W = synth.init_params(w, device=dev)
    WX = torch.empty((w.M, w.ld), dtype=torch.float32, device=dev)
    wire = plan.new_wire(dev)
    torch.cuda.synchronize()

    def one(t, ev=None):
        G = Gs[t % 2]
        if ev:
            ev[0].record()
        dqgan.step_scales(plan, w.eta, G, E, wire)
        if ev:
            ev[1].record()
        dqgan.step_apply(plan, w.eta, t, G, E, W, WX, wire)
        if ev:
            ev[2].record()

    for t in range(1, warmup + 1):
        one(t)
    torch.cuda.synchronize()
    if copy_calibration:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    graph = None
    if graph_mode:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for k in range(steps):
                one(warmup + 1 + k)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record()
    if graph is not None:
        graph.replay()
    else:
        for k in range(steps):
            one(warmup + 1 + k, evs[k])
    stop.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    total_ms = start.elapsed_time(stop)
    if graph is not None:
        # per-pass times: the same iterations again, eagerly, with events
        for k in range(steps):
            one(warmup + 1 + k, evs[k])
        torch.cuda.synchronize()
    scales_ms = [e[0].elapsed_time(e[1]) for e in evs]
    apply_ms = [e[1].elapsed_time(e[2]) for e in evs]
    ms_step = total_ms / steps
    grad_bytes = w.M * w.d * 4.0
    value = grad_bytes / (ms_step * 1e-3) / 1e9
    b_alg = algorithmic_bytes(w)
    t_apply = sum(apply_ms) / len(apply_ms)
    t_scales = sum(scales_ms) / len(scales_ms)
    achieved = b_alg / (t_apply * 1e-3) / 1e9
    step_ach = b_alg / (ms_step * 1e-3) / 1e9
    kernel_key = "apply_C%d" % w.index
    traffic = traffic_record(kernel_key, "dense")  # the apply pass of every compressor is in dense.hip
    # the statistics pass's main kernel: segment partials, or top-k's full pass
    stats_traffic = traffic_record("stats_C%d" % w.index, "topk" if w.kind == "topk" else "dense")
    step_counter = (traffic + stats_traffic) if (traffic and stats_traffic) else None
    out = {
        "value": round(value, 2), "unit": "GB/s", "steps": steps, "warmup": warmup,
        "ms_per_step": round(ms_step, 4),
        "config": {"workload": workload_label(w), "d": w.d, "M": w.M, "compressor": w.kind, "levels": w.levels,
                   "k": w.k, "segments": w.n_seg, "parallelism": "single GPU; M workers as rows",
                   "launch": "hip graph of the timed iterations" if graph_mode else "eager"},
        "roofline": {"bound": "hbm", "kernel": "dqgan_step_apply (fused encode+EF+aggregate+OMD pass)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": b_alg, "ms_per_launch": round(t_apply, 4)},
        "step_roofline": {"achieved": round(step_ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(step_ach / HBM_PEAK_GBS, 4), "ms_scales_pass": round(t_scales, 4),
                          "ms_apply_pass": round(t_apply, 4),
                          # HBM bytes the counters saw for the two main kernels of the step
                          # (re-reads of the statistics pass included) per step time
                          "counter_bytes": step_counter,
                          "counter_frac": (round(step_counter / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
                                           if step_counter else None)},
        "hbm_pct_of_peak": round(100 * step_ach / HBM_PEAK_GBS, 2),
        "wall_s_timed": round(t_wall, 3),
    }
    # Reference stream in the same process and on the same buffers (the
    # reachable HBM rate of mixed read/write streams differs between
    # allocations and boxes by up to 20 %): out = g + e, 2 reads + 1 write.
    ref_ms = []
    for _ in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        torch.add(Gs[0], E, out=WX)
        b.record()
        torch.cuda.synchronize()
        ref_ms.append(a.elapsed_time(b))
    ref_t = sorted(ref_ms)[1]
    out["reference_stream"] = {"op": "torch.add(g, e, out=WX) over the step's own [M][ld] buffers (2 reads, 1 write)",
                               "GB/s": round(3 * 4.0 * w.M * w.ld / (ref_t * 1e-3) / 1e9, 1),
                               "ms": round(ref_t, 4)}
    # Plain copy over the same buffers (1 read, 1 write; torch's vectorized
    # elementwise kernel, faster here than the runtime's copy kernel): the
    # reachable rate of a compute-free stream in this process, against which
    # the dominant kernel's rate is also given.
    cp_ms = []
    for _ in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        torch.mul(Gs[0], 1.0, out=WX)
        b.record()
        torch.cuda.synchronize()
        cp_ms.append(a.elapsed_time(b))
    cp_t = sorted(cp_ms)[1]
    cp_gbs = 2 * 4.0 * w.M * w.ld / (cp_t * 1e-3) / 1e9
    out["copy_ceiling"] = {"op": "torch.mul(g, 1.0, out=WX) over the step's own [M][ld] buffers (1 read, 1 write)",
                           "GB/s": round(cp_gbs, 1), "ms": round(cp_t, 4),
                           "roofline_frac_of_copy": round(achieved / cp_gbs, 4),
                           "step_frac_of_copy": round(step_ach / cp_gbs, 4),
                           "step_counter_frac_of_copy": (round(step_counter / (ms_step * 1e-3) / 1e9 / cp_gbs, 4)
                                                         if step_counter else None)}
    if extras:
        out["separate_calls"] = separate_calls(plan, w, Gs[0], E, W, WX, wire, dev)
    del graph
    plan.close()
    del Gs, E, W, WX, wire
    torch.cuda.empty_cache()
    return out


ALLOC_PADS_MIB = [0, 1, 3, 64, 130, 0, 2, 7, 513, 5]


def alloc_trials(w, n, steps):
    """Allocate the workload's buffers n times in this process (a padding
    allocation of a few MiB before each, freed and returned to the driver
    after each trial) and time `steps` iterations of each allocation.  The
    same kernels on the same sizes run at different speeds depending on the
    physical memory behind the buffers; this shows the spread.  One JSON line
    per trial: the apply pass and the step in ms."""
    import torch
    import synth
    from paper_2010_13359_amd import dqgan
    dev = torch.device("cuda:0")
    for trial in range(n):
        pad_mib = ALLOC_PADS_MIB[trial % len(ALLOC_PADS_MIB)]
        pad = torch.empty(pad_mib * 2 ** 18 + 1, device=dev) if pad_mib else None
        plan = dqgan.Plan.from_workload(w)
        G = synth.gradients(w, 1, device=dev)
        E = torch.zeros((w.M, w.ld), dtype=torch.float32, device=dev)
        W = synth.init_params(w, device=dev)
        WX = torch.empty((w.M, w.ld), dtype=torch.float32, device=dev)
        wire = plan.new_wire(dev)
        apply_ms, step_ms = [], []
        for t in range(steps + 1):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            ev[0].record()
            dqgan.step_scales(plan, w.eta, G, E, wire)
            ev[1].record()
            dqgan.step_apply(plan, w.eta, t + 1, G, E, W, WX, wire)
            ev[2].record()
            torch.cuda.synchronize()
            if t > 0:  # the first iteration of each allocation is a warmup
                apply_ms.append(ev[1].elapsed_time(ev[2]))
                step_ms.append(ev[0].elapsed_time(ev[2]))
        print(json.dumps({"trial": trial, "workload": workload_label(w), "pad_mib": pad_mib,
                          "apply_ms": round(sum(apply_ms) / len(apply_ms), 3),
                          "step_ms": round(sum(step_ms) / len(step_ms), 3)}), flush=True)
        del G, E, W, WX, wire, pad
        plan.close()
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3, help="workload index C0..C6 (default C3)")
    ap.add_argument("--also", default=None,
                    help="comma-separated workload indices timed after the headline one and reported in "
                         "`also_measured` (default: 4 when the headline is C3, else none; 'none' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain device copy of 1 GiB (counter calibration)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the timed iterations in one HIP graph and time its replay (launch-bound sizes); "
                         "the per-pass times then come from an eager run of the same iterations")
    ap.add_argument("--alloc-trials", type=int, default=0, metavar="N",
                    help="instead of the bench line: allocate the workload N times in one process and print "
                         "the apply-pass and step time of each allocation (one JSON line each)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU; --gpus %d is not offered (the M workers are the rows of "
              "one batched matrix on a single device)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import synth

    torch.cuda.set_device(torch.device("cuda:0"))
    w = synth.get(args.config)
    if args.alloc_trials:
        alloc_trials(w, args.alloc_trials, max(1, min(args.steps, 5)))
        return
    rec = measure(w, args.steps, args.warmup, args.graph, args.copy_calibration)
    out = {"metric": METRIC, "value": rec.pop("value"), "unit": rec.pop("unit"), "n_gpus": 1,
           "steps": rec.pop("steps"), "warmup": rec.pop("warmup"), "ms_per_step": rec.pop("ms_per_step"),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic"}
    out.update(rec)
    also = args.also if args.also is not None else ("4" if args.config == 3 else "none")
    if also != "none":
        # the other workload the HBM target names (C4, top-k over 64 x 10^8),
        # timed in the same process after the headline one
        out["also_measured"] = []
        for idx in [int(x) for x in also.split(",") if x.strip()]:
            other = measure(synth.get(idx), args.steps, min(args.warmup, 3), args.graph, extras=False)
            out["also_measured"].append(other)
    if not args.no_cpu_baseline:
        print("bench: timing the oracle on a sample", file=sys.stderr, flush=True)
        # about 10-30 s of single-core work: the sort-based top-k oracle is
        # slower per element than the quantizers'
        out["cpu_baseline"] = cpu_baseline(w, 4_000_000 if w.kind == "topk" else 18_000_000)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
