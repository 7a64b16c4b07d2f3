"""Summarize a rocprofv3 results database (rocpd SQLite): per kernel, the
dispatch count and duration statistics, and for counter runs the mean value of
each counter per dispatch.

    python -m paper_2010_13359_amd.rocprof_summary RESULTS.db [--skip-first N | --counters | --dispatches NAME |
                                                              --per-trial KERNEL GROUP]
"""
import argparse
import re
import sqlite3
import sys


def short_name(name):
    """'void ns::k_fused<1, 4, 32>(float const*, ...)' -> 'k_fused<1, 4, 32>'."""
    s = re.sub(r"^void\s+", "", name).replace("(anonymous namespace)", "anon")
    depth, cut, last_sep = 0, len(s), 0
    for i, ch in enumerate(s):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            cut = i
            break
        elif ch == ":" and depth == 0 and s[i:i + 2] == "::":
            last_sep = i + 2
    s = s[last_sep:cut]
    return s if len(s) <= 90 else s[:87] + "..."


def kernel_stats(db, skip_first=0):
    """Per kernel: dispatch count and duration statistics, leaving out the
    first `skip_first` dispatches of each kernel (warmup iterations)."""
    con = sqlite3.connect(db)
    rows = con.execute("select name, duration from kernels order by start").fetchall()
    agg = {}
    for name, dur in rows:
        key = short_name(name)
        a = agg.setdefault(key, [])
        a.append(float(dur))
    out = []
    for k, v in agg.items():
        v = v[skip_first:] if len(v) > skip_first else v
        v.sort()
        out.append((k, len(v), sum(v) / len(v) / 1e3, v[len(v) // 2] / 1e3, v[0] / 1e3, v[-1] / 1e3, sum(v) / 1e3))
    out.sort(key=lambda r: -r[6])
    return out


def counter_stats(db):
    con = sqlite3.connect(db)
    rows = con.execute("select kernel_name, counter_name, dispatch_id, value from counters_collection").fetchall()
    per = {}
    for name, ctr, disp, val in rows:
        key = (short_name(name), ctr)
        per.setdefault(key, {}).setdefault(disp, 0.0)
        per[key][disp] += float(val)
    out = []
    for (k, ctr), d in per.items():
        vals = list(d.values())
        out.append((k, ctr, len(vals), sum(vals) / len(vals)))
    out.sort()
    return out


def counter_dispatches(db, match):
    """Per dispatch of kernels whose name contains `match`: grid size and
    counter values (for the copy-kernel calibration of the byte counters)."""
    con = sqlite3.connect(db)
    cols = [r[1] for r in con.execute("pragma table_info(counters_collection)")]
    grid = next((c for c in ("grid_size_x", "grid_x", "grid_size") if c in cols), None)
    rows = con.execute("select kernel_name, counter_name, dispatch_id, value, %s from counters_collection"
                       % (grid or "0")).fetchall()
    per = {}
    for name, ctr, disp, val, grid in rows:
        if match not in name:
            continue
        d = per.setdefault(disp, {"kernel": short_name(name), "grid": grid})
        d[ctr] = d.get(ctr, 0.0) + float(val)
    return [dict(v, dispatch=k) for k, v in sorted(per.items())]


def per_trial(db, match, group):
    """Dispatches of the kernel whose short name equals `match`, in launch
    order, taken in consecutive groups of `group` (one group per allocation
    trial of bench.py --alloc-trials); per group, leaving out its first
    dispatch (the warmup): mean duration and mean of each counter."""
    con = sqlite3.connect(db)
    disp = [(d, float(u)) for n, u, d in con.execute("select name, duration, dispatch_id from kernels order by start")
            if short_name(n) == match]
    ctr = {}
    for name, c, d, v in con.execute("select kernel_name, counter_name, dispatch_id, value from counters_collection"):
        if short_name(name) == match:
            ctr.setdefault(d, {}).setdefault(c, 0.0)
            ctr[d][c] += float(v)
    out = []
    for t in range(len(disp) // group):
        grp = disp[group * t + 1: group * (t + 1)]
        if not grp:
            continue
        rec = {"trial": t, "us": sum(u for _, u in grp) / len(grp) / 1e3}
        names = sorted(ctr.get(grp[0][0], {}))
        for c in names:
            rec[c] = sum(ctr[d][c] for d, _ in grp) / len(grp)
        out.append(rec)
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("db")
    ap.add_argument("--counters", action="store_true")
    ap.add_argument("--dispatches", metavar="NAME", help="per-dispatch counters of kernels whose name contains NAME")
    ap.add_argument("--skip-first", type=int, default=0, metavar="N",
                    help="leave out the first N dispatches of each kernel (warmup) from the duration statistics")
    ap.add_argument("--per-trial", nargs=2, metavar=("KERNEL", "GROUP"),
                    help="mean duration and counters of KERNEL per consecutive group of GROUP dispatches")
    a = ap.parse_args(argv)
    if a.per_trial:
        for rec in per_trial(a.db, a.per_trial[0], int(a.per_trial[1])):
            print("trial %-3d %10.1f us  %s" % (rec.pop("trial"), rec.pop("us"),
                                                "  ".join("%s=%.1f" % kv for kv in rec.items())))
        return 0
    if a.dispatches:
        for d in counter_dispatches(a.db, a.dispatches):
            vals = "  ".join("%s=%.1f" % (k, v) for k, v in d.items() if k not in ("kernel", "grid", "dispatch"))
            print("dispatch %-6d %-40s grid %-10s %s" % (d["dispatch"], d["kernel"][:40], d["grid"], vals))
        return 0
    if a.counters:
        print("%-60s %-12s %8s %16s" % ("kernel", "counter", "calls", "mean/dispatch"))
        for k, ctr, n, mean in counter_stats(a.db):
            print("%-60s %-12s %8d %16.1f" % (k[:60], ctr, n, mean))
    else:
        print("%-60s %6s %12s %12s %12s %12s %14s" % ("kernel", "calls", "avg_us", "median_us", "min_us", "max_us",
                                                       "total_us"))
        for k, n, avg, med, mn, mx, tot in kernel_stats(a.db, a.skip_first):
            print("%-60s %6d %12.1f %12.1f %12.1f %12.1f %14.1f" % (k[:60], n, avg, med, mn, mx, tot))
    return 0


if __name__ == "__main__":
    sys.exit(main())
