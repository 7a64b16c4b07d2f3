"""Host logic of the profile summaries (paper_2010_13359_amd/rocprof_summary.py)
on a small synthetic rocpd-style SQLite database: kernel-name shortening,
warmup dispatches left out of the duration statistics, counters summed over
the samples of a dispatch and averaged over dispatches."""
import sqlite3

from paper_2010_13359_amd import rocprof_summary as rs

FUSED = ("void dq::(anonymous namespace)::k_fused_split<1, 4, 4, 8, false>(float const*, float*, float*, "
         "float*, float*, unsigned int*, unsigned int*, float*)")
STATS = "void dq::(anonymous namespace)::k_segment_partials<2>(float const*, float const*, float, long)"


def _db(tmp_path):
    path = str(tmp_path / "run_results.db")
    con = sqlite3.connect(path)
    con.execute("create table kernels (name text, duration integer, start integer)")
    # fused: a slow warmup dispatch, then 3000, 2000, 4000 ns; stats: 1000, 1000
    for i, (name, dur) in enumerate([(FUSED, 9000), (STATS, 1000), (FUSED, 3000), (FUSED, 2000), (STATS, 1000),
                                     (FUSED, 4000)]):
        con.execute("insert into kernels values (?, ?, ?)", (name, dur, 10 * i))
    con.execute("create table counters_collection (kernel_name text, counter_name text, dispatch_id integer, "
                "value real, grid_size_x integer)")
    # two samples per dispatch (summed), two dispatches (averaged)
    for disp, vals in ((7, (10.0, 20.0)), (9, (40.0, 50.0))):
        for v in vals:
            con.execute("insert into counters_collection values (?, ?, ?, ?, ?)", (FUSED, "FETCH_SIZE", disp, v, 4096))
    con.commit()
    con.close()
    return path


def test_short_names():
    assert rs.short_name(FUSED) == "k_fused_split<1, 4, 4, 8, false>"
    assert rs.short_name(STATS) == "k_segment_partials<2>"


def test_kernel_stats_skip_warmup(tmp_path):
    db = _db(tmp_path)
    rows = {r[0]: r for r in rs.kernel_stats(db, skip_first=1)}
    name, calls, avg, med, mn, mx, tot = rows["k_fused_split<1, 4, 4, 8, false>"]
    assert calls == 3 and avg == 3.0 and med == 3.0 and mn == 2.0 and mx == 4.0 and tot == 9.0
    assert rows["k_segment_partials<2>"][1] == 1
    all_rows = {r[0]: r for r in rs.kernel_stats(db)}
    assert all_rows["k_fused_split<1, 4, 4, 8, false>"][1] == 4


def test_counter_stats_sum_then_mean(tmp_path):
    db = _db(tmp_path)
    (k, ctr, n, mean), = rs.counter_stats(db)
    assert (k, ctr, n) == ("k_fused_split<1, 4, 4, 8, false>", "FETCH_SIZE", 2) and mean == 60.0
    disp = rs.counter_dispatches(db, "k_fused_split")
    assert [(d["dispatch"], d["grid"], d["FETCH_SIZE"]) for d in disp] == [(7, 4096, 30.0), (9, 4096, 90.0)]


def test_per_trial_groups_dispatches(tmp_path):
    """--per-trial: a kernel's dispatches in launch order, in groups (one per
    allocation trial); per group the first (warmup) is left out."""
    path = str(tmp_path / "trials.db")
    con = sqlite3.connect(path)
    con.execute("create table kernels (name text, duration integer, start integer, dispatch_id integer)")
    con.execute("create table counters_collection (kernel_name text, counter_name text, dispatch_id integer, "
                "value real)")
    # two trials of 3 dispatches each, a statistics dispatch between them
    plan = [(FUSED, 9000, 10.0), (FUSED, 2000, 1.0), (FUSED, 4000, 3.0), (STATS, 500, 99.0),
            (FUSED, 8000, 50.0), (FUSED, 6000, 5.0), (FUSED, 8000, 7.0)]
    for i, (name, dur, ctr) in enumerate(plan):
        con.execute("insert into kernels values (?, ?, ?, ?)", (name, dur, 10 * i, 100 + i))
        for half in (0.25, 0.75):  # two samples per dispatch, summed
            con.execute("insert into counters_collection values (?, ?, ?, ?)", (name, "X", 100 + i, half * ctr))
    con.commit()
    con.close()
    recs = rs.per_trial(path, "k_fused_split<1, 4, 4, 8, false>", 3)
    assert [r["trial"] for r in recs] == [0, 1]
    assert abs(recs[0]["us"] - 3.0) < 1e-9 and abs(recs[1]["us"] - 7.0) < 1e-9
    assert abs(recs[0]["X"] - 2.0) < 1e-9 and abs(recs[1]["X"] - 6.0) < 1e-9
