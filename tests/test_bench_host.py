"""Host-side checks of bench.py (no GPU): workload labels and algorithmic
byte counts for every workload, and the refusal of more than one GPU."""
import subprocess
import sys

import bench
import synth


def test_labels_and_bytes_for_every_workload():
    for i in range(7):
        w = synth.get(i)
        label = bench.workload_label(w)
        assert ("d=%d" % w.d) in label and ("M=%d" % w.M) in label
        b = bench.algorithmic_bytes(w)
        assert 16 * w.M * w.d < b < 18 * w.M * w.d + 8 * w.d + 4 * w.M * w.n_seg + 1


def test_c3_algorithmic_bytes():
    w = synth.get(3)
    # 16 B + 5 wire bits per (worker, element); 8 B per element for w; 4 B per scale
    assert bench.algorithmic_bytes(w) == w.M * w.d * (16 + 5 / 8) + 8 * w.d + 4 * w.M * w.n_seg


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=bench.ROOT, capture_output=True, text=True)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_code_hash_ignores_comments_only():
    src = "int a; // count\n/* block\n comment */\nint b;  \n\n"
    assert bench._code_only(src) == "int a;\nint b;"
    assert bench._code_only(src) == bench._code_only(src.replace("// count", "// another comment"))
    assert bench._code_only(src) != bench._code_only(src.replace("int b;", "int c;"))


def test_committed_counter_records_match_the_kernel_code():
    """profiles/traffic.json was taken on the kernel code in the tree (the
    bench reports its bytes only then)."""
    for key, group in (("apply_C3", "dense"), ("stats_C3", "dense"), ("apply_C4", "dense"), ("stats_C4", "topk")):
        assert bench.traffic_record(key, group), key
