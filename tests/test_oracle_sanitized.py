"""The oracle's pins again, with the oracle built under AddressSanitizer and
UndefinedBehaviorSanitizer (gcc, host code only): an out-of-bounds access,
a use after free, a signed overflow, an invalid shift or a misaligned access
anywhere the pins drive it stops the run.  The interpreter is not
instrumented, so the sanitizer runtimes are preloaded into the child
process; leak checking is off (the interpreter itself keeps memory to the
end).  CPU only."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_FILES = sorted(glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
SANITIZE = "-fsanitize=address,undefined -fno-sanitize-recover=all -fno-omit-frame-pointer -g"


def _runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=%s" % name], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _run_pins(tmp_path, source):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not (asan and ubsan):
        pytest.skip("gcc's sanitizer runtimes are not installed")
    d = str(tmp_path / "oracle")
    os.makedirs(d)
    with open(os.path.join(d, "dqgan_oracle.c"), "w") as f:
        f.write(source)
    # the runtimes first (ASan requires it), anything already preloaded kept
    preload = ":".join(p for p in (asan, ubsan, os.environ.get("LD_PRELOAD", "")) if p)
    env = dict(os.environ, DQGAN_ORACLE_DIR=d, DQGAN_ORACLE_EXTRA_CFLAGS=SANITIZE, LD_PRELOAD=preload,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    pins = [f for f in PIN_FILES if not f.endswith("test_oracle_sanitized.py")]
    # -s: a sanitizer report is written to file descriptor 2 just before the
    # process exits, past pytest's own capture
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-s", "-p", "no:cacheprovider", "-m", "not gpu"]
                       + pins, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    assert os.path.exists(os.path.join(d, "libdqgan_oracle.so")), (r.stdout + r.stderr)[-2000:]
    return r.returncode, r.stdout + r.stderr


def _oracle_source():
    with open(os.path.join(ROOT, "oracle", "dqgan_oracle.c")) as f:
        return f.read()


def test_pins_pass_under_sanitizers(tmp_path):
    rc, out = _run_pins(tmp_path, _oracle_source())
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert rc == 0, out[-4000:]


def test_sanitizers_catch_a_planted_overrun(tmp_path):
    """The instrumentation is live: the same run with the iteration's p
    buffer allocated one element short (the EF accumulate then writes past
    it) stops with an AddressSanitizer report."""
    src = _oracle_source()
    old = "float *p = (float *)malloc((size_t)d * sizeof(float));"
    assert old in src
    rc, out = _run_pins(tmp_path, src.replace(old, "float *p = (float *)malloc((size_t)(d - 1) * sizeof(float));"))
    assert rc != 0 and "AddressSanitizer" in out, out[-2000:]
