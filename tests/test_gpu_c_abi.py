"""The library from plain C (tests/c_abi/abi_demo.c, built by
__graft_entry__.build()): one fused iteration through include/dqgan.h with
device memory from the HIP runtime's C API, every output identical to the C
oracle's (teacher-forced with the GPU's scales), scales within 1e-5."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.timeout(120)
def test_pure_c_iteration_matches_oracle():
    exe = os.path.join(HERE, "c_abi", "abi_demo")
    assert os.path.exists(exe), "tests/c_abi/abi_demo is not built: run __graft_entry__.build()"
    print("pure-C iteration", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=100)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c abi demo ok" in r.stdout
