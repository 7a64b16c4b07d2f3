"""Host-side checks of the C ABI (no GPU needed): the library loads, it
exports every function include/dqgan.h declares, and descriptor validation
rejects invalid plans before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dqgan.h")).read()
    return sorted(set(re.findall(r"^\s*(?:dqgan_status|const char \*)\s*(dqgan_\w+)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def lib():
    from paper_2010_13359_amd import dqgan
    if not os.path.exists(dqgan.LIB_PATH):
        from paper_2010_13359_amd import build
        build.build()
    return dqgan.load()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) == 12, names
    for n in names:
        assert hasattr(lib, n), n
    from paper_2010_13359_amd import dqgan
    assert sorted(dqgan.EXPORTS) == names


def test_status_strings(lib):
    from paper_2010_13359_amd import dqgan
    for st in (0, -1, -2, -3, -4, -5):
        assert dqgan.status_string(st)
    assert dqgan.status_string(42) == "unknown status"


def _desc(**kw):
    from paper_2010_13359_amd import dqgan
    base = dict(d=5000, ld=5120, M=4, n_seg=2, kind=dqgan.SIGN, norm=dqgan.L1, levels=0, k=0, seed=0)
    base.update(kw)
    offs = kw.pop("offs", [0, 1000, base["d"]])
    arr = (ctypes.c_int64 * len(offs))(*offs)
    d = dqgan.Desc(base["d"], base["ld"], base["M"], base["n_seg"], arr, base["kind"], base["norm"], base["levels"],
                   0, base["k"], base["seed"])
    return d, arr


@pytest.mark.parametrize("bad", [
    dict(d=0), dict(ld=5000), dict(ld=4096), dict(M=0), dict(M=2000), dict(kind=9), dict(norm=2),
    dict(offs=[0, 1000, 4999]), dict(offs=[1, 1000, 5000]), dict(offs=[0, 1000, 1000]),
    dict(kind=1, norm=2, levels=7), dict(kind=1, norm=1, levels=15),
    dict(kind=2, norm=0, k=0), dict(kind=2, norm=0, k=5001), dict(kind=3, norm=1), dict(ld=1 << 40),
])
def test_invalid_descriptors_rejected(lib, bad):
    from paper_2010_13359_amd import dqgan
    d, arr = _desc(**bad)
    h = ctypes.c_void_p()
    assert lib.dqgan_plan_create(ctypes.byref(d), ctypes.byref(h)) == dqgan.EINVAL
    assert not h.value


def test_null_arguments(lib):
    from paper_2010_13359_amd import dqgan
    assert lib.dqgan_plan_create(None, None) == dqgan.EINVAL
    assert lib.dqgan_plan_destroy(None) == dqgan.OK
    w = dqgan.WireStruct()
    assert lib.dqgan_compress_ef(None, 0.1, 0, None, None, None, ctypes.byref(w), None) == dqgan.EINVAL
    assert lib.dqgan_step_fused(None, 0.1, 0, None, None, None, None, ctypes.byref(w), None, None) == dqgan.EINVAL
    assert lib.dqgan_omd_step(None, 0.1, None, None, None, None, None, None) == dqgan.EINVAL
    assert lib.dqgan_aggregate(None, ctypes.byref(w), None, None) == dqgan.EINVAL
    assert lib.dqgan_unpack(None, ctypes.byref(w), None, None) == dqgan.EINVAL
    assert lib.dqgan_pack(None, None, None, ctypes.byref(w), None) == dqgan.EINVAL
    assert lib.dqgan_wire_bytes(None, None, None, None, None, None) == dqgan.EINVAL
    assert lib.dqgan_step_scales(None, 0.1, None, None, ctypes.byref(w), None) == dqgan.EINVAL
    assert lib.dqgan_step_apply(None, 0.1, 0, None, None, None, None, ctypes.byref(w), None, None) == dqgan.EINVAL


def test_pure_c_demo_compiles_and_links(tmp_path):
    """include/dqgan.h is plain C: the demo builds with gcc -std=c11 -Werror
    and links against libdqgan.so, the C oracle and the HIP runtime."""
    import importlib.util
    from oracle import oracle as orc
    orc.lib()
    spec = importlib.util.spec_from_file_location("c_abi_build", os.path.join(ROOT, "tests", "c_abi", "build.py"))
    c_build = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(c_build)
    out = c_build.build(str(tmp_path / "abi_demo"))
    assert os.path.exists(out)
