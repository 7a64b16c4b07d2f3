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
    assert len(names) == 13, names
    for n in names:
        assert hasattr(lib, n), n
    from paper_2010_13359_amd import dqgan
    assert sorted(dqgan.EXPORTS) == names


def test_status_strings(lib):
    from paper_2010_13359_amd import dqgan
    for st in (0, -1, -2, -3, -4, -5, -6):
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
    assert lib.dqgan_step_fused_noalloc(None, 0.1, 0, None, None, None, None, ctypes.byref(w), None,
                                        None) == dqgan.EINVAL


def _noalloc(lib, d, M, offs=None, kind=None, norm=None, levels=0, k=0):
    """dqgan_step_fused_noalloc with stand-in (aligned, never dereferenced)
    buffer addresses: every status checked here is decided on the host,
    before any HIP call."""
    from paper_2010_13359_amd import dqgan
    offs = offs or [0, d]
    kind = dqgan.SIGN if kind is None else kind
    norm = dqgan.L1 if norm is None else norm
    arr = (ctypes.c_int64 * len(offs))(*offs)
    D = dqgan.Desc(d, (d + 1023) // 1024 * 1024, M, len(offs) - 1, arr, kind, norm, levels, 0, k, 0)
    fake = 0x10000
    w = dqgan.WireStruct(fake, fake, fake, fake, fake)
    p = ctypes.c_void_p(fake)
    return lib.dqgan_step_fused_noalloc(ctypes.byref(D), 0.1, 1, p, p, p, p, ctypes.byref(w), None, None)


def _noalloc_bytes(d, M, offs):
    """The scratch the header states: seven tables, each rounded up to 256
    bytes (offsets, first piece per segment, tile segment, pieces, binary64
    partials, binary32 maxima, 8-byte constants per worker and segment)."""
    r = lambda n: (n + 255) // 256 * 256
    S = len(offs) - 1
    piece = 32768 if M * (d // 32768) >= 16384 else 16384
    P = sum((offs[j + 1] - offs[j] + piece - 1) // piece for j in range(S))
    ld = (d + 1023) // 1024 * 1024
    return r(8 * (S + 1)) + r(4 * (S + 1)) + r(4 * (ld // 1024)) + r(16 * P) + r(8 * M * P) + r(4 * M * P) + r(8 * M * S)


def test_noalloc_scratch_limit(lib):
    """The workload that just fits the 8 MiB scratch passes the host checks
    (without a GPU the call then fails at the device query, DQGAN_EHIP); one
    piece more is refused with DQGAN_ESCRATCH and nothing enqueued."""
    from paper_2010_13359_amd import dqgan
    limit = 8 << 20
    fits, over = 674 * 32768, 675 * 32768
    assert _noalloc_bytes(fits, 1024, [0, fits]) <= limit < _noalloc_bytes(over, 1024, [0, over])
    assert _noalloc(lib, over, 1024) == dqgan.ESCRATCH
    assert _noalloc(lib, fits, 1024) in (dqgan.OK, dqgan.EHIP)
    # 255 segments fit the launch arguments, 256 do not
    offs = list(range(0, 257 * 4, 4))
    assert _noalloc(lib, offs[-1], 2, offs) == dqgan.ESCRATCH
    offs = list(range(0, 256 * 4, 4))
    assert _noalloc(lib, offs[-1], 2, offs) in (dqgan.OK, dqgan.EHIP)


def test_noalloc_rejects_what_the_plan_rejects(lib):
    from paper_2010_13359_amd import dqgan
    assert _noalloc(lib, 6000, 4, kind=dqgan.TOPK, norm=dqgan.NORM_NONE, k=60) == dqgan.EUNSUPPORTED
    assert _noalloc(lib, 6000, 0) == dqgan.EINVAL
    assert _noalloc(lib, 6000, 4, [0, 3000, 5999]) == dqgan.EINVAL
    assert _noalloc(lib, 6000, 4, kind=dqgan.QSGD, norm=dqgan.L2, levels=7) == dqgan.EINVAL
    assert _noalloc(lib, 6000, 4, kind=dqgan.SIGN, norm=dqgan.L2) == dqgan.EINVAL


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
