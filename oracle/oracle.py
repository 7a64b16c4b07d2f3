"""ctypes front end of the C oracle (``dqgan_oracle.c``).  TEST
INFRASTRUCTURE ONLY: used by ``tests/``, the smoke check and the benchmark's
CPU-baseline leg; never by the GPU library.

Every function here marshals numpy arrays and calls one C function; the
arithmetic lives in the C file, where each function cites the part of the
paper (arXiv:2010.13359) it follows.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# DQGAN_ORACLE_DIR names another directory holding a dqgan_oracle.c to build
# and load instead (the planted-mistake test uses it for altered copies).
_DIR = os.environ.get("DQGAN_ORACLE_DIR") or _HERE
SRC = os.path.join(_DIR, "dqgan_oracle.c")
LIB = os.path.join(_DIR, "libdqgan_oracle.so")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]
# DQGAN_ORACLE_EXTRA_CFLAGS adds flags (the sanitizer test builds an
# instrumented copy with it).
EXTRA_CFLAGS = os.environ.get("DQGAN_ORACLE_EXTRA_CFLAGS", "").split()

KIND = {"sign": 0, "qsgd": 1, "topk": 2, "identity": 3, "mbit": 4}
NORM = {"l1": 1, "l2": 2, "linf": 3}


def build():
    """Compile the oracle with gcc (no FMA contraction, no fast-math)."""
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc"] + CFLAGS + EXTRA_CFLAGS + ["-o", tmp, SRC, "-lm"])
    os.replace(tmp, LIB)
    return LIB


_lib = None


class _Desc(ctypes.Structure):
    _fields_ = [
        ("d", ctypes.c_int64), ("ld", ctypes.c_int64),
        ("M", ctypes.c_int32), ("n_seg", ctypes.c_int32),
        ("seg_offsets", ctypes.POINTER(ctypes.c_int64)),
        ("kind", ctypes.c_int32), ("norm", ctypes.c_int32),
        ("levels", ctypes.c_int32), ("k", ctypes.c_int64),
        ("seed", ctypes.c_uint64),
    ]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        L = ctypes.CDLL(LIB)
        i64, i32, u32, u64, f32 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float
        P = ctypes.c_void_p
        L.oracle_philox4x32_10.argtypes = [P, P, P]
        L.oracle_uniform.argtypes = [u64, i64, i32, u32]
        L.oracle_uniform.restype = f32
        L.oracle_ef_accumulate.argtypes = [i64, f32, P, P, P]
        for name in ("oracle_scale_l1mean", "oracle_scale_l2", "oracle_scale_linf"):
            getattr(L, name).argtypes = [i64, P]
            getattr(L, name).restype = f32
        L.oracle_sign_encode.argtypes = [i64, P, f32, P, P, P]
        L.oracle_qsgd_encode.argtypes = [i64, i64, P, f32, i32, u64, i32, u32, P, P, P, P]
        L.oracle_topk.argtypes = [i64, i64, P, P, P, P, P]
        L.oracle_topk.restype = ctypes.c_int
        L.oracle_pack_bits.argtypes = [i64, i32, P, P, i64]
        L.oracle_unpack_bits.argtypes = [i64, i32, P, P]
        L.oracle_decode_segment.argtypes = [i32, i64, P, P, f32, i32, P]
        L.oracle_mbit_fields.argtypes = [i64, i32, P, P, P]
        L.oracle_mbit_split.argtypes = [i64, i32, P, P, P]
        L.oracle_aggregate.argtypes = [i32, i64, i64, P, P]
        L.oracle_omd_update.argtypes = [i64, P, P]
        L.oracle_extrapolate.argtypes = [i64, f32, P, P, P, P]
        L.oracle_step.argtypes = [ctypes.POINTER(_Desc), f32, u32, P, P, P, P, P, P, P, P, P, P, P]
        L.oracle_step.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def philox4x32_10(counter, key):
    c = np.array(counter, dtype=np.uint32)
    k = np.array(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return [int(x) for x in out]


def uniform(seed, i, m, t):
    return lib().oracle_uniform(seed, i, m, t)


def ef_accumulate(eta, g, e):
    g, e = _f32(g), _f32(e)
    p = np.empty_like(g)
    lib().oracle_ef_accumulate(g.size, np.float32(eta), _ptr(g), _ptr(e), _ptr(p))
    return p


def scale(p, norm):
    p = _f32(p)
    fn = {"l1": "oracle_scale_l1mean", "l2": "oracle_scale_l2", "linf": "oracle_scale_linf"}[norm]
    return np.float32(getattr(lib(), fn)(p.size, _ptr(p)))


def sign_encode(p, s):
    p = _f32(p)
    bits = np.empty(p.size, np.uint8)
    phat = np.empty_like(p)
    e = np.empty_like(p)
    lib().oracle_sign_encode(p.size, _ptr(p), np.float32(s), _ptr(bits), _ptr(phat), _ptr(e))
    return bits, phat, e


def qsgd_encode(p, sigma, levels, seed, m, t, i0=0):
    p = _f32(p)
    bits = np.empty(p.size, np.uint8)
    lv = np.empty(p.size, np.uint16)
    phat = np.empty_like(p)
    e = np.empty_like(p)
    lib().oracle_qsgd_encode(p.size, i0, _ptr(p), np.float32(sigma), levels, seed, m, t,
                             _ptr(bits), _ptr(lv), _ptr(phat), _ptr(e))
    return bits, lv, phat, e


def topk(p, k):
    p = _f32(p)
    idx = np.empty(k, np.uint32)
    val = np.empty(k, np.float32)
    phat = np.empty_like(p)
    e = np.empty_like(p)
    rc = lib().oracle_topk(p.size, k, _ptr(p), _ptr(idx), _ptr(val), _ptr(phat), _ptr(e))
    if rc != 0:
        raise MemoryError("oracle_topk: allocation failed")
    return idx, val, phat, e


def pack_bits(fields, b, nwords):
    f = np.ascontiguousarray(fields, dtype=np.uint16)
    words = np.empty(nwords, np.uint32)
    lib().oracle_pack_bits(f.size, b, _ptr(f), _ptr(words), nwords)
    return words


def unpack_bits(words, b, n):
    w = np.ascontiguousarray(words, dtype=np.uint32)
    f = np.empty(n, np.uint16)
    lib().oracle_unpack_bits(n, b, _ptr(w), _ptr(f))
    return f


def decode_segment(kind, signs, levels, s, nlevels=0):
    signs = np.ascontiguousarray(signs, dtype=np.uint16)
    levels = np.ascontiguousarray(levels if levels is not None else np.zeros_like(signs), dtype=np.uint16)
    out = np.empty(signs.size, np.float32)
    lib().oracle_decode_segment(KIND[kind], signs.size, _ptr(signs), _ptr(levels), np.float32(s), nlevels, _ptr(out))
    return out


def mbit_fields(bits, levels, mbits):
    """Appendix A's m-bit sign-magnitude codes of (sign bit, level)."""
    b = np.ascontiguousarray(bits, dtype=np.uint8)
    lv = np.ascontiguousarray(levels, dtype=np.uint16)
    f = np.empty(b.size, np.uint16)
    lib().oracle_mbit_fields(b.size, mbits, _ptr(b), _ptr(lv), _ptr(f))
    return f


def mbit_split(fields, mbits):
    f = np.ascontiguousarray(fields, dtype=np.uint16)
    sg = np.empty(f.size, np.uint16)
    lv = np.empty(f.size, np.uint16)
    lib().oracle_mbit_split(f.size, mbits, _ptr(f), _ptr(sg), _ptr(lv))
    return sg, lv


def aggregate(phat, d):
    phat = _f32(phat)
    M, ld = phat.shape
    q = np.empty(d, np.float32)
    lib().oracle_aggregate(M, d, ld, _ptr(phat), _ptr(q))
    return q


def omd_update(qhat, w):
    qhat, w = _f32(qhat), _f32(w).copy()
    lib().oracle_omd_update(w.size, _ptr(qhat), _ptr(w))
    return w


def extrapolate(eta, w, g, e):
    w, g, e = _f32(w), _f32(g), _f32(e)
    wx = np.empty_like(g)
    lib().oracle_extrapolate(g.size, np.float32(eta), _ptr(w), _ptr(g), _ptr(e), _ptr(wx))
    return wx


def wire_words(kind, ld, levels=0):
    """Words per row of the sign plane and of the level (code) plane."""
    if kind == "mbit":
        return 0, ld * levels // 32
    b = {255: 8, 15: 4}.get(levels, 0)
    sign = ld // 32 if kind in ("sign", "qsgd") else 0
    lev = ld * b // 32 if kind == "qsgd" else 0
    return sign, lev


def step(cfg, eta, t, G, E, W, scales_in=None):
    """One iteration of Algorithm 2 over all M rows.

    cfg: dict with d, ld, M, seg_offsets, kind ('sign'|'qsgd'|'topk'|'identity'),
    norm ('l1'|'l2'|'linf'), levels, k, seed.  G, E are [M][ld] float32, W is
    [d] (or longer) float32.  E and W are updated in place (they must be
    C-contiguous float32 arrays).  Returns a dict with E, W, WX, qhat, scale,
    sign, level, val, idx.
    """
    d, ld, M = int(cfg["d"]), int(cfg["ld"]), int(cfg["M"])
    offs = np.ascontiguousarray(cfg.get("seg_offsets", [0, d]), dtype=np.int64)
    kind = cfg["kind"]
    levels = int(cfg.get("levels", 0))
    k = int(cfg.get("k", 0))
    assert G.dtype == np.float32 and G.flags.c_contiguous and G.shape == (M, ld)
    assert E.dtype == np.float32 and E.flags.c_contiguous and E.shape == (M, ld)
    assert W.dtype == np.float32 and W.flags.c_contiguous and W.size >= d
    nseg = offs.size - 1
    sw, lw = wire_words(kind, ld, levels)
    sign = np.zeros((M, max(sw, 1)), np.uint32)
    level = np.zeros((M, max(lw, 1)), np.uint32)
    sc = np.zeros((M, nseg), np.float32)
    if kind == "topk":
        val = np.zeros((M, k), np.float32)
        idx = np.zeros((M, k), np.uint32)
    elif kind == "identity":
        val = np.zeros((M, ld), np.float32)
        idx = np.zeros(1, np.uint32)
    else:
        val = np.zeros(1, np.float32)
        idx = np.zeros(1, np.uint32)
    WX = np.zeros((M, ld), np.float32)
    q = np.zeros(d, np.float32)
    sin = None if scales_in is None else _f32(scales_in)
    desc = _Desc(d, ld, M, nseg, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), KIND[kind],
                 NORM[cfg.get("norm", "l1" if kind == "sign" else "l2")], levels, k, int(cfg.get("seed", 0)))
    rc = lib().oracle_step(ctypes.byref(desc), np.float32(eta), t, _ptr(G), _ptr(E), _ptr(W), _ptr(WX),
                           _ptr(sign), _ptr(level), _ptr(sc), _ptr(val), _ptr(idx), _ptr(q), _ptr(sin))
    if rc != 0:
        raise RuntimeError("oracle_step failed")
    return {"E": E, "W": W, "WX": WX, "qhat": q, "scale": sc, "sign": sign[:, :sw], "level": level[:, :lw],
            "val": val, "idx": idx}
