"""Python binding of the DQGAN C ABI (``include/dqgan.h``).

Argument marshalling only: torch tensors supply device memory and the
stream; every step of the computation runs in the HIP library.  The library
must have been built (``paper_2010_13359_amd/build.py``); importing this
module on a machine without it raises, there is no fallback.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdqgan.so")

SIGN, QSGD, TOPK, IDENTITY, MBIT = 0, 1, 2, 3, 4
NORM_NONE, L1, L2, LINF = 0, 1, 2, 3
KINDS = {"sign": SIGN, "qsgd": QSGD, "topk": TOPK, "identity": IDENTITY, "mbit": MBIT}
NORMS = {"none": NORM_NONE, "l1": L1, "l2": L2, "linf": LINF}

OK, EINVAL, EALIGN, ENOMEM, EHIP, EUNSUPPORTED, ESCRATCH = 0, -1, -2, -3, -4, -5, -6

EXPORTS = ("dqgan_plan_create", "dqgan_plan_destroy", "dqgan_wire_bytes", "dqgan_compress_ef", "dqgan_pack",
           "dqgan_unpack", "dqgan_aggregate", "dqgan_omd_step", "dqgan_step_fused", "dqgan_step_scales",
           "dqgan_step_apply", "dqgan_step_fused_noalloc", "dqgan_status_string")


class DqganError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__("%s: %s (%d)" % (fn, status_string(status), status))


class Desc(ctypes.Structure):
    _fields_ = [
        ("d", ctypes.c_int64), ("ld", ctypes.c_int64),
        ("M", ctypes.c_int32), ("n_seg", ctypes.c_int32),
        ("seg_offsets", ctypes.POINTER(ctypes.c_int64)),
        ("kind", ctypes.c_int32), ("norm", ctypes.c_int32),
        ("levels", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("k", ctypes.c_int64), ("seed", ctypes.c_uint64),
    ]


class WireStruct(ctypes.Structure):
    _fields_ = [("sign", ctypes.c_void_p), ("level", ctypes.c_void_p), ("scale", ctypes.c_void_p),
                ("val", ctypes.c_void_p), ("idx", ctypes.c_void_p)]


_lib = None


def load():
    """Load the built library (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libdqgan.so is not built: run paper_2010_13359_amd/build.py (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, u32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_float
    L.dqgan_plan_create.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(ctypes.c_void_p)]
    L.dqgan_plan_destroy.argtypes = [P]
    L.dqgan_wire_bytes.argtypes = [P] + [ctypes.POINTER(ctypes.c_size_t)] * 5
    L.dqgan_compress_ef.argtypes = [P, f32, u32, P, P, P, ctypes.POINTER(WireStruct), P]
    L.dqgan_pack.argtypes = [P, P, P, ctypes.POINTER(WireStruct), P]
    L.dqgan_unpack.argtypes = [P, ctypes.POINTER(WireStruct), P, P]
    L.dqgan_aggregate.argtypes = [P, ctypes.POINTER(WireStruct), P, P]
    L.dqgan_omd_step.argtypes = [P, f32, P, P, P, P, P, P]
    L.dqgan_step_fused.argtypes = [P, f32, u32, P, P, P, P, ctypes.POINTER(WireStruct), P, P]
    L.dqgan_step_scales.argtypes = [P, f32, P, P, ctypes.POINTER(WireStruct), P]
    L.dqgan_step_apply.argtypes = [P, f32, u32, P, P, P, P, ctypes.POINTER(WireStruct), P, P]
    L.dqgan_step_fused_noalloc.argtypes = [ctypes.POINTER(Desc), f32, u32, P, P, P, P, ctypes.POINTER(WireStruct),
                                           P, P]
    L.dqgan_status_string.argtypes = [i32]
    L.dqgan_status_string.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name != "dqgan_status_string":
            getattr(L, name).restype = i32
    _lib = L
    return L


def status_string(status):
    return load().dqgan_status_string(status).decode()


def _check(fn, status):
    if status != OK:
        raise DqganError(fn, status)


F32 = (torch.float32,)
U32 = (torch.int32, torch.uint32)    # bit patterns of uint32 words
U16 = (torch.int16, torch.uint16)    # per-element codes of dqgan_pack


def _ptr(t, name="tensor", nbytes=0, dtypes=None, device=None):
    """Device pointer of `t` after the checks the C ABI cannot make: a
    contiguous device tensor of the expected dtype, on the plan's device,
    holding at least `nbytes` bytes.  None passes as NULL."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s: expected a torch.Tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s: tensor must be in device memory" % name)
    if not t.is_contiguous():
        raise ValueError("%s: tensor must be contiguous" % name)
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError("%s: dtype %s, expected %s" % (name, t.dtype, " or ".join(str(d) for d in dtypes)))
    if device is not None and t.device.index != device:
        raise ValueError("%s: on cuda:%s, the plan is on cuda:%d" % (name, t.device.index, device))
    if t.numel() * t.element_size() < nbytes:
        raise ValueError("%s: %d bytes, the plan needs %d" % (name, t.numel() * t.element_size(), nbytes))
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class Plan:
    """Owns a dqgan_plan (created on the current device)."""

    def __init__(self, d, M, kind, seg_offsets=None, norm=None, levels=0, k=0, seed=0, ld=None):
        self.d, self.M = int(d), int(M)
        self.ld = int(ld) if ld else (self.d + 1023) // 1024 * 1024
        self.kind = KINDS[kind] if isinstance(kind, str) else int(kind)
        if norm is None:
            norm = {SIGN: "l1", QSGD: "l2", MBIT: "linf"}.get(self.kind, "none")
        self.norm = NORMS[norm] if isinstance(norm, str) else int(norm)
        self.levels, self.k, self.seed = int(levels), int(k), int(seed)
        offs = list(seg_offsets) if seg_offsets is not None else [0, self.d]
        self.n_seg = len(offs) - 1
        self._offs = (ctypes.c_int64 * len(offs))(*offs)
        self.desc = Desc(self.d, self.ld, self.M, self.n_seg, self._offs, self.kind, self.norm, self.levels, 0,
                         self.k, self.seed)
        h = ctypes.c_void_p()
        _check("dqgan_plan_create", load().dqgan_plan_create(ctypes.byref(self.desc), ctypes.byref(h)))
        self.handle = h
        self.device = torch.cuda.current_device()
        self._wire_bytes = self.wire_bytes()

    # byte sizes of the arguments (include/dqgan.h)
    def _mat(self, t, name):
        return _ptr(t, name, 4 * self.M * self.ld, F32, self.device)

    def _vec(self, t, name):
        return _ptr(t, name, 4 * self.ld, F32, self.device)

    def _scales(self, t, name):
        return _ptr(t, name, 4 * self.M * self.n_seg, F32, self.device)

    @classmethod
    def from_workload(cls, w):
        return cls(w.d, w.M, w.kind, w.seg_offsets, w.norm if w.kind in ("sign", "qsgd", "mbit") else "none",
                   w.levels, w.k, w.quant_seed, w.ld)

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            load().dqgan_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def wire_bytes(self):
        out = [ctypes.c_size_t() for _ in range(5)]
        _check("dqgan_wire_bytes", load().dqgan_wire_bytes(self.handle, *[ctypes.byref(x) for x in out]))
        return tuple(x.value for x in out)

    def new_wire(self, device="cuda"):
        sb, lb, cb, vb, ib = self.wire_bytes()
        mk = lambda n, dt, per: torch.zeros(n // per, dtype=dt, device=device) if n else None
        return Wire(mk(sb, torch.int32, 4), mk(lb, torch.int32, 4), mk(cb, torch.float32, 4),
                    mk(vb, torch.float32, 4), mk(ib, torch.int32, 4))


class Wire:
    """The message planes (device tensors).  sign/level/idx hold uint32 bit
    patterns in int32 tensors."""

    def __init__(self, sign=None, level=None, scale=None, val=None, idx=None):
        self.sign, self.level, self.scale, self.val, self.idx = sign, level, scale, val, idx

    def struct(self, plan):
        """The dqgan_wire of these planes; each plane the plan's compressor
        uses must be present and large enough."""
        planes = (("sign", self.sign, U32), ("level", self.level, U32), ("scale", self.scale, F32),
                  ("val", self.val, F32), ("idx", self.idx, U32))
        ptrs = []
        for (name, t, dt), need in zip(planes, plan._wire_bytes):
            if need and t is None:
                raise ValueError("wire.%s: the plan's compressor needs this plane (%d bytes)" % (name, need))
            p = _ptr(t, "wire." + name, need, dt, plan.device)
            ptrs.append(None if p is None else p.value)
        return WireStruct(*ptrs)


def compress_ef(plan, eta, t, G, E, scales_in, wire, stream=None):
    ws = wire.struct(plan)
    _check("dqgan_compress_ef", load().dqgan_compress_ef(plan.handle, ctypes.c_float(eta), t, plan._mat(G, "G"),
                                                         plan._mat(E, "E"), plan._scales(scales_in, "scales_in"),
                                                         ctypes.byref(ws), _stream(stream)))


def pack(plan, codes, scales, wire, stream=None):
    ws = wire.struct(plan)
    _check("dqgan_pack", load().dqgan_pack(plan.handle, _ptr(codes, "codes", 2 * plan.M * plan.ld, U16, plan.device),
                                           plan._scales(scales, "scales"), ctypes.byref(ws), _stream(stream)))


def unpack(plan, wire, Phat, stream=None):
    ws = wire.struct(plan)
    _check("dqgan_unpack", load().dqgan_unpack(plan.handle, ctypes.byref(ws), plan._mat(Phat, "Phat"),
                                               _stream(stream)))


def aggregate(plan, wire, Qhat, stream=None):
    ws = wire.struct(plan)
    _check("dqgan_aggregate", load().dqgan_aggregate(plan.handle, ctypes.byref(ws), plan._vec(Qhat, "Qhat"),
                                                     _stream(stream)))


def omd_step(plan, eta, Qhat, W, G, E, WX, stream=None):
    _check("dqgan_omd_step", load().dqgan_omd_step(plan.handle, ctypes.c_float(eta), plan._vec(Qhat, "Qhat"),
                                                   plan._vec(W, "W"), plan._mat(G, "G"), plan._mat(E, "E"),
                                                   plan._mat(WX, "WX"), _stream(stream)))


def step_fused(plan, eta, t, G, E, W, WX, wire, Qhat=None, stream=None):
    ws = wire.struct(plan)
    _check("dqgan_step_fused", load().dqgan_step_fused(plan.handle, ctypes.c_float(eta), t, plan._mat(G, "G"),
                                                       plan._mat(E, "E"), plan._vec(W, "W"), plan._mat(WX, "WX"),
                                                       ctypes.byref(ws), plan._vec(Qhat, "Qhat"), _stream(stream)))


def step_scales(plan, eta, G, E, wire, stream=None):
    ws = wire.struct(plan)
    _check("dqgan_step_scales", load().dqgan_step_scales(plan.handle, ctypes.c_float(eta), plan._mat(G, "G"),
                                                         plan._mat(E, "E"), ctypes.byref(ws), _stream(stream)))


def step_apply(plan, eta, t, G, E, W, WX, wire, Qhat=None, stream=None):
    ws = wire.struct(plan)
    _check("dqgan_step_apply", load().dqgan_step_apply(plan.handle, ctypes.c_float(eta), t, plan._mat(G, "G"),
                                                       plan._mat(E, "E"), plan._vec(W, "W"), plan._mat(WX, "WX"),
                                                       ctypes.byref(ws), plan._vec(Qhat, "Qhat"), _stream(stream)))


def step_fused_noalloc(plan, eta, t, G, E, W, WX, wire, Qhat=None, stream=None):
    """dqgan_step_fused_noalloc with the descriptor of `plan` (the plan only
    supplies the descriptor and the byte sizes the arguments are checked
    against; the call itself uses neither the plan nor any allocation)."""
    ws = wire.struct(plan)
    _check("dqgan_step_fused_noalloc",
           load().dqgan_step_fused_noalloc(ctypes.byref(plan.desc), ctypes.c_float(eta), t, plan._mat(G, "G"),
                                           plan._mat(E, "E"), plan._vec(W, "W"), plan._mat(WX, "WX"),
                                           ctypes.byref(ws), plan._vec(Qhat, "Qhat"), _stream(stream)))
