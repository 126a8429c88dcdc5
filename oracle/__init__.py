"""ctypes wrapper around the plain C oracle of the RAC codec (rac_oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The product library never imports this
package, and this package imports nothing from the product.

All arrays are numpy, on the host: bf16 tensors travel as uint16 bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rac_oracle.c")
LIB_PATH = os.path.join(_HERE, "librac_oracle.so")

ORC_OK, ORC_ERR_INVALID, ORC_ERR_CAPACITY, ORC_ERR_FORMAT, ORC_ERR_NONFINITE = 0, 1, 3, 5, 6
FLAG_FIXED_STEP = 1
FLAG_XHAT_BF16 = 2
FLAG_GROUP_OUTLIERS = 4


def build(verbose: bool = False) -> str:
    """Compile the oracle with plain gcc, binary32 arithmetic, no contraction."""
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
           "-shared", "-Wall", "-Wextra", "-o", LIB_PATH + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


class _Cfg(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_int64), ("hidden", ctypes.c_int32),
                ("group_align", ctypes.c_int32), ("group_quant", ctypes.c_int32),
                ("bits", ctypes.c_int32), ("outlier_k", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


class _Layout(ctypes.Structure):
    _fields_ = [("off_coef", ctypes.c_uint64), ("off_scale", ctypes.c_uint64),
                ("off_codes", ctypes.c_uint64), ("off_outl", ctypes.c_uint64),
                ("total", ctypes.c_uint64), ("off_ooff", ctypes.c_uint64)]


class Moments(ctypes.Structure):
    _fields_ = [("n", ctypes.c_float), ("mr", ctypes.c_float), ("mx", ctypes.c_float),
                ("crr", ctypes.c_float), ("crx", ctypes.c_float)]


_lib = None


def _load(path: str):
    L = ctypes.CDLL(path)
    vp, u16p, f32p = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p
    L.orc_layout_of.argtypes = [ctypes.POINTER(_Cfg), ctypes.POINTER(_Layout)]
    L.orc_encode.argtypes = [ctypes.POINTER(_Cfg), u16p, u16p, f32p, vp, ctypes.c_size_t, vp]
    L.orc_decode.argtypes = [ctypes.POINTER(_Cfg), vp, u16p, f32p, vp]
    L.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
    L.orc_bf16_to_f32.restype = ctypes.c_float
    L.orc_f32_to_bf16.argtypes = [ctypes.c_float]
    L.orc_f32_to_bf16.restype = ctypes.c_uint16
    L.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
    L.orc_f16_to_f32.restype = ctypes.c_float
    L.orc_f16_rne_sat.argtypes = [ctypes.c_float]
    L.orc_f16_rne_sat.restype = ctypes.c_uint16
    L.orc_f16_rne.argtypes = [ctypes.c_float]
    L.orc_f16_rne.restype = ctypes.c_uint16
    L.orc_f16_wire.argtypes = [ctypes.c_uint16]
    L.orc_f16_wire.restype = ctypes.c_float
    L.orc_scale_roundup.argtypes = [ctypes.c_float, ctypes.c_int32]
    L.orc_scale_roundup.restype = ctypes.c_uint16
    L.orc_step_roundup.argtypes = [ctypes.c_float]
    L.orc_step_roundup.restype = ctypes.c_uint16
    L.orc_tsum.argtypes = [f32p, ctypes.c_int32]
    L.orc_tsum.restype = ctypes.c_float
    L.orc_fit_group.argtypes = [f32p, f32p, ctypes.c_int32, ctypes.POINTER(ctypes.c_float),
                                ctypes.POINTER(ctypes.c_float)]
    L.orc_topk_row.argtypes = [f32p, ctypes.c_int32, ctypes.c_int32, vp]
    L.orc_encode_pooled.argtypes = [ctypes.POINTER(_Cfg), u16p, u16p, ctypes.c_int64, vp, f32p, vp,
                                    ctypes.c_size_t, vp]
    L.orc_moments_row.argtypes = [f32p, f32p, ctypes.c_int32, ctypes.POINTER(Moments)]
    L.orc_moments_merge.argtypes = [ctypes.POINTER(Moments), ctypes.POINTER(Moments), ctypes.POINTER(Moments)]
    L.orc_moments_pool.argtypes = [vp, ctypes.c_int64, ctypes.POINTER(Moments)]
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC):
            build()
        _lib = _load(LIB_PATH)
    return _lib


class swapped_library:
    """Context manager: route every call to another build of the oracle source
    (used by the mutation tests, which plant mistakes in a copy)."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        self._saved = lib()
        _lib = _load(self.path)
        return _lib

    def __exit__(self, *exc):
        global _lib
        _lib = self._saved
        return False


def _cfg(tokens, hidden, group_align, group_quant, bits, outlier_k=0, flags=0) -> _Cfg:
    return _Cfg(int(tokens), int(hidden), int(group_align), int(group_quant), int(bits),
                int(outlier_k), int(flags))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def layout(**cfg) -> dict:
    out = _Layout()
    rc = lib().orc_layout_of(ctypes.byref(_cfg(**cfg)), ctypes.byref(out))
    if rc != ORC_OK:
        raise ValueError(f"oracle rejects config {cfg}: status {rc}")
    return {f: int(getattr(out, f)) for f, _ in _Layout._fields_}


def encode(x, ref=None, steps=None, *, want_xhat=True, wire_cap=None, **cfg):
    """Return (status, wire uint8[total], xhat) for bf16-pattern inputs."""
    c = _cfg(**cfg)
    lay = layout(**cfg)
    x = np.ascontiguousarray(x, dtype=np.uint16)
    ref = None if ref is None else np.ascontiguousarray(ref, dtype=np.uint16)
    steps = None if steps is None else np.ascontiguousarray(steps, dtype=np.float32)
    cap = lay["total"] if wire_cap is None else int(wire_cap)
    wire = np.zeros(max(cap, 1), dtype=np.uint8)
    xhat = None
    if want_xhat:
        dt = np.uint16 if (c.flags & FLAG_XHAT_BF16) else np.float32
        xhat = np.zeros((c.tokens, c.hidden), dtype=dt)
    rc = lib().orc_encode(ctypes.byref(c), _ptr(x), _ptr(ref), _ptr(steps), _ptr(wire),
                          cap, _ptr(xhat))
    return rc, wire[:lay["total"]], xhat


def decode(wire, ref=None, steps=None, **cfg):
    """Return (status, xhat) reconstructed from a wire and the receiver's ref."""
    c = _cfg(**cfg)
    wire = np.ascontiguousarray(wire, dtype=np.uint8)
    ref = None if ref is None else np.ascontiguousarray(ref, dtype=np.uint16)
    steps = None if steps is None else np.ascontiguousarray(steps, dtype=np.float32)
    dt = np.uint16 if (c.flags & FLAG_XHAT_BF16) else np.float32
    xhat = np.zeros((c.tokens, c.hidden), dtype=dt)
    rc = lib().orc_decode(ctypes.byref(c), _ptr(wire), _ptr(ref), _ptr(steps), _ptr(xhat))
    return rc, xhat


# ---- single pieces, for pinning ------------------------------------------

def bf16_to_f32(h: int) -> float:
    return float(lib().orc_bf16_to_f32(int(h)))


def f32_to_bf16(v: float) -> int:
    return int(lib().orc_f32_to_bf16(float(v)))


def f16_to_f32(h: int) -> float:
    return float(lib().orc_f16_to_f32(int(h)))


def f16_rne_sat(v: float) -> int:
    return int(lib().orc_f16_rne_sat(float(v)))


def f16_rne(v: float) -> int:
    return int(lib().orc_f16_rne(float(v)))


def f16_wire(h: int) -> float:
    return float(lib().orc_f16_wire(int(h)))


def scale_roundup(m: float, qmax: int) -> int:
    return int(lib().orc_scale_roundup(float(m), int(qmax)))


def step_roundup(step: float) -> int:
    return int(lib().orc_step_roundup(float(step)))


def tsum(v) -> float:
    v = np.ascontiguousarray(v, dtype=np.float32)
    return float(lib().orc_tsum(_ptr(v), int(v.size)))


def fit_group(r, x):
    r = np.ascontiguousarray(r, dtype=np.float32)
    x = np.ascontiguousarray(x, dtype=np.float32)
    a, b = ctypes.c_float(), ctypes.c_float()
    lib().orc_fit_group(_ptr(r), _ptr(x), int(r.size), ctypes.byref(a), ctypes.byref(b))
    return float(a.value), float(b.value)


def topk_row(e, k: int):
    e = np.ascontiguousarray(e, dtype=np.float32)
    idx = np.zeros(max(int(k), 1), dtype=np.uint16)
    lib().orc_topk_row(_ptr(e), int(e.size), int(k), _ptr(idx))
    return idx[:k].copy()


def encode_pooled(x, ref, seg_start, steps=None, *, want_xhat=True, **cfg):
    """Encode with the fit pooled over segments (seg_start: [S+1] row starts).
    Returns (status, wire, xhat)."""
    c = _cfg(**cfg)
    lay = layout(**cfg)
    x = np.ascontiguousarray(x, dtype=np.uint16)
    ref = None if ref is None else np.ascontiguousarray(ref, dtype=np.uint16)
    steps = None if steps is None else np.ascontiguousarray(steps, dtype=np.float32)
    seg = np.ascontiguousarray(seg_start, dtype=np.int32)
    wire = np.zeros(max(lay["total"], 1), dtype=np.uint8)
    xhat = None
    if want_xhat:
        dt = np.uint16 if (c.flags & FLAG_XHAT_BF16) else np.float32
        xhat = np.zeros((c.tokens, c.hidden), dtype=dt)
    rc = lib().orc_encode_pooled(ctypes.byref(c), _ptr(x), _ptr(ref), seg.size - 1, _ptr(seg), _ptr(steps),
                                 _ptr(wire), lay["total"], _ptr(xhat))
    return rc, wire[:lay["total"]], xhat


def moments_row(r, x) -> Moments:
    r = np.ascontiguousarray(r, dtype=np.float32)
    x = np.ascontiguousarray(x, dtype=np.float32)
    m = Moments()
    lib().orc_moments_row(_ptr(r), _ptr(x), int(r.size), ctypes.byref(m))
    return m


def moments_pool(rows) -> Moments:
    arr = (Moments * len(rows))(*rows)
    m = Moments()
    lib().orc_moments_pool(ctypes.cast(arr, ctypes.c_void_p), len(rows), ctypes.byref(m))
    return m
