"""MI355X (gfx950) RAC aligned residual codec: Python binding of librac.so.

This module only marshals arguments to the C ABI declared in include/rac.h
(same names, same semantics); every step of the codec runs in the HIP
kernels of csrc/rac.hip.  PyTorch supplies device memory and the stream.

    cfg = RacConfig(tokens=T, hidden=d, group_align=128, group_quant=128,
                    bits=4, outlier_k=8)
    wire = torch.empty(rac_wire_size(cfg), dtype=torch.uint8, device="cuda")
    rac_encode(cfg, x, ref, None, wire, xhat)          # x, ref: bf16 [T, d]
    rac_decode(cfg, wire, ref, None, xhat_receiver)

There is no fallback: if librac.so is missing the calls raise.
"""
from __future__ import annotations

import ctypes
import functools
import os
from dataclasses import dataclass

__all__ = [
    "RacConfig", "RacError", "RAC_FLAG_FIXED_STEP", "RAC_FLAG_XHAT_BF16", "RAC_FLAG_GROUP_OUTLIERS",
    "STATUS",
    "library", "library_path", "rac_wire_layout", "rac_wire_size", "rac_parse_header",
    "rac_encode", "rac_reconstruct", "rac_decode", "rac_encode_gather", "rac_decode_gather",
    "rac_status_string", "SpanIndex", "rac_encode_pooled", "rac_saturation_summary",
    "rac_recon_error_workspace", "rac_recon_error", "rac_calibrate_workspace", "rac_calibrate",
    "PredictorConfig", "rac_predictor_layout", "rac_predictor_cache_bytes", "rac_predictor_workspace_bytes",
    "predictor_pack", "rac_predictor_step",
]

RAC_FLAG_FIXED_STEP = 1
RAC_FLAG_XHAT_BF16 = 2
RAC_FLAG_GROUP_OUTLIERS = 4
RAC_FLAG_LAUNCH_STRIDED = 8    # launch hints: change no result, only the launch shape
RAC_FLAG_LAUNCH_PER_ROW = 16
STATUS = {0: "RAC_OK", 1: "RAC_ERR_INVALID", 2: "RAC_ERR_ALIGN", 3: "RAC_ERR_CAPACITY",
          4: "RAC_ERR_HIP", 5: "RAC_ERR_FORMAT", 6: "RAC_ERR_UNSUPPORTED", 7: "RAC_ERR_NOMEM"}

_HERE = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(_HERE, "lib", "librac.so")


class RacError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {STATUS.get(status, status)} ({rac_status_string(status)})")
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_int64), ("hidden", ctypes.c_int32),
                ("group_align", ctypes.c_int32), ("group_quant", ctypes.c_int32),
                ("bits", ctypes.c_int32), ("outlier_k", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


class _Layout(ctypes.Structure):
    _fields_ = [("off_coef", ctypes.c_uint64), ("off_scale", ctypes.c_uint64),
                ("off_codes", ctypes.c_uint64), ("off_outl", ctypes.c_uint64),
                ("total", ctypes.c_uint64), ("off_ooff", ctypes.c_uint64)]


class _Candidate(ctypes.Structure):
    _fields_ = [("cfg", _Config), ("wire_bytes", ctypes.c_uint64), ("sq_err", ctypes.c_double),
                ("sq_x", ctypes.c_double), ("max_abs", ctypes.c_double), ("nmse", ctypes.c_double),
                ("feasible", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class _PredConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("hidden", "model", "heads", "ffn", "window", "max_batch")]


class _PredOffsets(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in ("w_in", "g1", "w_qkv", "w_o", "g2", "w_gu", "w_down", "g3",
                                               "w_out", "total")]


@dataclass(frozen=True)
class PredictorConfig:
    hidden: int
    model: int
    heads: int
    ffn: int
    window: int
    max_batch: int

    def _c(self) -> _PredConfig:
        return _PredConfig(self.hidden, self.model, self.heads, self.ffn, self.window, self.max_batch)


@dataclass(frozen=True)
class RacConfig:
    tokens: int
    hidden: int
    group_align: int
    group_quant: int
    bits: int
    outlier_k: int = 0
    flags: int = 0

    def _c(self) -> _Config:
        return _cfg_struct(self)


@functools.lru_cache(maxsize=512)
def _cfg_struct(cfg: "RacConfig") -> _Config:
    # (the library reads the struct during the call only, so one instance per
    # configuration can be passed to every call)
    return _Config(cfg.tokens, cfg.hidden, cfg.group_align, cfg.group_quant, cfg.bits,
                   cfg.outlier_k, cfg.flags)


_lib = None


def library():
    """Load librac.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -m paper_2608_04991_amd.build`")
        L = ctypes.CDLL(path)
        cp = ctypes.POINTER(_Config)
        vp = ctypes.c_void_p
        L.rac_wire_layout.argtypes = [cp, ctypes.POINTER(_Layout)]
        L.rac_wire_layout.restype = ctypes.c_int
        L.rac_wire_size.argtypes = [cp]
        L.rac_wire_size.restype = ctypes.c_size_t
        L.rac_parse_header.argtypes = [vp, ctypes.c_size_t, cp, ctypes.POINTER(ctypes.c_int)]
        L.rac_parse_header.restype = ctypes.c_int
        L.rac_encode.argtypes = [cp, vp, vp, vp, vp, ctypes.c_size_t, vp, vp]
        L.rac_encode.restype = ctypes.c_int
        L.rac_reconstruct.argtypes = [cp, vp, vp, vp, vp, vp]
        L.rac_reconstruct.restype = ctypes.c_int
        L.rac_decode.argtypes = [cp, vp, vp, vp, vp, vp]
        L.rac_decode.restype = ctypes.c_int
        L.rac_encode_gather.argtypes = [cp, vp, vp, ctypes.c_int64, vp, vp, vp, ctypes.c_size_t, vp, vp]
        L.rac_encode_gather.restype = ctypes.c_int
        L.rac_decode_gather.argtypes = [cp, vp, vp, ctypes.c_int64, vp, vp, vp, vp]
        L.rac_decode_gather.restype = ctypes.c_int
        L.rac_encode_pooled.argtypes = [cp, vp, vp, ctypes.c_int64, vp, vp, vp, ctypes.c_size_t, vp, vp]
        L.rac_encode_pooled.restype = ctypes.c_int
        L.rac_span_index_create.argtypes = [ctypes.c_int32]
        L.rac_span_index_create.restype = vp
        L.rac_span_index_destroy.argtypes = [vp]
        L.rac_span_index_destroy.restype = None
        L.rac_span_index_add.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int64]
        L.rac_span_index_add.restype = ctypes.c_int
        L.rac_span_select.argtypes = [vp, vp, ctypes.c_int64, vp, ctypes.POINTER(ctypes.c_int64)]
        L.rac_span_select.restype = ctypes.c_int
        L.rac_saturation_summary.argtypes = [cp, vp, ctypes.c_size_t, ctypes.POINTER(ctypes.c_int64),
                                             ctypes.POINTER(ctypes.c_uint32)]
        L.rac_saturation_summary.restype = ctypes.c_int
        L.rac_recon_error_workspace.argtypes = [ctypes.c_int64]
        L.rac_recon_error_workspace.restype = ctypes.c_size_t
        L.rac_recon_error.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, vp, vp, vp, vp,
                                      ctypes.c_size_t, vp]
        L.rac_recon_error.restype = ctypes.c_int
        candp = ctypes.POINTER(_Candidate)
        L.rac_calibrate_workspace.argtypes = [candp, ctypes.c_int32]
        L.rac_calibrate_workspace.restype = ctypes.c_size_t
        L.rac_calibrate.argtypes = [vp, vp, candp, ctypes.c_int32, ctypes.c_double, vp, ctypes.c_size_t,
                                    ctypes.POINTER(ctypes.c_int32), vp]
        L.rac_calibrate.restype = ctypes.c_int
        pcp = ctypes.POINTER(_PredConfig)
        L.rac_predictor_layout.argtypes = [pcp, ctypes.POINTER(_PredOffsets)]
        L.rac_predictor_layout.restype = ctypes.c_int
        L.rac_predictor_cache_bytes.argtypes = [pcp]
        L.rac_predictor_cache_bytes.restype = ctypes.c_size_t
        L.rac_predictor_workspace_bytes.argtypes = [pcp]
        L.rac_predictor_workspace_bytes.restype = ctypes.c_size_t
        L.rac_predictor_step.argtypes = [pcp, vp, vp, vp, ctypes.c_int32, vp, vp, vp, ctypes.c_size_t, vp]
        L.rac_predictor_step.restype = ctypes.c_int
        L.rac_status_string.argtypes = [ctypes.c_int]
        L.rac_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _ptr(t):
    """Device address of a tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _dev(t, what: str, elem_bytes, count: int):
    """Address of a device tensor argument after checking, before anything is
    enqueued, that the kernels can read or write `count` elements of
    `elem_bytes` bytes there: a GPU tensor,
    contiguous, of that element size, holding at least `count` elements.
    None and raw integer addresses pass through unchecked (the C ABI checks
    what it can)."""
    if t is None or isinstance(t, int):
        return t
    if not (getattr(t, "is_cuda", False) and t.is_contiguous()):
        raise ValueError(f"{what}: expected a contiguous GPU tensor")
    es = t.element_size()
    if es != elem_bytes:
        raise ValueError(f"{what}: expected {elem_bytes}-byte elements, got {es}")
    if t.numel() < count:
        raise ValueError(f"{what}: holds {t.numel()} elements, needs {count}")
    return t.data_ptr()


def _xhat_bytes(cfg) -> int:
    return 2 if cfg.flags & RAC_FLAG_XHAT_BF16 else 4


def _nsteps(cfg) -> int:
    return cfg.hidden // cfg.group_quant if cfg.flags & RAC_FLAG_FIXED_STEP else 0


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, what: str):
    if status != 0:
        raise RacError(status, what)


def rac_status_string(status: int) -> str:
    return library().rac_status_string(int(status)).decode()


def rac_wire_layout(cfg: RacConfig) -> dict:
    out = _Layout()
    _check(library().rac_wire_layout(ctypes.byref(cfg._c()), ctypes.byref(out)), "rac_wire_layout")
    return {f: int(getattr(out, f)) for f, _ in _Layout._fields_}


def rac_wire_size(cfg: RacConfig) -> int:
    return _wire_size(cfg, library())


@functools.lru_cache(maxsize=512)
def _wire_size(cfg: RacConfig, lib) -> int:
    return int(lib.rac_wire_size(ctypes.byref(cfg._c())))


def rac_parse_header(header: bytes):
    """Parse a host copy of a wire header; returns (RacConfig, zero_ref)."""
    buf = ctypes.create_string_buffer(bytes(header), len(header))
    c = _Config()
    zr = ctypes.c_int(0)
    _check(library().rac_parse_header(buf, len(header), ctypes.byref(c), ctypes.byref(zr)),
           "rac_parse_header")
    return RacConfig(c.tokens, c.hidden, c.group_align, c.group_quant, c.bits, c.outlier_k,
                     c.flags), bool(zr.value)


def rac_saturation_summary(cfg: RacConfig, wire) -> tuple[int, int]:
    """(token rows with a saturated fp16 field, OR of 1 coefficient / 2 scale
    / 4 outlier value) of a wire in host memory (bytes-like or a numpy uint8
    array of at least rac_wire_size(cfg) bytes)."""
    import numpy as np
    a = np.ascontiguousarray(np.frombuffer(bytes(wire), dtype=np.uint8) if isinstance(wire, (bytes, bytearray))
                             else np.asarray(wire, dtype=np.uint8))
    rows, bits = ctypes.c_int64(0), ctypes.c_uint32(0)
    _check(library().rac_saturation_summary(ctypes.byref(cfg._c()), a.ctypes.data, a.size, ctypes.byref(rows),
                                            ctypes.byref(bits)), "rac_saturation_summary")
    return int(rows.value), int(bits.value)


def rac_encode(cfg: RacConfig, x, ref, fixed_steps, wire, xhat=None, stream=None,
               wire_cap: int | None = None) -> None:
    """Encode x against ref into wire (+ fused sender reconstruction)."""
    cap = wire_cap if wire_cap is not None else (_nbytes(wire) if not isinstance(wire, int) else 0)
    n = cfg.tokens * cfg.hidden
    _check(library().rac_encode(ctypes.byref(cfg._c()), _dev(x, "x", 2, n), _dev(ref, "ref", 2, n),
                                _dev(fixed_steps, "fixed_steps", 4, _nsteps(cfg)), _dev(wire, "wire", 1, 0),
                                cap, _dev(xhat, "xhat", _xhat_bytes(cfg), n), _stream(stream)), "rac_encode")


def rac_reconstruct(cfg: RacConfig, wire, ref, fixed_steps, xhat, stream=None) -> None:
    """Sender-side reconstruction from the sender's own wire."""
    n = cfg.tokens * cfg.hidden
    _check(library().rac_reconstruct(ctypes.byref(cfg._c()), _dev(wire, "wire", 1, rac_wire_size(cfg)),
                                     _dev(ref, "ref", 2, n), _dev(fixed_steps, "fixed_steps", 4, _nsteps(cfg)),
                                     _dev(xhat, "xhat", _xhat_bytes(cfg), n), _stream(stream)),
           "rac_reconstruct")


def rac_decode(cfg: RacConfig, wire, ref, fixed_steps, xhat, stream=None) -> None:
    """Receiver-side reconstruction from a wire and the receiver's reference."""
    n = cfg.tokens * cfg.hidden
    _check(library().rac_decode(ctypes.byref(cfg._c()), _dev(wire, "wire", 1, rac_wire_size(cfg)),
                                _dev(ref, "ref", 2, n), _dev(fixed_steps, "fixed_steps", 4, _nsteps(cfg)),
                                _dev(xhat, "xhat", _xhat_bytes(cfg), n), _stream(stream)), "rac_decode")


def _rows(store, store_rows):
    if store_rows is not None:
        return int(store_rows)
    return 0 if store is None or isinstance(store, int) else int(store.shape[0])


def rac_encode_gather(cfg: RacConfig, x, store, ref_rows, fixed_steps, wire, xhat=None, stream=None,
                      store_rows: int | None = None, wire_cap: int | None = None) -> None:
    """Encode x against the store rows that ref_rows names (int32 [T]; an index
    outside the store means a zero reference row)."""
    cap = wire_cap if wire_cap is not None else (_nbytes(wire) if not isinstance(wire, int) else 0)
    n, sr = cfg.tokens * cfg.hidden, _rows(store, store_rows)
    _check(library().rac_encode_gather(ctypes.byref(cfg._c()), _dev(x, "x", 2, n),
                                       _dev(store, "store", 2, sr * cfg.hidden), sr,
                                       _dev(ref_rows, "ref_rows", 4, cfg.tokens),
                                       _dev(fixed_steps, "fixed_steps", 4, _nsteps(cfg)), _dev(wire, "wire", 1, 0),
                                       cap, _dev(xhat, "xhat", _xhat_bytes(cfg), n), _stream(stream)),
           "rac_encode_gather")


def rac_decode_gather(cfg: RacConfig, wire, store, ref_rows, fixed_steps, xhat, stream=None,
                      store_rows: int | None = None) -> None:
    """Receiver-side reconstruction with the reference gathered from a store."""
    n, sr = cfg.tokens * cfg.hidden, _rows(store, store_rows)
    _check(library().rac_decode_gather(ctypes.byref(cfg._c()), _dev(wire, "wire", 1, rac_wire_size(cfg)),
                                       _dev(store, "store", 2, sr * cfg.hidden), sr,
                                       _dev(ref_rows, "ref_rows", 4, cfg.tokens),
                                       _dev(fixed_steps, "fixed_steps", 4, _nsteps(cfg)),
                                       _dev(xhat, "xhat", _xhat_bytes(cfg), n), _stream(stream)),
           "rac_decode_gather")


class SpanIndex:
    """Host-side index of earlier requests for the prefill-uplink reference
    selection (rac_span_index_* / rac_span_select); tokens are int32 arrays."""

    def __init__(self, window: int):
        import numpy as np
        self._np = np
        self._h = library().rac_span_index_create(int(window))
        if not self._h:
            raise RacError(1, "rac_span_index_create")

    def add(self, tokens, store_row0: int) -> None:
        t = self._np.ascontiguousarray(tokens, dtype=self._np.int32)
        _check(library().rac_span_index_add(self._h, t.ctypes.data, t.size, int(store_row0)), "rac_span_index_add")

    def select(self, tokens):
        """Returns (ref_rows int32[n], covered positions)."""
        t = self._np.ascontiguousarray(tokens, dtype=self._np.int32)
        out = self._np.empty(t.size, dtype=self._np.int32)
        cov = ctypes.c_int64(0)
        _check(library().rac_span_select(self._h, t.ctypes.data, t.size, out.ctypes.data, ctypes.byref(cov)),
               "rac_span_select")
        return out, int(cov.value)

    def close(self) -> None:
        if self._h:
            library().rac_span_index_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def rac_encode_pooled(cfg: RacConfig, x, ref, seg_start, fixed_steps, wire, xhat=None, stream=None,
                      segments: int | None = None, wire_cap: int | None = None) -> None:
    """Encode with the fit pooled over segments of rows (seg_start: device
    int32 [segments + 1] row starts)."""
    cap = wire_cap if wire_cap is not None else (_nbytes(wire) if not isinstance(wire, int) else 0)
    nseg = int(segments) if segments is not None else int(seg_start.numel()) - 1
    n = cfg.tokens * cfg.hidden
    _check(library().rac_encode_pooled(ctypes.byref(cfg._c()), _dev(x, "x", 2, n), _dev(ref, "ref", 2, n), nseg,
                                       _dev(seg_start, "seg_start", 4, nseg + 1),
                                       _dev(fixed_steps, "fixed_steps", 4, _nsteps(cfg)), _dev(wire, "wire", 1, 0),
                                       cap, _dev(xhat, "xhat", _xhat_bytes(cfg), n), _stream(stream)),
           "rac_encode_pooled")


def rac_recon_error_workspace(tokens: int) -> int:
    return int(library().rac_recon_error_workspace(int(tokens)))


def rac_recon_error(tokens: int, hidden: int, x, xhat, stats, workspace, flags: int = 0, stream=None,
                    workspace_bytes: int | None = None) -> None:
    """Reconstruction error of xhat against x into stats (device float64[3]:
    sum of squared errors, sum of x^2, max |x - xhat|)."""
    n = int(tokens) * int(hidden)
    cap = workspace_bytes if workspace_bytes is not None else (
        _nbytes(workspace) if workspace is not None and not isinstance(workspace, int) else 0)
    _check(library().rac_recon_error(int(tokens), int(hidden), int(flags), _dev(x, "x", 2, n),
                                     _dev(xhat, "xhat", 2 if flags & RAC_FLAG_XHAT_BF16 else 4, n),
                                     _dev(stats, "stats", 8, 3), _dev(workspace, "workspace", 1, 0), cap,
                                     _stream(stream)), "rac_recon_error")


def _candidates(configs):
    arr = (_Candidate * len(configs))()
    for i, c in enumerate(configs):
        arr[i].cfg = _Config(c.tokens, c.hidden, c.group_align, c.group_quant, c.bits, c.outlier_k, c.flags)
    return arr


def rac_calibrate_workspace(configs) -> int:
    arr = _candidates(configs)
    return int(library().rac_calibrate_workspace(arr, len(configs)))


def rac_calibrate(x, ref, configs, target_nmse: float, workspace=None, stream=None):
    """Offline calibration over candidate configurations (RacConfig with the
    sample's tokens and hidden) on the device sample x against ref.  Returns
    (chosen index, per-candidate dicts of wire_bytes, sq_err, sq_x, max_abs,
    nmse, feasible).  Allocates the workspace with torch when none is given."""
    arr = _candidates(configs)
    need = int(library().rac_calibrate_workspace(arr, len(configs)))
    if need == 0:
        raise RacError(1, "rac_calibrate_workspace")
    if workspace is None:
        import torch
        workspace = torch.empty(need, dtype=torch.uint8, device="cuda")
    cap = _nbytes(workspace) if not isinstance(workspace, int) else need
    n = configs[0].tokens * configs[0].hidden
    chosen = ctypes.c_int32(-1)
    _check(library().rac_calibrate(_dev(x, "x", 2, n), _dev(ref, "ref", 2, n), arr, len(configs),
                                   float(target_nmse), _dev(workspace, "workspace", 1, need), cap,
                                   ctypes.byref(chosen), _stream(stream)), "rac_calibrate")
    res = [dict(cfg=configs[i], wire_bytes=int(a.wire_bytes), sq_err=a.sq_err, sq_x=a.sq_x, max_abs=a.max_abs,
                nmse=a.nmse, feasible=bool(a.feasible)) for i, a in enumerate(arr)]
    return int(chosen.value), res


def rac_predictor_layout(cfg: PredictorConfig) -> dict:
    out = _PredOffsets()
    _check(library().rac_predictor_layout(ctypes.byref(cfg._c()), ctypes.byref(out)), "rac_predictor_layout")
    return {f: int(getattr(out, f)) for f, _ in _PredOffsets._fields_}


def rac_predictor_cache_bytes(cfg: PredictorConfig) -> int:
    return int(library().rac_predictor_cache_bytes(ctypes.byref(cfg._c())))


def rac_predictor_workspace_bytes(cfg: PredictorConfig) -> int:
    return int(library().rac_predictor_workspace_bytes(ctypes.byref(cfg._c())))


def predictor_pack(cfg: PredictorConfig, weights: dict):
    """The weight blob (numpy uint8) from named bf16 arrays (uint16 patterns
    of the shapes rac_predictor_layout documents), placed at the library's
    section offsets."""
    import numpy as np
    lay = rac_predictor_layout(cfg)
    blob = np.zeros(lay["total"], dtype=np.uint8)
    for name, arr in weights.items():
        a = np.ascontiguousarray(arr, dtype=np.uint16).view(np.uint8).ravel()
        blob[lay[name]:lay[name] + a.size] = a
    return blob


def rac_predictor_step(cfg: PredictorConfig, weights, cache, pos, h_prev, ref_out, workspace, batch: int | None = None,
                       stream=None) -> None:
    """One predictor step: h_prev (bf16 [batch][hidden]) -> ref_out, updating
    the key-value cache; pos: device int32 [batch]."""
    B = int(batch) if batch is not None else int(pos.numel())
    n = B * cfg.hidden
    _check(library().rac_predictor_step(ctypes.byref(cfg._c()), _dev(weights, "weights", 1, 0),
                                        _dev(cache, "cache", 2, rac_predictor_cache_bytes(cfg) // 2),
                                        _dev(pos, "pos", 4, B), B, _dev(h_prev, "h_prev", 2, n),
                                        _dev(ref_out, "ref_out", 2, n),
                                        _dev(workspace, "workspace", 1, rac_predictor_workspace_bytes(cfg)),
                                        _nbytes(workspace) if not isinstance(workspace, int) else
                                        rac_predictor_workspace_bytes(cfg), _stream(stream)), "rac_predictor_step")
