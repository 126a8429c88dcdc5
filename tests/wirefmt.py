"""Test-side reader of the RAC wire format (header + sections), in numpy.

Written against the documented layout only, so tests can inspect wires from
either the oracle or the HIP library without trusting either one's code:

  0  u32 magic 'RAC1'   4 u16 version   6 u16 flags (1 outliers, 2 fixed step,
                                                      4 zero reference)
  8  u32 tokens        12 u32 hidden   16 u32 g_a   20 u32 g_q
  24 u8 bits  25 u8 coef fmt  26 u8 scale fmt  27 u8 outlier fmt  28 u16 k
  32 u64 off_coef  40 off_scale  48 off_codes  56 off_outl  64 total
  72 u64 off_ooff (per-group outliers only, else 0)
  sections 256-byte aligned, zero padded; version 2.

Outliers: per token (flag 1, fmt 1) one u32 per entry, channel in the low
half and the fp16 value in the high half; per quantization group (flag 8,
fmt 2) fp16 values [T][G][k_g] at off_outl and u8 in-group offsets
[T][G][k_g] at off_ooff.

The fp16 fields (coefficients, scales, outlier values) hold IEEE fp16: +-inf
marks a rounding past the fp16 range (read as +-65504 by both ends).
"""
from __future__ import annotations

import numpy as np

MAGIC = 0x31434152


def up256(v: int) -> int:
    return (v + 255) // 256 * 256


GROUP_OUTLIERS = 4   # config flag of the per-group outlier mode


def expected_layout(tokens, hidden, group_align, group_quant, bits, outlier_k=0, flags=0):
    coef = tokens * (hidden // group_align) * 4
    scale = 0 if (flags & 1) else tokens * (hidden // group_quant) * 2
    codes = tokens * hidden * bits // 8
    off_coef = 256
    off_scale = up256(off_coef + coef)
    off_codes = up256(off_scale + scale)
    off_outl = up256(off_codes + codes)
    if flags & GROUP_OUTLIERS:
        n = tokens * (hidden // group_quant) * outlier_k
        off_ooff = up256(off_outl + 2 * n)
        total = up256(off_ooff + n)
    else:
        off_ooff = 0
        total = up256(off_outl + tokens * outlier_k * 4)
    return dict(off_coef=off_coef, off_scale=off_scale, off_codes=off_codes,
                off_outl=off_outl, total=total, off_ooff=off_ooff)


def header(wire: np.ndarray) -> dict:
    w = np.asarray(wire, dtype=np.uint8)
    u32 = lambda o: int(w[o:o + 4].view(np.uint32)[0])
    u16 = lambda o: int(w[o:o + 2].view(np.uint16)[0])
    u64 = lambda o: int(w[o:o + 8].view(np.uint64)[0])
    return dict(magic=u32(0), version=u16(4), flags=u16(6), tokens=u32(8), hidden=u32(12),
                group_align=u32(16), group_quant=u32(20), bits=int(w[24]), coef_fmt=int(w[25]),
                scale_fmt=int(w[26]), outl_fmt=int(w[27]), outlier_k=u16(28),
                off_coef=u64(32), off_scale=u64(40), off_codes=u64(48), off_outl=u64(56),
                total=u64(64), off_ooff=u64(72))


def sections(wire: np.ndarray) -> dict:
    """Split a wire into typed per-row arrays (views)."""
    w = np.asarray(wire, dtype=np.uint8)
    h = header(w)
    T, d, ga, gq, b, k = (h["tokens"], h["hidden"], h["group_align"], h["group_quant"],
                          h["bits"], h["outlier_k"])
    fixed = bool(h["flags"] & 2)
    out = {"header": h}
    n = T * (d // ga) * 2
    out["coef"] = w[h["off_coef"]:h["off_coef"] + 2 * n].view(np.uint16).reshape(T, d // ga, 2)
    if fixed:
        out["scale"] = None
    else:
        n = T * (d // gq)
        out["scale"] = w[h["off_scale"]:h["off_scale"] + 2 * n].view(np.uint16).reshape(T, d // gq)
    n = T * d * b // 8
    out["codes"] = w[h["off_codes"]:h["off_codes"] + n].reshape(T, d * b // 8)
    if h["flags"] & 8:
        n = T * (d // gq) * k
        out["outl"] = None
        out["gval"] = w[h["off_outl"]:h["off_outl"] + 2 * n].view(np.uint16).reshape(T, d // gq, k)
        out["goff"] = w[h["off_ooff"]:h["off_ooff"] + n].reshape(T, d // gq, k)
    else:
        n = T * k
        out["outl"] = w[h["off_outl"]:h["off_outl"] + 4 * n].view(np.uint32).reshape(T, k)
        out["gval"] = out["goff"] = None
    return out


def unpack_codes(code_rows: np.ndarray, hidden: int, bits: int) -> np.ndarray:
    """Signed integer codes [T, hidden] from packed rows (LSB-first bit string)."""
    rows = np.asarray(code_rows, dtype=np.uint8)
    bitstr = np.unpackbits(rows, axis=1, bitorder="little")[:, :hidden * bits]
    bitstr = bitstr.reshape(rows.shape[0], hidden, bits).astype(np.int64)
    u = (bitstr << np.arange(bits, dtype=np.int64)).sum(axis=2)
    return np.where(u >= (1 << (bits - 1)), u - (1 << bits), u)


def padding_is_zero(wire: np.ndarray) -> bool:
    """Every byte outside the header fields and the sections is zero."""
    w = np.asarray(wire, dtype=np.uint8)
    h = header(w)
    T, d, ga, gq, b, k = (h["tokens"], h["hidden"], h["group_align"], h["group_quant"],
                          h["bits"], h["outlier_k"])
    used = np.zeros(w.size, dtype=bool)
    used[:80] = True
    used[h["off_coef"]:h["off_coef"] + T * (d // ga) * 4] = True
    if not (h["flags"] & 2):
        used[h["off_scale"]:h["off_scale"] + T * (d // gq) * 2] = True
    used[h["off_codes"]:h["off_codes"] + T * d * b // 8] = True
    if h["flags"] & 8:
        n = T * (d // gq) * k
        used[h["off_outl"]:h["off_outl"] + 2 * n] = True
        used[h["off_ooff"]:h["off_ooff"] + n] = True
    else:
        used[h["off_outl"]:h["off_outl"] + T * k * 4] = True
        used[72:80] = False   # off_ooff is 0 without per-group outliers
    return bool(np.all(w[~used] == 0)) and bool(np.all(w[30:32] == 0))


def _inf16(a) -> np.ndarray:
    return (np.asarray(a, dtype=np.uint16) & 0x7FFF) == 0x7C00


def saturation_marks(wire: np.ndarray) -> np.ndarray:
    """Per token row, the OR of 1 (an alpha or beta field holds +-inf), 2 (a
    scale holds +inf) and 4 (an outlier value holds +-inf)."""
    s = sections(wire)
    T = s["header"]["tokens"]
    m = np.zeros(T, dtype=np.int64)
    m |= np.where(_inf16(s["coef"]).reshape(T, -1).any(axis=1), 1, 0)
    if s["scale"] is not None:
        m |= np.where(_inf16(s["scale"]).reshape(T, -1).any(axis=1), 2, 0)
    if s["outl"] is not None:
        m |= np.where(_inf16(s["outl"] >> 16).reshape(T, -1).any(axis=1), 4, 0)
    if s["gval"] is not None:
        m |= np.where(_inf16(s["gval"]).reshape(T, -1).any(axis=1), 4, 0)
    return m
