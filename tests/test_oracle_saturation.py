"""Pins of the oracle's saturation marks.

The wire's fp16 fields hold the IEEE rounding of their value: an alpha* or
beta* whose round-to-nearest-even overflows (|v| >= 65520, where the tie at
65520 goes to the even significand past the range) is +-infinity, and so is
an outlier value; the scale of a quantization group whose max|E^d| exceeds
65504 * Qmax, which no finite fp16 step covers (Eq. residual-quantization's
guarantee of no dense clipping fails and the codes clip), is +infinity.  Both
ends compute with +-65504 there.

Every case is built from bf16-exact values, so which field overflows, and
what the codes and the reconstruction must then be, follow from the
construction alone.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2608_04991_amd import workloads as wl
from tests import wirefmt

BF16 = lambda a: wl.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))
INF, NINF, MAX = 0x7C00, 0xFC00, 0x7BFF


def cfgd(T, d, ga, gq, b, k=0, flags=0):
    return dict(tokens=T, hidden=d, group_align=ga, group_quant=gq, bits=b, outlier_k=k, flags=flags)


def _enc(x, ref, **c):
    rc, wire, xhat = oracle.encode(BF16(x), None if ref is None else BF16(ref), **c)
    assert rc == 0
    return wirefmt.sections(wire), wire, xhat


def test_ordinary_rows_have_no_marks():
    xb, rb, _ = wl.prefill_uplink(0, rows=(0, 8))
    rc, wire, xhat = oracle.encode(xb, rb, **cfgd(8, 4096, 128, 128, 4, 8))
    assert not wirefmt.saturation_marks(wire).any() and np.isfinite(xhat).all()


def test_scale_past_the_range_is_infinity_and_the_codes_clip():
    # zero reference: alpha = 0, beta = mean = 0 for the +-2^20 group, so E = x
    x = np.ones((1, 1024), np.float32)
    x[0, 0:128] = np.tile([2.0 ** 20, -2.0 ** 20], 64)
    sec, wire, xhat = _enc(x, None, **cfgd(1, 1024, 128, 128, 4))
    # 2^20 > 65504 * 7: no finite step covers the group; it is coded with 65504
    assert sec["scale"][0, 0] == INF and (sec["scale"][0, 1:] != INF).all()
    codes = wirefmt.unpack_codes(sec["codes"], 1024, 4)[0]
    assert (codes[0:128] == np.tile([7, -7], 64)).all()
    assert (xhat[0, 0:128] == np.tile([7 * 65504.0, -7 * 65504.0], 64)).all()
    assert wirefmt.saturation_marks(wire).tolist() == [2]
    # at 8 bits 65504 * 127 covers 2^20: a finite scale, nothing marked
    sec, wire, _ = _enc(x, None, **cfgd(1, 1024, 128, 128, 8))
    assert sec["scale"][0, 0] != INF and not wirefmt.saturation_marks(wire).any()


def test_beta_overflow_threshold_is_the_fp16_rounding_overflow():
    # group means 65280 + 4j over 64 bf16 values (j of them 65536, the rest
    # 65280): 65516 rounds to 65504, 65520 rounds past the range
    def row(j):
        v = np.full(64, 65280.0, np.float32)
        v[:j] = 65536.0
        return v
    x = np.zeros((2, 128), np.float32)
    x[0, 0:64] = row(59)
    x[1, 64:128] = row(60)
    sec, wire, xhat = _enc(x, None, **cfgd(2, 128, 64, 64, 4))
    assert sec["coef"][0, 0, 1] == MAX and sec["coef"][1, 1, 1] == INF
    assert wirefmt.saturation_marks(wire).tolist() == [0, 1]
    # the overflowed beta is used as 65504: E = x - 65504 is 32 or -224, all finite
    assert np.isfinite(xhat).all() and np.abs(xhat[1, 64:128] - x[1, 64:128]).max() <= 224 / 7 / 2 + 1e-3


def test_alpha_overflow_is_infinity_with_its_sign():
    r = np.ones((1, 256), np.float32)
    x = np.ones((1, 256), np.float32)
    r[0, 128:256] = np.tile([2.0 ** -10, -2.0 ** -10], 64)
    x[0, 128:256] = np.tile([-1024.0, 1024.0], 64)          # alpha* = -2^20
    sec, wire, xhat = _enc(x, r, **cfgd(1, 256, 128, 128, 4))
    assert sec["coef"][0, 1, 0] == NINF and sec["coef"][0, 0, 0] != NINF
    assert wirefmt.saturation_marks(wire).tolist() == [1] and np.isfinite(xhat).all()


def test_outlier_value_overflow_is_infinity_and_reconstructs_as_65504():
    x = np.zeros((1, 1024), np.float32)
    x[0, 600], x[0, 601] = 131072.0, -131072.0   # group 4: mean 0, |E| = 2^17
    x[0, 100], x[0, 101] = 65280.0, -65280.0     # |E| = 65280 stays finite
    for c, k in ((cfgd(1, 1024, 128, 128, 8, 4), None), (cfgd(1, 1024, 128, 128, 8, 1, oracle.FLAG_GROUP_OUTLIERS), 1)):
        sec, wire, xhat = _enc(x, None, **c)
        if k is None:
            vals = {int(v & 0xFFFF): int(v >> 16) for v in sec["outl"][0]}
            assert vals[600] == INF and vals[601] == NINF and vals[100] == 0x7BF8
        else:
            assert sec["gval"][0, 4, 0] == INF and sec["goff"][0, 4, 0] == 600 % 128
        assert xhat[0, 600] == 65504.0
        assert wirefmt.saturation_marks(wire).tolist() == [4]


def test_pooled_fit_marks_every_row_of_a_saturated_segment():
    T, d = 6, 512
    x = np.full((T, d), 65536.0, np.float32)    # rows 0-3: pooled beta* = 65536
    x[4:] = 65280.0                              # rows 4-5: 65280, finite
    rc, wire, _ = oracle.encode_pooled(BF16(x), None, np.array([0, 4, 6], np.int32), **cfgd(T, d, 64, 64, 4))
    assert rc == 0
    assert wirefmt.saturation_marks(wire).tolist() == [1, 1, 1, 1, 0, 0]
    # the decode reads the marked wire back to the same finite reconstruction
    rc, xh = oracle.decode(wire, None, **cfgd(T, d, 64, 64, 4))
    assert rc == 0 and np.isfinite(xh).all()
