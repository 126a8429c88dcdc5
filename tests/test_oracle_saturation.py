"""Pins of the oracle's saturation report.

The wire carries one byte per token row and 512-channel block: bit 1 when an
alignment coefficient (alpha* or beta*) of a group starting in the block
overflows fp16 (|v| >= 65520, which round-to-nearest-even takes to infinity;
the field holds +-65504), bit 2 when no fp16 scale covers a quantization group
starting in the block (max|E^d| > 65504 * Qmax: Eq. residual-quantization's
guarantee of no dense clipping fails and the codes clip), bit 4 when an outlier
value of a channel in the block overflows fp16.

Every case below is built from bf16-exact values so the overflowing field, and
the block it belongs to, follow from the construction alone.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2608_04991_amd import workloads as wl
from tests import wirefmt

BF16 = lambda a: wl.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def cfgd(T, d, ga, gq, b, k=0, flags=0):
    return dict(tokens=T, hidden=d, group_align=ga, group_quant=gq, bits=b, outlier_k=k, flags=flags)


def _sat(x, ref, **c):
    rc, wire, _ = oracle.encode(BF16(x), None if ref is None else BF16(ref), **c)
    assert rc == 0
    return wirefmt.sections(wire)["sat"], wirefmt.sections(wire)


def test_ordinary_rows_report_nothing():
    xb, rb, _ = wl.prefill_uplink(0, rows=(0, 8))
    rc, wire, _ = oracle.encode(xb, rb, **cfgd(8, 4096, 128, 128, 4, 8))
    s = wirefmt.sections(wire)["sat"]
    assert s.shape == (8, 8) and not s.any()


def test_scale_saturation_depends_on_qmax_and_marks_the_group_block():
    # zero reference: alpha = 0, beta = mean = 0 for the +-2^20 group, so E = x
    x = np.ones((1, 1024), np.float32)
    x[0, 0:128] = np.tile([2.0 ** 20, -2.0 ** 20], 64)        # block 0, group 0
    x[0, 640:768] = np.tile([65536.0, -65536.0], 64)           # block 1, group 5
    s4, sec = _sat(x, None, **cfgd(1, 1024, 128, 128, 4))
    # 2^20 > 65504 * 7: the scale saturates at 65504 and the codes clip at +-7
    assert s4.tolist() == [[2, 0]]
    assert sec["scale"][0, 0] == 0x7BFF
    codes = wirefmt.unpack_codes(sec["codes"], 1024, 4)[0]
    assert (np.abs(codes[0:128]) == 7).all()
    # 2^20 <= 65504 * 127: at 8 bits a scale covers the group
    s8, _ = _sat(x, None, **cfgd(1, 1024, 128, 128, 8))
    assert s8.tolist() == [[0, 0]]


def test_beta_overflow_threshold_is_the_fp16_rounding_overflow():
    # group means 65280 + 4j over 64 bf16 values (j of them 65536, the rest
    # 65280): 65516 rounds to 65504 (no overflow), 65520 rounds past it
    def row(j):
        v = np.full(64, 65280.0, np.float32)
        v[:j] = 65536.0
        return v
    x = np.zeros((1, 1024), np.float32)
    x[0, 0:64] = row(59)        # mean 65516, block 0
    x[0, 512:576] = row(60)     # mean 65520, block 1
    s, sec = _sat(x, None, **cfgd(1, 1024, 64, 64, 4))
    assert s.tolist() == [[0, 1]]
    assert sec["coef"][0, 0, 1] == 0x7BFF and sec["coef"][0, 8, 1] == 0x7BFF  # both stored as 65504


def test_alpha_overflow_marks_the_alignment_group_block():
    # r = +-2^-10, x = +-2^10 in one group: alpha* = 2^20
    r = np.ones((1, 1024), np.float32)
    x = np.ones((1, 1024), np.float32)
    r[0, 512:640] = np.tile([2.0 ** -10, -2.0 ** -10], 64)
    x[0, 512:640] = np.tile([1024.0, -1024.0], 64)
    s, sec = _sat(x, r, **cfgd(1, 1024, 128, 128, 4))
    assert s.tolist() == [[0, 1]]
    assert sec["coef"][0, 4, 0] == 0x7BFF


def test_outlier_value_overflow_marks_the_channel_block():
    x = np.zeros((1, 1024), np.float32)
    x[0, 600], x[0, 601] = 131072.0, -131072.0   # group 4 (block 1): mean 0, |E| = 2^17
    x[0, 100] = 65280.0                           # block 0: largest |E| there stays below 65520
    x[0, 101] = -65280.0
    # k = 3: channels 600, 601 and (ties -> lower channel) 100
    s, sec = _sat(x, None, **cfgd(1, 1024, 128, 128, 8, 3))
    assert sorted(int(v & 0xFFFF) for v in sec["outl"][0]) == [100, 600, 601]
    assert s.tolist() == [[0, 4]]
    # per-group mode: k_g = 1 of every group of 128
    s, sec = _sat(x, None, **cfgd(1, 1024, 128, 128, 8, 1, oracle.FLAG_GROUP_OUTLIERS))
    assert s.tolist() == [[0, 4]]


def test_pooled_fit_reports_every_row_of_a_saturated_segment():
    T, d = 6, 512
    x = np.full((T, d), 65536.0, np.float32)    # rows 0-3: pooled beta* = 65536
    x[4:] = 65280.0                              # rows 4-5: 65280, no overflow
    xb = BF16(x)
    c = cfgd(T, d, 64, 64, 4)
    rc, wire, _ = oracle.encode_pooled(xb, None, np.array([0, 4, 6], np.int32), **c)
    assert rc == 0
    assert wirefmt.sections(wire)["sat"][:, 0].tolist() == [1, 1, 1, 1, 0, 0]
