"""Pins of the oracle's per-group outlier mode (the outlier paragraph of the
paper's encoding section: the mask M_j keeps the k_g largest magnitudes of
every fixed quantization group, and the packet carries in-group offsets and
the fp16-rounded values).

Each check rebuilds what the mode must produce from the wire's coefficients
and the inputs, in numpy, and compares: a brute-force sort of every group by
(larger |E| first, lower offset first), the fp16 rounding of the chosen
values, the dense base with those positions zeroed, the round-up scale of the
dense base, and the reconstruction R~ + O-hat at the outliers.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2608_04991_amd import workloads as wl
from tests import wirefmt

QMAX = {2: 1, 3: 3, 4: 7, 8: 127}
G = oracle.FLAG_GROUP_OUTLIERS


def f16val(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


def cfgd(T, d, ga, gq, b, k=0, flags=0):
    return dict(tokens=T, hidden=d, group_align=ga, group_quant=gq, bits=b, outlier_k=k,
                flags=flags)


def _residual(wire, xb, rb, ga):
    """E = x - (alpha r + beta) in numpy binary32 from the wire's fp16 pair
    (alpha*r is exact for an fp16 alpha and a bf16 r, so one rounding)."""
    s = wirefmt.sections(wire)
    x = wl.bf16_bits_to_f32(xb)
    r = np.zeros_like(x) if rb is None else wl.bf16_bits_to_f32(rb)
    a = np.repeat(f16val(s["coef"][..., 0]), ga, axis=1)
    b = np.repeat(f16val(s["coef"][..., 1]), ga, axis=1)
    rt = (a * r + b).astype(np.float32)
    return s, x, rt, (x - rt).astype(np.float32)


def _brute_force_offsets(e, gq, kg):
    """[T, G, kg] in-group offsets: per group the kg largest |e|, ties to the
    lower offset, listed ascending."""
    T, d = e.shape
    out = np.zeros((T, d // gq, kg), np.int64)
    for t in range(T):
        for g in range(d // gq):
            seg = e[t, g * gq:(g + 1) * gq]
            order = sorted(range(gq), key=lambda o: (-abs(float(seg[o])), o))
            out[t, g] = sorted(order[:kg])
    return out


def _check_group_mode(c, xb, rb, wire, xhat):
    T, d, ga, gq, bits, kg = (c["tokens"], c["hidden"], c["group_align"], c["group_quant"],
                              c["bits"], c["outlier_k"])
    q = QMAX[bits]
    s, x, rt, e = _residual(wire, xb, rb, ga)
    offs = _brute_force_offsets(e, gq, kg)
    assert np.array_equal(s["goff"].astype(np.int64), offs)
    ch = offs + (np.arange(d // gq) * gq)[None, :, None]
    e_at = np.take_along_axis(e, ch.reshape(T, -1), axis=1).reshape(T, d // gq, kg)
    assert np.array_equal(s["gval"], np.clip(e_at, -65504, 65504).astype(np.float16).view(np.uint16))
    dense = np.ones((T, d), bool)
    np.put_along_axis(dense, ch.reshape(T, -1), False, axis=1)
    ed = np.where(dense, e, np.float32(0)).reshape(T, d // gq, gq)
    codes = wirefmt.unpack_codes(s["codes"], d, bits)
    assert np.all(codes[~dense] == 0)
    if not (c["flags"] & oracle.FLAG_FIXED_STEP):
        m = np.abs(ed).max(axis=2)
        sc = s["scale"]
        nz = m > 0
        assert np.all(sc[~nz] == 0)
        assert np.all(f16val(sc[nz]) * q >= m[nz])
        below = (sc.astype(np.int32) - 1).clip(0).astype(np.uint16)
        assert np.all((f16val(below)[nz] * q < m[nz]) | (sc[nz] <= 1))
        sce = np.repeat(f16val(sc), gq, axis=1)
        want = np.clip(np.rint(np.where(sce > 0, ed.reshape(T, d) / np.where(sce > 0, sce, 1), 0)),
                       -q, q)
        assert np.array_equal(codes, want.astype(np.int64))
        eh = codes.astype(np.float32) * sce
    else:
        eh = None
    if xhat is not None and xhat.dtype == np.float32:
        # outliers: R~ + O-hat, one binary32 rounding
        val = f16val(s["gval"]).reshape(T, -1)
        rt_at = np.take_along_axis(rt, ch.reshape(T, -1), axis=1)
        got = np.take_along_axis(xhat, ch.reshape(T, -1), axis=1)
        assert np.array_equal(got.view(np.uint32), (rt_at + val).astype(np.float32).view(np.uint32))
        if eh is not None:
            assert np.array_equal(xhat[dense].view(np.uint32), (rt + eh)[dense].view(np.uint32))
    return s


@pytest.mark.parametrize("gq,kg,bits", [(64, 1, 4), (128, 2, 4), (128, 4, 2), (256, 8, 8),
                                        (32, 8, 3), (8, 2, 4)])
def test_group_outliers_match_brute_force_on_uplink_rows(gq, kg, bits):
    T, d = 12, 512
    xb, rb, _ = wl.prefill_uplink(0, rows=(0, T), hidden=d)
    c = cfgd(T, d, 128 if gq >= 128 else 64, gq, bits, kg, G)
    rc, wire, xhat = oracle.encode(xb, rb, **c)
    assert rc == 0
    _check_group_mode(c, xb, rb, wire, xhat)


def test_group_outliers_ties_go_to_the_lower_offset():
    """ref = 0 and x = c + p per group with sum(p) = 0, so beta = c exactly and
    E = p: small integers with many equal magnitudes and signed zeros."""
    rng = np.random.default_rng(5)
    T, d, gq, kg = 6, 256, 32, 8
    x = np.zeros((T, d), np.float32)
    for t in range(T):
        for g in range(d // gq):
            v = rng.integers(-3, 4, gq // 2).astype(np.float32)
            p = np.concatenate([v, -v])[rng.permutation(gq)]
            x[t, g * gq:(g + 1) * gq] = 1.5 + p
    xb = wl.f32_to_bf16_bits(x)
    c = cfgd(T, d, gq, gq, 4, kg, G)
    rc, wire, xhat = oracle.encode(xb, None, **c)
    assert rc == 0
    s = _check_group_mode(c, xb, None, wire, xhat)
    assert np.all(f16val(s["coef"][..., 1]) == 1.5)
    # a group whose residual is all zero gives offsets 0..kg-1 and zero values
    xb0 = wl.f32_to_bf16_bits(np.full((1, d), 0.25, np.float32))
    rc, wire, xhat = oracle.encode(xb0, None, **cfgd(1, d, gq, gq, 4, kg, G))
    s = wirefmt.sections(wire)
    assert np.array_equal(s["goff"][0], np.tile(np.arange(kg, dtype=np.uint8), (d // gq, 1)))
    assert np.all(s["gval"] == 0) and np.all(s["scale"] == 0)
    assert np.all(xhat == 0.25)


def test_one_group_per_row_selects_what_the_per_token_mode_selects():
    """With g_q = d the per-group mode has one group per row; its outliers,
    codes and reconstruction must equal the per-token mode's."""
    T, d, k = 16, 256, 8
    xb, rb, _ = wl.prefill_uplink(2, rows=(0, T), hidden=d)
    rc1, w_tok, x_tok = oracle.encode(xb, rb, **cfgd(T, d, 64, d, 4, k))
    rc2, w_grp, x_grp = oracle.encode(xb, rb, **cfgd(T, d, 64, d, 4, k, G))
    assert rc1 == rc2 == 0
    st, sg = wirefmt.sections(w_tok), wirefmt.sections(w_grp)
    assert np.array_equal(sg["goff"][:, 0, :].astype(np.uint32), st["outl"] & 0xFFFF)
    assert np.array_equal(sg["gval"][:, 0, :].astype(np.uint32), st["outl"] >> 16)
    for key in ("coef", "scale", "codes"):
        assert np.array_equal(sg[key], st[key]), key
    assert np.array_equal(x_grp.view(np.uint32), x_tok.view(np.uint32))


def test_group_outlier_layout_header_and_padding():
    for c in [cfgd(4096, 4096, 128, 128, 4, 1, G), cfgd(3, 520, 8, 8, 3, 2, G),
              cfgd(5, 256, 32, 16, 8, 4, G | oracle.FLAG_FIXED_STEP), cfgd(0, 512, 64, 256, 2, 16, G)]:
        assert oracle.layout(**c) == wirefmt.expected_layout(**c)
    lay = oracle.layout(**cfgd(4096, 4096, 128, 128, 4, 1, G))
    # 4-bit codes + fp16 scale + fp16 (alpha, beta) + one 3-byte outlier per group of 128
    assert lay["total"] == 256 + 4096 * (32 * 4 + 32 * 2 + 2048) + 4096 * 32 * 3
    T, d = 5, 520
    xb, rb, _ = wl.affine_pair(wl.AffineRecipe(T, d, 8), 0)
    rc, wire, _ = oracle.encode(xb, rb, **cfgd(T, d, 8, 8, 3, 2, G))
    h = wirefmt.header(wire)
    assert h["flags"] == 8 and h["outl_fmt"] == 2 and h["outlier_k"] == 2
    assert h["off_ooff"] == oracle.layout(**cfgd(T, d, 8, 8, 3, 2, G))["off_ooff"] > h["off_outl"]
    assert wirefmt.padding_is_zero(wire)


@pytest.mark.parametrize("flags", [0, oracle.FLAG_XHAT_BF16, oracle.FLAG_FIXED_STEP])
def test_group_mode_sender_equals_receiver_bitwise(flags):
    T, d, gq = 10, 384, 64
    xb, rb, _ = wl.prefill_uplink(4, rows=(0, T), hidden=d)
    steps = np.full(d // gq, 0.03, np.float32)
    c = cfgd(T, d, 128, gq, 4, 3, G | flags)
    rc, wire, xhat = oracle.encode(xb, rb, steps, **c)
    rc2, xdec = oracle.decode(wire, rb, steps, **c)
    assert rc == rc2 == 0
    assert np.array_equal(xhat.view(np.uint8), xdec.view(np.uint8))
    if flags == oracle.FLAG_FIXED_STEP:
        _check_group_mode(c, xb, rb, wire, xhat)


def test_group_mode_error_paths():
    ok = cfgd(2, 256, 64, 64, 4, 2, G)
    for bad in [dict(group_quant=512, hidden=512), dict(outlier_k=0), dict(outlier_k=17),
                dict(outlier_k=17, group_quant=128), dict(group_quant=8, outlier_k=3)]:
        with pytest.raises(ValueError):
            oracle.layout(**dict(ok, **bad))
    assert oracle.layout(**dict(ok, group_quant=8, hidden=256, outlier_k=2))
    xb = wl.f32_to_bf16_bits(np.random.default_rng(1).standard_normal((2, 256)))
    rc, wire, _ = oracle.encode(xb, None, **ok)
    assert rc == 0
    bad = wire.copy()
    bad[wirefmt.header(wire)["off_ooff"]] = 64          # in-group offset >= g_q
    assert oracle.decode(bad, None, **ok)[0] == oracle.ORC_ERR_FORMAT
    assert oracle.decode(wire, None, **dict(ok, flags=0))[0] == oracle.ORC_ERR_FORMAT
