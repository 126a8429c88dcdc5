"""Pins of the oracle's pooled fit (one (alpha, beta) per segment of rows and
channel group: the affine-fit equation over all fitting positions of the
segment).

Against things other than the oracle itself: exact rational least squares
over the pooled data, float64 pooled moments, exact affine data that holds
across a segment, the zero-variance rule over a segment, and the per-token
fit (independently pinned) for one-row segments.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2608_04991_amd import workloads as wl
from tests import wirefmt


def f16val(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


def cfgd(T, d, ga, gq, b, k=0, flags=0):
    return dict(tokens=T, hidden=d, group_align=ga, group_quant=gq, bits=b, outlier_k=k, flags=flags)


def test_one_row_segments_are_the_per_token_fit():
    T, d = 12, 512
    xb, rb, _ = wl.prefill_uplink(1, rows=(0, T), hidden=d)
    for k, flags in ((0, 0), (8, 0), (2, oracle.FLAG_GROUP_OUTLIERS)):
        c = cfgd(T, d, 128, 128, 4, k, flags)
        rc1, w1, x1 = oracle.encode(xb, rb, **c)
        rc2, w2, x2 = oracle.encode_pooled(xb, rb, np.arange(T + 1), **c)
        assert rc1 == rc2 == 0
        assert wirefmt.header(w2)["flags"] == wirefmt.header(w1)["flags"] | 16
        w2 = w2.copy()
        w2[6] = w1[6]
        assert np.array_equal(w1, w2) and np.array_equal(x1.view(np.uint32), x2.view(np.uint32))


def _exact_pooled_ls(r, x):
    """Exact least squares of x ~ a r + b over all pooled values."""
    R = [Fraction(float(v)) for v in r.ravel()]
    X = [Fraction(float(v)) for v in x.ravel()]
    n = len(R)
    mr, mx = sum(R) / n, sum(X) / n
    crr = sum((a - mr) ** 2 for a in R)
    crx = sum((a - mr) * (b - mx) for a, b in zip(R, X))
    if crr == 0:
        return Fraction(0), mx
    a = crx / crr
    return a, mx - a * mr


def _near_f16_boundary(v, rel=1e-5):
    f = np.float32(v)
    h = np.float16(f)
    lo, hi = np.nextafter(h, np.float16(-np.inf)), np.nextafter(h, np.float16(np.inf))
    mids = [(np.float64(h) + np.float64(lo)) / 2, (np.float64(h) + np.float64(hi)) / 2]
    return any(abs(float(v) - m) <= rel * (1 + abs(float(v))) for m in mids)


@pytest.mark.parametrize("seed", range(4))
def test_pooled_fit_matches_exact_rational_least_squares(seed):
    rng = np.random.default_rng(seed)
    T, d, g = 9, 32, 16
    seg = np.array([0, 2, 3, 7, 9])
    r = rng.standard_normal((T, d)).astype(np.float32) * 2
    x = (0.7 * r + 0.3 + rng.standard_normal((T, d)) * 0.4).astype(np.float32)
    xb, rb = wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(r)
    rc, wire, _ = oracle.encode_pooled(xb, rb, seg, **cfgd(T, d, g, g, 8))
    assert rc == 0
    coef = wirefmt.sections(wire)["coef"]
    rf, xf = wl.bf16_bits_to_f32(rb), wl.bf16_bits_to_f32(xb)
    for s in range(seg.size - 1):
        lo, hi = seg[s], seg[s + 1]
        for j in range(d // g):
            a, b = _exact_pooled_ls(rf[lo:hi, j * g:(j + 1) * g], xf[lo:hi, j * g:(j + 1) * g])
            for t in range(lo, hi):   # every row of the segment carries the pair
                assert coef[t, j, 0] == coef[lo, j, 0] and coef[t, j, 1] == coef[lo, j, 1]
            for got, want in ((coef[lo, j, 0], a), (coef[lo, j, 1], b)):
                exact16 = np.float16(float(want)).view(np.uint16)
                assert got == exact16 or _near_f16_boundary(float(want)), (s, j, got, exact16, float(want))


def test_pooled_moments_match_float64():
    rng = np.random.default_rng(3)
    for n in (1, 2, 3, 5, 8, 13, 64, 65, 200):
        rows = rng.standard_normal((n, 16)).astype(np.float32) + rng.standard_normal((n, 1)).astype(np.float32) * 3
        xs = (rows * 1.5 - 2 + rng.standard_normal((n, 16)) * 0.1).astype(np.float32)
        ms = [oracle.moments_row(rows[i], xs[i]) for i in range(n)]
        m = oracle.moments_pool(ms)
        r64, x64 = rows.astype(np.float64).ravel(), xs.astype(np.float64).ravel()
        assert m.n == 16 * n
        np.testing.assert_allclose(m.mr, r64.mean(), rtol=1e-5, atol=1e-5)
        np.testing.assert_allclose(m.mx, x64.mean(), rtol=1e-5, atol=1e-5)
        np.testing.assert_allclose(m.crr, ((r64 - r64.mean()) ** 2).sum(), rtol=1e-4)
        np.testing.assert_allclose(m.crx, ((r64 - r64.mean()) * (x64 - x64.mean())).sum(), rtol=1e-4)


def test_exact_affine_across_a_segment_gives_zero_codes_and_exact_reconstruction():
    rng = np.random.default_rng(8)
    T, d, g = 10, 256, 64
    r = rng.integers(-32, 33, (T, d)).astype(np.float32) / 4
    x = np.float32(1.25) * r - np.float32(0.5)          # one pair for every row
    xb, rb = wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(r)
    rc, wire, xhat = oracle.encode_pooled(xb, rb, np.array([0, 3, 10]), **cfgd(T, d, g, g, 4))
    s = wirefmt.sections(wire)
    assert np.all(f16val(s["coef"][..., 0]) == 1.25) and np.all(f16val(s["coef"][..., 1]) == -0.5)
    assert np.all(s["codes"] == 0) and np.all(s["scale"] == 0)
    assert np.array_equal(xhat, wl.bf16_bits_to_f32(xb))


def test_constant_reference_over_a_segment_gives_alpha_zero_and_the_pooled_mean():
    T, d, g = 6, 64, 32
    r = np.full((T, d), 3.0, np.float32)
    x = (np.arange(T * d, dtype=np.float32).reshape(T, d) % 7) / 8   # dyadic, exact pooled mean
    xb, rb = wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(r)
    seg = np.array([0, 4, 6])
    rc, wire, _ = oracle.encode_pooled(xb, rb, seg, **cfgd(T, d, g, g, 4))
    coef = wirefmt.sections(wire)["coef"]
    for s in range(2):
        for j in range(d // g):
            block = x[seg[s]:seg[s + 1], j * g:(j + 1) * g].astype(np.float64)
            assert coef[seg[s], j, 0] == 0
            assert coef[seg[s], j, 1] == np.float16(block.mean()).view(np.uint16)


def test_pooled_wire_decodes_to_the_sender_reconstruction():
    T, d = 20, 512
    xb, rb, _ = wl.prefill_uplink(2, rows=(0, T), hidden=d)
    c = cfgd(T, d, 64, 128, 4, 4)
    rc, wire, xhat = oracle.encode_pooled(xb, rb, np.array([0, 5, 6, 20]), **c)
    rc2, xdec = oracle.decode(wire, rb, **c)
    assert rc == rc2 == 0 and np.array_equal(xhat.view(np.uint32), xdec.view(np.uint32))


def test_pooled_segment_errors():
    xb = wl.f32_to_bf16_bits(np.ones((4, 64), np.float32))
    c = cfgd(4, 64, 64, 64, 4)
    for seg in ([0, 4, 4], [1, 4], [0, 3], [0, 2, 1, 4]):
        assert oracle.encode_pooled(xb, None, np.array(seg), **c)[0] == oracle.ORC_ERR_INVALID
