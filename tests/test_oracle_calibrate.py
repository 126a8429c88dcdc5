"""Pins of the calibration oracle (oracle/calibrate.py) against what does not
come from it: exact rational sums, the error bound of Eq. error-bound, the
documented wire layout, hand-worked decision tables, exact affine data (zero
error for every candidate) and planted mistakes."""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import calibrate as cal
from paper_2608_04991_amd import workloads as wl
from tests import wirefmt


def cfgd(T, d, ga, gq, b, k=0, flags=0):
    return dict(tokens=T, hidden=d, group_align=ga, group_quant=gq, bits=b, outlier_k=k, flags=flags)


def _exact_stats(x_bits, xhat):
    x = [Fraction(float(v)) for v in wl.bf16_bits_to_f32(x_bits).ravel()]
    h = [Fraction(float(v)) for v in np.asarray(xhat, np.float32).ravel()]
    se = sum((a - b) ** 2 for a, b in zip(x, h))
    sx = sum(a * a for a in x)
    mx = max(abs(a - b) for a, b in zip(x, h))
    return se, sx, mx


def test_error_sums_match_exact_rational_arithmetic():
    rng = np.random.default_rng(0)
    xb = wl.f32_to_bf16_bits(rng.standard_normal((3, 40)).astype(np.float32) * 10.0 ** rng.integers(-3, 4, (3, 40)))
    xh = (wl.bf16_bits_to_f32(xb) * (1 + rng.standard_normal((3, 40)).astype(np.float32) * 1e-3)).astype(np.float32)
    se, sx, mx = cal.error_stats(xb, xh)
    ese, esx, emx = _exact_stats(xb, xh)
    assert abs(Fraction(se) - ese) <= ese * Fraction(1, 10 ** 14)
    assert Fraction(sx) == esx or abs(Fraction(sx) - esx) <= esx * Fraction(1, 10 ** 15)
    assert Fraction(mx) == emx


def test_bf16_reconstructions_are_read_as_bf16():
    xb = wl.f32_to_bf16_bits(np.float32([[1.0, 2.0, -3.0, 0.5]]))
    hb = wl.f32_to_bf16_bits(np.float32([[1.0, 2.5, -3.0, 0.25]]))
    se, sx, mx = cal.error_stats(xb, hb, xhat_bf16=True)
    assert (se, sx, mx) == (0.25 + 0.0625, 1 + 4 + 9 + 0.25, 0.5)


def test_exact_affine_rows_have_zero_error_for_every_candidate_and_the_cheapest_wins():
    # x = 1.25 r - 0.5 exactly (dyadic values): every configuration reconstructs x exactly
    # (64 rows, so that the sections' sizes differ by more than their padding)
    rng = np.random.default_rng(1)
    r = rng.integers(-32, 33, (64, 256)).astype(np.float32) / 4
    xb, rb = wl.f32_to_bf16_bits(1.25 * r - 0.5), wl.f32_to_bf16_bits(r)
    cands = [cfgd(64, 256, 64, 64, 8), cfgd(64, 256, 128, 128, 2),
             cfgd(64, 256, 32, 32, 4, 2, oracle.FLAG_GROUP_OUTLIERS), cfgd(64, 256, 256, 256, 2)]
    i, res = cal.calibrate(xb, rb, cands, target=0.0)
    assert all(rr["sq_err"] == 0.0 and rr["max_abs"] == 0.0 and rr["feasible"] for rr in res)
    assert i == 3 and res[3]["wire_bytes"] == min(rr["wire_bytes"] for rr in res)


def test_wire_cost_is_the_documented_layout():
    for c in [cfgd(64, 4096, 128, 128, 4, 8), cfgd(16, 4096, 64, 4096, 2), cfgd(7, 520, 8, 8, 3, 2, 4),
              cfgd(256, 3584, 128, 64, 8, 1, 4)]:
        assert cal.wire_bytes(c) == wirefmt.expected_layout(**c)["total"]


def test_error_of_a_coded_sample_respects_the_error_bound():
    """Eq. error-bound without outliers: sum (x - H-hat)^2 is at most
    sum over groups of g_q * s^2 / 4, up to the binary32 roundings of E and
    H-hat (slack of 1e-4 relative plus a per-element term)."""
    T, d, g = 32, 1024, 64
    xb, rb, _ = wl.prefill_uplink(0, rows=(0, T), hidden=d)
    for bits in (2, 4, 8):
        c = cfgd(T, d, g, g, bits)
        rc, wire, xhat = oracle.encode(xb, rb, **c)
        se, sx, _ = cal.error_stats(xb, xhat)
        s = np.asarray(wirefmt.sections(wire)["scale"], np.uint16).view(np.float16).astype(np.float64)
        bound = float((g * s * s / 4).sum())
        assert 0 < se <= bound * (1 + 1e-4) + T * d * 1e-12


def test_decision_rule_on_hand_worked_tables():
    R = lambda b, e, n: dict(wire_bytes=b, sq_err=e, nmse=n)
    # feasible: 1, 2, 3 (nmse <= 0.01); fewest bytes 100 at 1 and 3, smaller error at 3
    t = [R(90, 5.0, 0.05), R(100, 2.0, 0.008), R(120, 1.0, 0.004), R(100, 1.5, 0.006)]
    assert cal.choose(t, 0.01) == 3
    # equal bytes and error: the earlier candidate
    assert cal.choose([R(10, 1.0, 0.1), R(10, 1.0, 0.1)], 0.5) == 0
    # nothing meets the target: smallest error (ties to fewer bytes)
    t = [R(90, 5.0, 0.5), R(100, 2.0, 0.2), R(80, 2.0, 0.2)]
    assert cal.choose(t, 0.01) == 2
    # no target: the cheapest overall
    assert cal.choose(t, math.inf) == 2
    # the target is inclusive
    assert cal.choose([R(50, 3.0, 0.01), R(40, 4.0, 0.0100001)], 0.01) == 0


def test_more_bits_lower_the_error_and_the_target_picks_the_bit_width():
    T, d = 16, 4096
    xb, rb, _ = wl.prefill_uplink(0, rows=(0, T))
    cands = [cfgd(T, d, 128, 128, b, 8) for b in (2, 3, 4, 8)]
    res = [cal.evaluate(xb, rb, c) for c in cands]
    e = [r["nmse"] for r in res]
    assert e[0] > e[1] > e[2] > e[3] > 0
    assert [r["wire_bytes"] for r in res] == sorted(r["wire_bytes"] for r in res)
    # a target between the 3- and 4-bit errors picks 4 bits
    i, _ = cal.calibrate(xb, rb, cands, target=math.sqrt(e[1] * e[2]))
    assert i == 2


def test_quality_is_invariant_under_power_of_two_scaling():
    """Scaling x and ref by 2^k scales every coefficient, scale, outlier
    and reconstruction by 2^k exactly (the codec's metamorphic relation), so
    the squared error grows by 4^k while the normalized error and the choice
    do not change."""
    T, d = 8, 1024
    xb, rb, _ = wl.prefill_uplink(0, rows=(0, T), hidden=d)
    up = lambda b: wl.f32_to_bf16_bits(wl.bf16_bits_to_f32(b) * np.float32(4.0))
    c = cfgd(T, d, 128, 128, 4, 4)
    a, b = cal.evaluate(xb, rb, c), cal.evaluate(up(xb), up(rb), c)
    assert b["sq_err"] == a["sq_err"] * 16 and b["max_abs"] == a["max_abs"] * 4
    assert b["nmse"] == a["nmse"] and a["nmse"] < 0.01


PLANTED = [
    ("bytes_maximized", "choose", lambda results, target: max(range(len(results)),
                                                              key=lambda i: results[i]["wire_bytes"])),
    ("unnormalized_error", "nmse", lambda se, sx: se),
    ("float32_differences", "error_stats", lambda x, h, b=False: (
        float(np.sum((wl.bf16_bits_to_f32(x) - np.asarray(h, np.float32)) ** 2, dtype=np.float32)),
        float(np.sum(wl.bf16_bits_to_f32(x) ** 2, dtype=np.float32)), 0.0)),
    ("target_exclusive", "choose", lambda results, target: (
        min([i for i, r in enumerate(results) if r["nmse"] < target] or [0],
            key=lambda i: (results[i]["wire_bytes"], results[i]["sq_err"], i)))),
]


@pytest.mark.parametrize("name,attr,fn", PLANTED, ids=[p[0] for p in PLANTED])
def test_planted_calibration_mistake_fails_a_pin(monkeypatch, name, attr, fn):
    monkeypatch.setattr(cal, attr, fn)
    pins = [test_error_sums_match_exact_rational_arithmetic, test_bf16_reconstructions_are_read_as_bf16,
            test_exact_affine_rows_have_zero_error_for_every_candidate_and_the_cheapest_wins,
            test_decision_rule_on_hand_worked_tables,
            test_more_bits_lower_the_error_and_the_target_picks_the_bit_width,
            test_quality_is_invariant_under_power_of_two_scaling]
    caught = 0
    for p in pins:
        try:
            p()
        except (AssertionError, TypeError, ValueError):
            caught += 1
    assert caught, f"no pin caught {name}"
