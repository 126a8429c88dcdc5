"""GPU parity of the HIP codec against the CPU oracle, through the C ABI.

Small cases run the oracle on every row; they span several wavefront tiles
(four rows per block), ragged row counts, a partial last 512-channel chunk,
every bit width, groups below and above one chunk, per-token outliers with
ties (both selection paths), zero references, bf16 output and the fixed-step
mode.  The full benchmark shapes are checked on sampled rows, which the
oracle can compute one by one because rows are independent.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2608_04991_amd as rac
from paper_2608_04991_amd import workloads as wl
from tests import wirefmt
from tests.gpu_util import assert_parity, cfgd, gpu_run, oracle_run, say

pytestmark = pytest.mark.gpu
GRP = rac.RAC_FLAG_GROUP_OUTLIERS


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rac.library()


def _zero_sum_integer_rows(T, d, g, n_big, big, seed):
    """Rows of integers in [-2, 2] built from (v, -v) pairs inside every
    group (so each group mean is exactly 0); in n_big groups of each row one
    pair is (big, -big).  Against a zero reference the residual is the row
    itself, full of ties."""
    rng = np.random.default_rng(seed)
    x = np.zeros((T, d), np.float32)
    for t in range(T):
        big_groups = set(rng.choice(d // g, n_big, replace=False).tolist()) if n_big else set()
        for j in range(d // g):
            v = rng.integers(-2, 3, g // 2).astype(np.float32)
            if j in big_groups:
                v[0] = big
            grp = np.concatenate([v, -v])
            rng.shuffle(grp)
            x[t, j * g:(j + 1) * g] = grp
    return x


def _dyadic_exact_rows(T, d, seed):
    rng = np.random.default_rng(seed)
    r = rng.integers(-32, 33, (T, d)).astype(np.float32) / 4
    x = np.float32(1.25) * r - np.float32(0.5)
    return wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(r)


def _downlink_rows(T, d, seed=0):
    """Downlink inputs whose reference is the oracle's reconstruction of a
    synthetic uplink (the same-round reference of the prefill downlink)."""
    xu, ru, _ = wl.prefill_downlink_uplink(seed, rows=(0, T), tokens=T, hidden=d)
    rc, _, uhat = oracle.encode(xu, ru, **cfgd(T, d, 128, 128, 4, 4))
    assert rc == 0
    ref = wl.f32_to_bf16_bits(uhat)
    return wl.prefill_downlink(ref, seed, rows=(0, T), tokens=T, hidden=d), ref


def _affine(T, d, g, seed=0, **kw):
    x, r, _ = wl.affine_pair(wl.AffineRecipe(T, d, g, **kw), seed)
    return x, r


def _half_integer_rows(T, d, g, with_pair, seed):
    """Rows against a zero reference whose groups hold (v, -v) pairs of
    half-integers below 4 and one (7, -7) pair, so each group's scale is 1
    (b = 4) and most quotients E/s are exact ties of the rounding.  With
    with_pair, one group of each row also holds 24 and -23 (balanced by two
    -0.5), the two largest |E| of the row, neither tied."""
    rng = np.random.default_rng(seed)
    x = np.zeros((T, d), np.float32)
    for t in range(T):
        j0 = int(rng.integers(0, d // g))
        for j in range(d // g):
            v = rng.choice(np.array([0.5, 1.5, 2.5, 3.5], np.float32), g // 2)
            v[0] = 7.0
            grp = np.concatenate([v, -v])
            if with_pair and j == j0:
                grp[1], grp[g // 2 + 1] = 24.0, -23.0
                grp[2], grp[g // 2 + 2] = -0.5, -0.5
            rng.shuffle(grp)
            x[t, j * g:(j + 1) * g] = grp
    return wl.f32_to_bf16_bits(x)


def _scaled(xb, factor):
    """bf16 rows multiplied by a power of two (exact)."""
    return wl.f32_to_bf16_bits(wl.bf16_bits_to_f32(xb) * np.float32(factor))


def _signed_zero_rows(T, d, distinct):
    """x tiny and negative, ref a negative constant: alpha = 0, beta = -0, so
    R~ = -0 and every residual rounds to -0 in fp16; an outlier's
    reconstruction is then -0 while quantized zeros give +0.  With distinct,
    magnitudes grow along the row so the largest ones are not tied."""
    c = np.arange(d)
    mag = (np.float32(2.0) ** -100 * (1 + (c % 128) / 128) * 2.0 ** (c // 128)) if distinct \
        else np.full(d, np.float32(2.0) ** -100)
    x = np.tile(-mag.astype(np.float32), (T, 1))
    return wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(np.full((T, d), -1.0, np.float32))


def _mixed_tie_rows(T, d, g):
    """Even rows from the uplink workload with their references, odd rows
    integer rows full of ties with a zero reference: some wavefronts of a
    launch find their groups' k_g-th largest untied, others do not."""
    x, r, _ = wl.prefill_uplink(5, rows=(0, T))
    xt = wl.f32_to_bf16_bits(_zero_sum_integer_rows(T, d, g, 2, 3.0, 9))
    x, r = x.copy(), r.copy()
    x[1::2], r[1::2] = xt[1::2], 0
    return x, r


CASES = {
    "tiny_64x512_g64_b4": (cfgd(64, 512, 64, 64, 4), lambda: wl.tiny(0)[:2]),
    "uplink_37x4096_g128_b4_k8": (cfgd(37, 4096, 128, 128, 4, 8),
                                  lambda: wl.prefill_uplink(0, rows=(0, 37))[:2]),
    "uplink_21x4096_ga64_gq128_b8_k16": (cfgd(21, 4096, 64, 128, 8, 16),
                                         lambda: wl.prefill_uplink(1, rows=(100, 121))[:2]),
    "downlink_40x3584_g128_b4_k4": (cfgd(40, 3584, 128, 128, 4, 4), lambda: _downlink_rows(40, 3584)),
    "long_29x4096_g64_b3_k16": (cfgd(29, 4096, 64, 64, 3, 16),
                                lambda: wl.long_context(0, rows=(0, 29), group=64)[:2]),
    "long_29x4096_g128_b2_k16": (cfgd(29, 4096, 128, 128, 2, 16),
                                 lambda: wl.long_context(0, rows=(0, 29), group=128)[:2]),
    "long_13x4096_g128_b8_k16": (cfgd(13, 4096, 128, 128, 8, 16),
                                 lambda: wl.long_context(2, rows=(500, 513), group=128)[:2]),
    # Uplink rows with more candidates above the first threshold than the
    # list holds (about a quarter of them at g = 64, k = 16; at k = 32 the
    # threshold from the two largest of each wavefront lane leaves few, and
    # k = 64 ranks a list of 128), whose outliers come from the histogram
    # search
    "overflow_uplink_32x4096_g64_b4_k16": (cfgd(32, 4096, 64, 64, 4, 16),
                                           lambda: wl.prefill_uplink(0, rows=(0, 32))[:2]),
    "overflow_uplink_24x4096_g128_b4_k32": (cfgd(24, 4096, 128, 128, 4, 32),
                                            lambda: wl.prefill_uplink(0, rows=(40, 64))[:2]),
    "overflow_uplink_16x4096_g64_b8_k64": (cfgd(16, 4096, 64, 64, 8, 64),
                                           lambda: wl.prefill_uplink(2, rows=(64, 80))[:2]),
    # k > 16 with ties everywhere: the two-per-lane threshold, then the
    # histogram search
    "ties_heavy_zero_ref_6x4096_g128_k24": (cfgd(6, 4096, 128, 128, 4, 24),
                                            lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 4096, 128, 0, 0.0, 2)), None)),
    "uplink_17x4096_g128_b4_k20": (cfgd(17, 4096, 128, 128, 4, 20), lambda: wl.prefill_uplink(4, rows=(200, 217))[:2]),
    # k > 48: the list of 128 candidates, two per lane; with ties everywhere
    # it overflows into the histogram search
    "ties_heavy_zero_ref_6x4096_g128_k60": (cfgd(6, 4096, 128, 128, 4, 60),
                                            lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 4096, 128, 0, 0.0, 4)), None)),
    "uplink_23x4096_g128_b4_k49": (cfgd(23, 4096, 128, 128, 4, 49), lambda: wl.prefill_uplink(6, rows=(300, 323))[:2]),
    "uplink_19x2048_g128_b4_k64": (cfgd(19, 2048, 128, 128, 4, 64),
                                   lambda: wl.prefill_uplink(7, rows=(0, 19), hidden=2048)[:2]),
    "long_300x4096_g64_b2_k56": (cfgd(300, 4096, 64, 64, 2, 56),
                                 lambda: wl.long_context(3, rows=(1000, 1300), group=64)[:2]),
    # rows of 4097..8192 channels (four chunks per wavefront)
    "wide_uplink_12x8192_g128_b4_k16": (cfgd(12, 8192, 128, 128, 4, 16),
                                        lambda: wl.prefill_uplink(0, rows=(0, 12), hidden=8192)[:2]),
    "wide_overflow_8x8192_g64_b4_k64": (cfgd(8, 8192, 64, 64, 4, 64),
                                        lambda: wl.prefill_uplink(3, rows=(20, 28), hidden=8192)[:2]),
    "wide_partial_chunk_7x4864_g256_b3_k6": (cfgd(7, 4864, 256, 256, 3, 6), lambda: _affine(7, 4864, 256)),
    "partial_chunk_13x2880_ga64_gq32_b4_k5": (cfgd(13, 2880, 64, 32, 4, 5), lambda: _affine(13, 2880, 64)),
    "bytewise3_11x2888_g8_b3_k3": (cfgd(11, 2888, 8, 8, 3, 3), lambda: _affine(11, 2888, 8)),
    "d8192_9x8192_ga128_gq256_b4_k8": (cfgd(9, 8192, 128, 256, 4, 8), lambda: _affine(9, 8192, 128)),
    "large_groups_10x4096_ga1024_gq2048_b4_k8": (cfgd(10, 4096, 1024, 2048, 4, 8),
                                                 lambda: _affine(10, 4096, 1024)),
    "gq_eq_d_16x4096_b4": (cfgd(16, 4096, 128, 4096, 4), lambda: wl.decode_step(16)),
    "mixed_groups_17x4096_ga64_gq128_b4_k0": (cfgd(17, 4096, 64, 128, 4), lambda: wl.prefill_uplink(0, rows=(50, 67))[:2]),
    "mixed_groups_15x4096_ga128_gq64_b2_k0": (cfgd(15, 4096, 128, 64, 2), lambda: wl.prefill_uplink(1, rows=(9, 24))[:2]),
    "mixed_groups_11x8192_ga128_gq64_b4_k8": (cfgd(11, 8192, 128, 64, 4, 8),
                                              lambda: wl.prefill_uplink(2, rows=(0, 11), hidden=8192)[:2]),
    "mixed_groups_group_outliers_9x4096_ga64_gq128_b8_kg2": (cfgd(9, 4096, 64, 128, 8, 2, GRP),
                                                             lambda: wl.prefill_uplink(3, rows=(0, 9))[:2]),
    "all_outliers_12x64_ga8_gq16_k64": (cfgd(12, 64, 8, 16, 4, 64), lambda: _affine(12, 64, 8)),
    "smallest_5x8_b4_k2": (cfgd(5, 8, 8, 8, 4, 2), lambda: _affine(5, 8, 8)),
    "zero_reference_19x1024_b4_k4": (cfgd(19, 1024, 128, 64, 4, 4),
                                     lambda: (_affine(19, 1024, 128)[0], None)),
    "ties_fast_path_9x4096_zero_ref_k8": (cfgd(9, 4096, 128, 128, 4, 8),
                                          lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(9, 4096, 128, 5, 3.0, 0)), None)),
    "ties_slow_path_exact_affine_7x1024_k5": (cfgd(7, 1024, 64, 32, 4, 5), lambda: _dyadic_exact_rows(7, 1024, 3)),
    "ties_heavy_zero_ref_6x512_k12": (cfgd(6, 512, 64, 64, 4, 12),
                                      lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 512, 64, 0, 0.0, 1)), None)),
    "bf16_out_25x4096_g128_b4_k8": (cfgd(25, 4096, 128, 128, 4, 8, rac.RAC_FLAG_XHAT_BF16),
                                    lambda: wl.prefill_uplink(0, rows=(7, 32))[:2]),
    "half_integer_quotients_8x4096_g128_b4_k2": (cfgd(8, 4096, 128, 128, 4, 2),
                                                 lambda: (_half_integer_rows(8, 4096, 128, True, 0), None)),
    "half_integer_quotients_8x4096_g128_b4_k0": (cfgd(8, 4096, 128, 128, 4, 0),
                                                 lambda: (_half_integer_rows(8, 4096, 128, False, 1), None)),
    "saturated_scales_13x4096_g128_b4_k4": (cfgd(13, 4096, 128, 128, 4, 4),
                                            lambda: (_scaled(_affine(13, 4096, 128)[0], 2.0 ** 22), None)),
    "saturated_scales_13x4096_g128_b4_k0": (cfgd(13, 4096, 128, 128, 4, 0),
                                            lambda: (_scaled(_affine(13, 4096, 128)[0], 2.0 ** 22), None)),
    "saturated_scales_ref_7x2048_g64_b8_k6": (cfgd(7, 2048, 64, 64, 8, 6),
                                              lambda: tuple(_scaled(a, 2.0 ** 24) for a in _affine(7, 2048, 64))),
    "signed_zero_outliers_tied_6x1024_g128_b4_k3": (cfgd(6, 1024, 128, 128, 4, 3),
                                                    lambda: _signed_zero_rows(6, 1024, False)),
    "signed_zero_outliers_distinct_6x1024_g128_b4_k3": (cfgd(6, 1024, 128, 128, 4, 3),
                                                        lambda: _signed_zero_rows(6, 1024, True)),
    # per-group outliers (k_g per quantization group, u8 in-group offsets)
    "group_uplink_37x4096_g128_b4_kg1": (cfgd(37, 4096, 128, 128, 4, 1, GRP),
                                         lambda: wl.prefill_uplink(0, rows=(0, 37))[:2]),
    "group_uplink_21x4096_ga64_gq128_b8_kg4": (cfgd(21, 4096, 64, 128, 8, 4, GRP),
                                               lambda: wl.prefill_uplink(1, rows=(100, 121))[:2]),
    "group_long_29x4096_g64_b3_kg2": (cfgd(29, 4096, 64, 64, 3, 2, GRP),
                                      lambda: wl.long_context(0, rows=(0, 29), group=64)[:2]),
    "group_long_13x4096_g128_b2_kg16": (cfgd(13, 4096, 128, 128, 2, 16, GRP),
                                        lambda: wl.long_context(2, rows=(500, 513), group=128)[:2]),
    "group_partial_chunk_7x4864_g256_b2_kg8": (cfgd(7, 4864, 256, 256, 2, 8, GRP), lambda: _affine(7, 4864, 256)),
    "group_g8_partial_chunk_11x2888_b3_kg2": (cfgd(11, 2888, 8, 8, 3, 2, GRP), lambda: _affine(11, 2888, 8)),
    "group_g32_full_lanes_13x2880_ga64_b4_kg8": (cfgd(13, 2880, 64, 32, 4, 8, GRP), lambda: _affine(13, 2880, 64)),
    "group_wide_9x8192_ga128_gq256_b4_kg4": (cfgd(9, 8192, 128, 256, 4, 4, GRP), lambda: _affine(9, 8192, 128)),
    "group_ties_zero_ref_6x512_g64_kg16": (cfgd(6, 512, 64, 64, 4, 16, GRP),
                                           lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 512, 64, 0, 0.0, 1)), None)),
    "group_ties_exact_affine_7x1024_ga64_gq32_kg5": (cfgd(7, 1024, 64, 32, 4, 5, GRP), lambda: _dyadic_exact_rows(7, 1024, 3)),
    "group_bf16_out_25x4096_g128_b4_kg2": (cfgd(25, 4096, 128, 128, 4, 2, GRP | rac.RAC_FLAG_XHAT_BF16),
                                           lambda: wl.prefill_uplink(0, rows=(7, 32))[:2]),
    "group_saturated_scales_13x4096_g128_b4_kg3": (cfgd(13, 4096, 128, 128, 4, 3, GRP),
                                                   lambda: (_scaled(_affine(13, 4096, 128)[0], 2.0 ** 22), None)),
    "group_signed_zero_6x1024_g128_b4_kg3": (cfgd(6, 1024, 128, 128, 4, 3, GRP),
                                             lambda: _signed_zero_rows(6, 1024, False)),
    "group_smallest_5x8_b4_kg2": (cfgd(5, 8, 8, 8, 4, 2, GRP), lambda: _affine(5, 8, 8)),
    # k_g <= 4: the k_g-th largest first, and the round-by-round choice where
    # a tie crosses it (every group here, some rows or some groups there)
    "group_ties_zero_ref_6x4096_g128_kg1": (cfgd(6, 4096, 128, 128, 4, 1, GRP),
                                            lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 4096, 128, 0, 0.0, 3)), None)),
    "group_ties_zero_ref_6x4096_g128_kg4": (cfgd(6, 4096, 128, 128, 4, 4, GRP),
                                            lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 4096, 128, 0, 0.0, 4)), None)),
    "group_tied_pairs_9x4096_g128_kg2": (cfgd(9, 4096, 128, 128, 4, 2, GRP),
                                         lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(9, 4096, 128, 5, 3.0, 5)), None)),
    "group_tied_pairs_9x4096_g128_kg3": (cfgd(9, 4096, 128, 128, 4, 3, GRP),
                                         lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(9, 4096, 128, 5, 3.0, 6)), None)),
    "group_mixed_tie_rows_16x4096_g128_kg4": (cfgd(16, 4096, 128, 128, 4, 4, GRP), lambda: _mixed_tie_rows(16, 4096, 128)),
    "group_mixed_tie_rows_16x4096_g128_kg1": (cfgd(16, 4096, 128, 128, 4, 1, GRP), lambda: _mixed_tie_rows(16, 4096, 128)),
    "group_ties_g256_4x4096_kg4": (cfgd(4, 4096, 256, 256, 4, 4, GRP),
                                   lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(4, 4096, 256, 3, 5.0, 7)), None)),
    "group_g256_9x8192_kg3": (cfgd(9, 8192, 128, 256, 4, 3, GRP), lambda: _affine(9, 8192, 128, seed=2)),
    "group_ties_g8_6x1024_kg2": (cfgd(6, 1024, 8, 8, 4, 2, GRP),
                                 lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 1024, 8, 0, 0.0, 8)), None)),
    "group_g16_11x2880_ga64_b4_kg3": (cfgd(11, 2880, 64, 16, 4, 3, GRP), lambda: _affine(11, 2880, 64, seed=3)),
    "group_g32_13x2880_ga64_b4_kg4": (cfgd(13, 2880, 64, 32, 4, 4, GRP), lambda: _affine(13, 2880, 64, seed=4)),
    # ties at the largest k_g of each lane-block width (2, 4 and 32 lanes per
    # group): every round of the choice meets several lanes holding the maximum
    "group_ties_g16_8x2048_ga64_kg4": (cfgd(8, 2048, 64, 16, 4, 4, GRP),
                                       lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(8, 2048, 16, 9, 3.0, 10)), None)),
    "group_ties_g32_6x2048_ga64_kg8": (cfgd(6, 2048, 64, 32, 4, 8, GRP),
                                       lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(6, 2048, 32, 7, 4.0, 11)), None)),
    "group_ties_g256_4x4096_kg16": (cfgd(4, 4096, 256, 256, 4, 16, GRP),
                                    lambda: (wl.f32_to_bf16_bits(_zero_sum_integer_rows(4, 4096, 256, 3, 5.0, 12)), None)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_small_parity(name):
    c, gen = CASES[name]
    xb, rb = gen()
    say(f"[gpu] {name}: T={c['tokens']} d={c['hidden']} ga={c['group_align']} gq={c['group_quant']} "
        f"b={c['bits']} k={c['outlier_k']} flags={c['flags']}")
    ow, ox = oracle_run(c, xb, rb)
    gw, gx, gd, gr = gpu_run(c, xb, rb)
    assert_parity(c, gw, gx, ow, ox)
    # sender reconstruction == receiver decode == standalone reconstruct, bitwise
    assert np.array_equal(gx.view(np.uint8), gd.view(np.uint8))
    assert np.array_equal(gx.view(np.uint8), gr.view(np.uint8))


def _fixed_steps(d, g, seed=1):
    """Calibrated steps of the tiny workload: 2 std(E) / (2^4 - 1) per channel
    group, from the oracle's residuals on a separate seed."""
    xb, rb, _ = wl.tiny(seed)
    rc, wire, _ = oracle.encode(xb, rb, want_xhat=False, **cfgd(64, d, g, g, 4))
    s = wirefmt.sections(wire)
    a = np.repeat(s["coef"][..., 0].view(np.float16).astype(np.float32), g, axis=1)
    b = np.repeat(s["coef"][..., 1].view(np.float16).astype(np.float32), g, axis=1)
    e = wl.bf16_bits_to_f32(xb) - (a * wl.bf16_bits_to_f32(rb) + b)
    return (2 * e.reshape(64, d // g, g).transpose(1, 0, 2).reshape(d // g, -1).std(axis=1)
            / 15).astype(np.float32)


def test_fixed_step_tiny():
    c = cfgd(64, 512, 64, 64, 4, 0, rac.RAC_FLAG_FIXED_STEP)
    steps = _fixed_steps(512, 64)
    xb, rb, _ = wl.tiny(0)
    say(f"[gpu] fixed step tiny: steps[:3]={steps[:3]}")
    rc, ow, ox = oracle.encode(xb, rb, steps, **c)
    assert rc == 0
    gw, gx, gd, gr = gpu_run(c, xb, rb, steps)
    assert_parity(c, gw, gx, ow, ox)
    assert np.array_equal(gx, gd) and np.array_equal(gx, gr)


def test_fixed_step_tiny_with_group_outliers():
    c = cfgd(64, 512, 64, 64, 4, 2, rac.RAC_FLAG_FIXED_STEP | GRP)
    steps = _fixed_steps(512, 64)
    xb, rb, _ = wl.tiny(0)
    say("[gpu] fixed step tiny, two outliers per group")
    rc, ow, ox = oracle.encode(xb, rb, steps, **c)
    assert rc == 0
    gw, gx, gd, gr = gpu_run(c, xb, rb, steps)
    assert_parity(c, gw, gx, ow, ox)
    assert np.array_equal(gx, gd) and np.array_equal(gx, gr)


@pytest.mark.parametrize("batch", [1, 16, 64, 256])
@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("gq", [128, 4096])
def test_decode_step_batches(batch, bits, gq):
    c = cfgd(batch, 4096, 128, gq, bits)
    xb, rb = wl.decode_step(batch)
    say(f"[gpu] decode step B={batch} b={bits} gq={gq}")
    ow, ox = oracle_run(c, xb, rb)
    gw, gx, gd, _ = gpu_run(c, xb, rb)
    assert_parity(c, gw, gx, ow, ox)
    assert np.array_equal(gx, gd)


def test_empty_token_batch_writes_header_only():
    c = cfgd(0, 512, 64, 64, 4, 2)
    xb = np.zeros((0, 512), np.uint16)
    for ref in (None, xb):
        gw, gx, gd, _ = gpu_run(c, xb, ref)
        ow, _ = oracle_run(c, xb, None)  # an empty device tensor has no address: zero reference
        assert gw.size == 256 and np.array_equal(gw, ow)


def test_without_xhat_and_on_a_side_stream_deterministic():
    import torch
    c = cfgd(33, 4096, 128, 128, 4, 8)
    xb, rb, _ = wl.prefill_uplink(5, rows=(0, 33))
    s = torch.cuda.Stream()
    say("[gpu] side stream, no xhat, twice")
    w1, _, d1, _ = gpu_run(c, xb, rb, stream=s, want_xhat=False)
    w2, _, d2, _ = gpu_run(c, xb, rb, stream=s, want_xhat=False, garbage=0x11)
    assert np.array_equal(w1, w2) and np.array_equal(d1, d2)
    ow, ox = oracle_run(c, xb, rb)
    assert_parity(c, w1, d1, ow, ox)


def test_graph_capture_replays_match_eager():
    """Encode + decode of decode-phase batches captured in one HIP graph and
    replayed three times, with other eager calls and synchronizations between
    the replays: every replay rewrites (over poisoned buffers) exactly the
    eager wire and reconstructions, which match the oracle."""
    import torch
    from tests.gpu_util import to_dev
    for k in (0, 4):
        c = cfgd(16, 4096, 128, 128, 4, k)
        cfg = rac.RacConfig(**c)
        xb, rb = wl.decode_step(16)
        say(f"[gpu] graph capture B=16 k={k}")
        x, ref = to_dev(xb), to_dev(rb)
        size = rac.rac_wire_size(cfg)
        wire = torch.empty(size, dtype=torch.uint8, device="cuda")
        xh = torch.empty(16, 4096, dtype=torch.float32, device="cuda")
        xd = torch.empty_like(xh)
        rac.rac_encode(cfg, x, ref, None, wire, xh)
        rac.rac_decode(cfg, wire, ref, None, xd)
        torch.cuda.synchronize()
        eager = [t.clone() for t in (wire, xh, xd)]
        ow, ox = oracle_run(c, xb, rb)
        assert_parity(c, eager[0].cpu().numpy(), eager[1].cpu().numpy(), ow, ox)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            rac.rac_encode(cfg, x, ref, None, wire, xh)
            rac.rac_decode(cfg, wire, ref, None, xd)
        # other work on the same buffers between replays
        w2 = torch.empty_like(wire)
        for rep in range(3):
            for t in (wire, xh, xd):
                t.view(torch.uint8).fill_(0x5A)
            rac.rac_encode(cfg, x, x, None, w2, None)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for t, e in zip((wire, xh, xd), eager):
                assert torch.equal(t, e), f"replay {rep} differs from the eager result"


# ---------------------------------------------------------------------------
# Full benchmark shapes, sampled rows

def _sample(T, n, seed=0):
    rng = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([[0, 1, 2, 3, T - 2, T - 1], rng.choice(T, n, replace=False)]))
    return rows


def test_full_prefill_uplink_4096x4096_sampled():
    c = cfgd(4096, 4096, 128, 128, 4, 8)
    say("[gpu] full prefill uplink 4096x4096: generating")
    xb, rb, _ = wl.prefill_uplink(0)
    gw, gx, gd, _ = gpu_run(c, xb, rb)
    assert np.array_equal(gx, gd)
    rows = _sample(4096, 48)
    ow, ox = oracle_run(dict(c, tokens=rows.size), xb[rows], rb[rows])
    n = assert_parity(c, gw, gx, ow, ox, g_rows=rows, o_rows=slice(None))
    assert n == rows.size
    assert wirefmt.padding_is_zero(gw) and wirefmt.header(gw)["tokens"] == 4096


def test_full_prefill_uplink_4096x4096_k64_sampled():
    """k = 64 at the uplink's full size: the list of 128 candidates ranked two
    per lane, on the strided grid."""
    c = cfgd(4096, 4096, 128, 128, 4, 64)
    say("[gpu] full prefill uplink 4096x4096, k = 64: generating")
    xb, rb, _ = wl.prefill_uplink(0)
    gw, gx, gd, _ = gpu_run(c, xb, rb)
    assert np.array_equal(gx, gd)
    rows = _sample(4096, 48, seed=3)
    ow, ox = oracle_run(dict(c, tokens=rows.size), xb[rows], rb[rows])
    assert_parity(c, gw, gx, ow, ox, g_rows=rows, o_rows=slice(None))


def test_full_prefill_uplink_4096x4096_group_outliers_sampled():
    c = cfgd(4096, 4096, 128, 128, 4, 1, GRP)
    say("[gpu] full prefill uplink 4096x4096, one outlier per group: generating")
    xb, rb, _ = wl.prefill_uplink(0)
    gw, gx, gd, _ = gpu_run(c, xb, rb)
    assert np.array_equal(gx, gd)
    rows = _sample(4096, 48, seed=3)
    ow, ox = oracle_run(dict(c, tokens=rows.size), xb[rows], rb[rows])
    assert_parity(c, gw, gx, ow, ox, g_rows=rows, o_rows=slice(None))
    assert wirefmt.padding_is_zero(gw) and wirefmt.header(gw)["off_ooff"] > 0


def test_full_long_context_32768x4096_g128_b4_sampled():
    c = cfgd(32768, 4096, 128, 128, 4, 16)
    say("[gpu] full long context 32768x4096: generating")
    xb, rb, _ = wl.long_context(0, group=128)
    gw, gx, gd, _ = gpu_run(c, xb, rb)
    assert np.array_equal(gx, gd)
    rows = _sample(32768, 40, seed=1)
    ow, ox = oracle_run(dict(c, tokens=rows.size), xb[rows], rb[rows])
    assert_parity(c, gw, gx, ow, ox, g_rows=rows, o_rows=slice(None))
    h = wirefmt.header(gw)
    assert h["tokens"] == 32768 and wirefmt.padding_is_zero(gw)


def test_full_prefill_downlink_65536x3584_sampled():
    """The same-round reference: the GPU reconstructs the uplink of all rows;
    on the sampled rows the oracle reconstructs it too (asserted equal) and
    encodes the downlink from its own reference."""
    import torch
    T, d = 65536, 3584
    cu = cfgd(T, d, 128, 128, 4, 4)
    say("[gpu] full downlink 65536x3584: uplink generation")
    xu, ru, _ = wl.prefill_downlink_uplink(0)
    uw, uhat, _, _ = gpu_run(cu, xu, ru)
    ref = wl.f32_to_bf16_bits(uhat)
    del uw, uhat
    say("[gpu] full downlink: downlink generation")
    xd = wl.prefill_downlink(ref, 0)
    gw, gx, gd, _ = gpu_run(cu, xd, ref)
    assert np.array_equal(gx, gd)
    rows = _sample(T, 32, seed=2)
    rc, _, uhat_o = oracle.encode(xu[rows], ru[rows], **dict(cu, tokens=rows.size))
    ref_o = wl.f32_to_bf16_bits(uhat_o)
    assert np.array_equal(ref_o, ref[rows]), "uplink reconstruction differs from the oracle"
    xd_o = wl.prefill_downlink(ref_o, 0, rows=rows)
    assert np.array_equal(xd_o, xd[rows])
    ow, ox = oracle_run(dict(cu, tokens=rows.size), xd_o, ref_o)
    assert_parity(cu, gw, gx, ow, ox, g_rows=rows, o_rows=slice(None))
    torch.cuda.empty_cache()
