"""Mutation check of the oracle's pins.

Each case plants one plausible mistake in a temporary copy of the oracle
source (on the CPU), builds it with gcc, and runs the pin tests against that
build: at least one pin must fail.  This is what makes the pins a check of the
oracle rather than a restatement of it.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

import oracle
from tests import test_oracle_group_outliers as gpins
from tests import test_oracle_pooled as ppins
from tests import test_oracle_pins as pins
from tests import test_oracle_saturation as spins

# (name, text in rac_oracle.c, replacement)
MUTANTS = [
    ("beta_sign", "*beta_star = mx - a * mr;", "*beta_star = mx + a * mr;"),
    ("uncentred_fit", "const float u = r[c] - mr;", "const float u = r[c];"),
    ("transposed_alpha", "const float a = crx / crr;", "const float a = crr / crx;"),
    ("zero_variance_beta", "*beta_star = mx;\n", "*beta_star = 0.0f;\n"),
    ("scale_round_down", "    return (uint16_t)lo;\n}\n\nuint16_t orc_step_roundup",
     "    return (uint16_t)(lo - 1);\n}\n\nuint16_t orc_step_roundup"),
    ("half_away_from_zero", "float rq = rintf(tq);", "float rq = roundf(tq);"),
    ("qmax_off_by_one", "const int32_t qmax = (1 << (bits - 1)) - 1;",
     "const int32_t qmax = (1 << (bits - 1));"),
    ("msb_first_packing", "row[pos / 8] |= (uint8_t)(1u << (pos % 8));",
     "row[pos / 8] |= (uint8_t)(1u << (7 - pos % 8));"),
    ("outlier_ties_to_higher", "return (a->idx < b->idx) ? -1 : (a->idx > b->idx);",
     "return (a->idx > b->idx) ? -1 : (a->idx < b->idx);"),
    ("outlier_left_in_dense", "is_out[c] = 1;\n                ed[c] = 0.0f;\n", "is_out[c] = 1;\n"),
    ("aligned_ref_drops_beta", "                rt[c] = fmaf(a, r[c], b0);", "                rt[c] = a * r[c];"),
    ("decoder_drops_outliers", "eh[c] = orc_f16_wire((uint16_t)(w >> 16));", "(void)c;"),
    ("alpha_beta_swapped", "put16(coef + 4 * j, ah);", "put16(coef + 4 * j, bh);"),
    ("outlier_value_unrounded_recon", "? orc_f16_wire(oval[c]) :", "? e[c] :"),
    ("f16_ties_up", "p = (lo & 1u) ? lo + 1 : lo; /* tie: even fraction */",
     "p = lo + 1; /* tie: even fraction */"),
    ("group_offset_absolute", "orow[(uint64_t)g * k + i] = (uint8_t)sel[i];",
     "orow[(uint64_t)g * k + i] = (uint8_t)c;"),
    ("group_selects_from_first_group", "orc_topk_row(e + g * gq, gq, k, sel);",
     "orc_topk_row(e, gq, k, sel);"),
    ("group_outlier_left_in_dense", "is_out[c] = 1;\n                    ed[c] = 0.0f;\n",
     "is_out[c] = 1;\n"),
    ("group_decoder_ignores_group", "eh[g * gq + (int32_t)o] =", "eh[(int32_t)o] ="),
    ("pool_drops_between_term", "m.crr = (a->crr + b->crr) + (dr * dr) * w;", "m.crr = a->crr + b->crr;"),
    ("pool_weight_of_wrong_side", "const float fb = b->n / n;", "const float fb = a->n / n;"),
    ("pool_crx_uses_dr_twice", "m.crx = (a->crx + b->crx) + (dr * dx) * w;",
     "m.crx = (a->crx + b->crx) + (dr * dr) * w;"),
    ("pool_repeats_the_first_row", "seg[i] = mom[(lo + i) * G + j];", "seg[i] = mom[lo * G + j];"),
    ("group_values_in_reverse", "put16(vrow + 2 * ((uint64_t)g * k + i), oval[c]);",
     "put16(vrow + 2 * ((uint64_t)g * k + (k - 1 - i)), oval[c]);"),
    ("wire_fields_clamped_not_infinite", "    if (fabsf(f) >= ORC_F16_OVERFLOW) return (uint16_t)((signbit(f) ? 0x8000u : 0u) | ORC_F16_INF_BITS);",
     "    if (fabsf(f) >= ORC_F16_OVERFLOW) return (uint16_t)((signbit(f) ? 0x8000u : 0u) | ORC_F16_MAX_BITS);"),
    ("overflow_threshold_at_the_largest_fp16", "#define ORC_F16_OVERFLOW 65520.0f", "#define ORC_F16_OVERFLOW 65504.0f"),
    ("scale_past_range_clamped", "    if (orc_f16_to_f32(ORC_F16_MAX_BITS) * q < m) return ORC_F16_INF_BITS;",
     "    if (orc_f16_to_f32(ORC_F16_MAX_BITS) * q < m) return ORC_F16_MAX_BITS;"),
    ("infinity_used_unclamped", "    return v > m ? m : (v < -m ? -m : v);", "    return v;"),
]

PINS = [
    pins.test_f16_rne_matches_numpy_including_ties_and_subnormals,
    lambda: pins.test_scale_roundup_is_smallest_fp16_covering_the_max(7),
    lambda: pins.test_fit_matches_exact_rational_least_squares(16),
    pins.test_fit_zero_variance_reference_gives_alpha_zero_beta_mean,
    pins.test_topk_matches_brute_force_with_ties,
    pins.test_hand_worked_example_bit_exact,
    lambda: pins.test_pack_known_answers_via_zero_reference(4, [1, -1, 7, -7, 0, 0, 0, 0], "f1970000"),
    pins.test_quantizer_rounds_half_to_even,
    pins.test_exact_affine_rows_give_zero_codes_and_exact_reconstruction,
    pins.test_zero_reference_is_textbook_grouped_absmax_quantization,
    lambda: pins.test_error_bound_and_equivalence_on_uplink_rows(4, 8),
    pins.test_sender_reconstruction_equals_receiver_decode_bitwise,
    lambda: gpins.test_group_outliers_match_brute_force_on_uplink_rows(128, 2, 4),
    gpins.test_group_outliers_ties_go_to_the_lower_offset,
    lambda: gpins.test_group_mode_sender_equals_receiver_bitwise(0),
    lambda: ppins.test_pooled_fit_matches_exact_rational_least_squares(0),
    ppins.test_pooled_moments_match_float64,
    ppins.test_constant_reference_over_a_segment_gives_alpha_zero_and_the_pooled_mean,
    spins.test_ordinary_rows_have_no_marks,
    spins.test_scale_past_the_range_is_infinity_and_the_codes_clip,
    spins.test_beta_overflow_threshold_is_the_fp16_rounding_overflow,
    spins.test_alpha_overflow_is_infinity_with_its_sign,
    spins.test_outlier_value_overflow_is_infinity_and_reconstructs_as_65504,
    spins.test_pooled_fit_marks_every_row_of_a_saturated_segment,
    pins.test_f16_rne_is_the_ieee_conversion_with_overflow_to_infinity,
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(tmp_path, name, old, new):
    src = open(oracle._SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    shutil.copy(os.path.join(os.path.dirname(oracle._SRC), "rac_oracle.h"), tmp_path)
    (tmp_path / "m.c").write_text(src.replace(old, new))
    so = str(tmp_path / "libm.so")
    subprocess.run(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-o", so,
                    str(tmp_path / "m.c"), "-lm"], check=True)
    caught = []
    with oracle.swapped_library(so):
        for pin in PINS:
            try:
                pin()
            except AssertionError:
                caught.append(getattr(pin, "__name__", "lambda"))
    assert caught, f"no pin caught mutant {name}"
