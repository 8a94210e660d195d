"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake into a copy of the oracle's C source (on the CPU,
in a temporary directory), builds it, and runs the pin checks of
``test_oracle_pins`` against the mutated build: at least one check must fail.
"""
import importlib.util
import os
import shutil

import pytest

import tests.test_oracle_backward_pins as bpins
import tests.test_oracle_bits_pins as kpins
import tests.test_oracle_convert_pins as cpins
import tests.test_oracle_layer_pins as lpins
import tests.test_oracle_pins as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

MUTATIONS = {
    "truncate_instead_of_floor": ("q -= 1;                   /* move truncation down to the floor */",
                                  "q -= 0;"),
    "negate_then_shift": ("int64_t t = floor_div_pow2((int64_t)x, shift);",
                          "int64_t t = floor_div_pow2(negative ? -(int64_t)x : (int64_t)x, shift);"
                          " if (negative) return t;"),
    "zero_code_as_shift_15": ("if (shift == 15)\n        return 0;", "if (shift == 99)\n        return 0;"),
    "sign_ignored": ("return negative ? -t : t;", "return t;"),
    "conv_bias_dropped": ("int64_t acc = bias ? (int64_t)bias[k] : 0;\n    for (int64_t c = 0; c < C; ++c)\n        for (int64_t r",
                          "int64_t acc = 0;\n    for (int64_t c = 0; c < C; ++c)\n        for (int64_t r"),
    "kernel_r_s_transposed": ("uint8_t code = codes[((k * C + c) * R + r) * S + s];",
                              "uint8_t code = codes[((k * C + c) * S + s) * R + r];"),
    "input_h_w_transposed": ("int32_t xv = x[((n * C + c) * H + ih) * W + iw];",
                             "int32_t xv = x[((n * C + c) * W + iw) * H + ih];"),
    "stride_h_w_swapped": ("int64_t ih = oh * sh - ph + r;", "int64_t ih = oh * sw - ph + r;"),
    "pad_off_by_one": ("int64_t iw = ow * sw - pw + s;\n                if", "int64_t iw = ow * sw - pw + s + 1;\n                if"),
    "saturate_instead_of_wrap": ("uint32_t u = (uint32_t)(uint64_t)v;\n    return (int32_t)u;",
                                 "return v > 2147483647 ? 2147483647 : (v < -2147483647 - 1 ? -2147483647 - 1 : (int32_t)v);"),
    "linear_codes_transposed": ("acc += oracle_term(x[b * in + i], codes[o * in + i]);",
                                "acc += oracle_term(x[b * in + i], codes[(i * out + o) % (in * out)]);"),
    "pack_pad_with_zero": ("col < cols ? codes[r * cols + col] : 15u;", "col < cols ? codes[r * cols + col] : 0u;"),
    "pack_bit_offset": ("word |= (code & 31u) << (5 * j);", "word |= (code & 31u) << (5 * (5 - j));"),
    "drop_last_term": ("for (int64_t s = 0; s < S; ++s) {\n                int64_t ih",
                       "for (int64_t s = 0; s < S - (c == C - 1 && r == R - 1); ++s) {\n                int64_t ih"),
    # float -> code converter and fixed point
    "q_floor_instead_of_round": ("return (w2 >= ldexp(1.0, 2 * p + 1)) ? p + 1 : p;", "return p;"),
    "q_boundary_one_off": ("ldexp(1.0, 2 * p + 1)", "ldexp(1.0, 2 * p + 2)"),
    "q_sign_dropped": ("return (uint8_t)((s < 0 ? 16 : 0) | (-p));", "return (uint8_t)(-p);"),
    "clip_below_to_zero_code": ("if (p < -max_shift) p = -max_shift;", "if (p < -max_shift) return 15;"),
    "clip_range_ignored": ("if (p < -max_shift) p = -max_shift;", "if (p < -14) p = -14;"),
    "zero_weight_as_shift_0": ("if (s == 0) return 15;", "if (s == 0) return 0;"),
    "ps_strict_threshold": ("int s = sv <= -0.5f ? -1 : (sv >= 0.5f ? 1 : 0);",
                            "int s = sv < -0.5f ? -1 : (sv > 0.5f ? 1 : 0);"),
    "ps_round_half_even": ("const double r = round((double)P[i]);", "const double r = nearbyint((double)P[i]);"),
    "fixed_truncate": ("const double t = round(ldexp(v, frac_bits));", "const double t = trunc(ldexp(v, frac_bits));"),
    "fixed_half_even": ("const double t = round(ldexp(v, frac_bits));", "const double t = nearbyint(ldexp(v, frac_bits));"),
    "fixed_no_saturation": ("if (t >= 2147483647.0) out[i] = 2147483647;", "if (0) out[i] = 0;"),
    # layers for chained inference
    "epilogue_truncating_shift": ("v = floor_div_pow2_64(v * (int64_t)mul[k], mul_shift);",
                                  "v = (v * (int64_t)mul[k]) / ((int64_t)1 << mul_shift);"),
    "epilogue_relu_before_residual": ("if (residual)\n                    v = wrap32(v + (int64_t)residual[i]);\n                if (relu && v < 0)\n                    v = 0;",
                                      "if (relu && v < 0)\n                    v = 0;\n                if (residual)\n                    v = wrap32(v + (int64_t)residual[i]);"),
    "epilogue_add_dropped": ("v = wrap32(v + (add ? (int64_t)add[k] : 0));", "v = wrap32(v);"),
    "maxpool_padding_as_zero": ("if (ih < 0 || ih >= H || iw < 0 || iw >= W)\n                                continue;\n                            int64_t v = x[",
                                "int64_t v = (ih < 0 || ih >= H || iw < 0 || iw >= W) ? 0 : x["),
    "avgpool_truncates": ("if (sum % HW != 0 && sum < 0)\n            q -= 1;", ""),
    # input gradients
    "bwd_window_not_rotated": ("int64_t ih = oh * sh - ph + r, iw = ow * sw - pw + s;\n                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)\n                                    continue;  /* the forward pass read padding here */",
                               "int64_t ih = oh * sh - ph + (R - 1 - r), iw = ow * sw - pw + (S - 1 - s);\n                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)\n                                    continue;  /* the forward pass read padding here */"),
    "bwd_channels_transposed": ("oracle_term(g, codes[((k * C + c) * R + r) * S + s]);",
                                "oracle_term(g, codes[(((c * K + k) % (K * C)) * R + r) * S + s]);"),
    "bwd_stride_ignored": ("int64_t ih = oh * sh - ph + r, iw = ow * sw - pw + s;\n                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)\n                                    continue;  /* the forward pass read padding here */",
                           "int64_t ih = oh - ph + r, iw = ow - pw + s;\n                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)\n                                    continue;  /* the forward pass read padding here */"),
    "bwd_pad_sign": ("int64_t ih = oh * sh - ph + r, iw = ow * sw - pw + s;\n                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)\n                                    continue;  /* the forward pass read padding here */",
                     "int64_t ih = oh * sh + ph - r, iw = ow * sw + pw - s;\n                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)\n                                    continue;  /* the forward pass read padding here */"),
    "bwd_last_output_row_dropped": ("for (int64_t oh = 0; oh < OH; ++oh)\n                    for (int64_t ow = 0; ow < OW; ++ow) {\n                        int32_t g",
                                    "for (int64_t oh = 0; oh < OH - 1; ++oh)\n                    for (int64_t ow = 0; ow < OW; ++ow) {\n                        int32_t g"),
    "bwd_linear_codes_not_transposed": ("acc += oracle_term(dy[b * out + o], codes[o * in + i]);",
                                        "acc += oracle_term(dy[b * out + o], codes[(i * out + o) % (in * out)]);"),
    # b-bit packed codes
    "bits_padding_as_plus_one": ("uint32_t field = ones, sign = 0;", "uint32_t field = 0, sign = 0;"),
    "bits_sign_one_too_high": ("word |= ((sign << (bits - 1)) | field) << (bits * j);",
                               "word |= ((sign << bits) | field) << (bits * j);"),
    "bits_codes_per_word_off": ("int64_t per = 32 / bits, wpr = (cols + per - 1) / per;\n    uint32_t ones = (1u << (bits - 1)) - 1u;\n    for (int64_t i",
                                "int64_t per = 32 / bits - (bits == 3), wpr = (cols + per - 1) / per;\n    uint32_t ones = (1u << (bits - 1)) - 1u;\n    for (int64_t i"),
    "bits_range_check_off_by_one": ("if (shift != 15u && shift >= ones)", "if (shift != 15u && shift > ones)"),
    "bwd_points_divisibility_ignored": ("if (a < 0 || a % sh != 0 || a / sh >= OH)", "if (a < 0 || a / sh >= OH)"),
}

LAYER_CHECKS = [
    *[(lpins.test_epilogue_affine_matches_numpy_shift, (m,)) for m in (5, 16)],
    (lpins.test_epilogue_residual_then_relu_order, ()),
    (lpins.test_epilogue_wraps_residual_sum, ()),
    *[(lpins.test_maxpool_matches_torch, (sh,)) for sh in ((2, 3, 9, 9, 3, 2, 1), (1, 4, 8, 7, 3, 2, 1))],
    (lpins.test_avgpool_global_matches_numpy, ()),
]

CONVERT_CHECKS = [
    *[(cpins.test_q_matches_library_log2_round, (m,)) for m in (14, 3)],
    (cpins.test_q_boundary_neighbours_round_up_and_down, ()),
    (cpins.test_q_nearest_power_property_exact, ()),
    (cpins.test_q_special_values, ()),
    (cpins.test_ps_sign_threshold_equals_sign_of_round, ()),
    (cpins.test_ps_round_p_halves_away_and_clips, ()),
    (cpins.test_ps_nan_gives_zero_weight, ()),
    *[(cpins.test_fixed_matches_exact_rounding, (f,)) for f in (16, 31)],
    (cpins.test_golden_examples, ()),
]

BITS_CHECKS = [
    *[(kpins.test_pack_matches_bitstream, (b,)) for b in kpins.BITS],
    (kpins.test_pack_literal_words, ()),
    *[(kpins.test_round_trip_and_range, (b,)) for b in kpins.BITS],
]

BACKWARD_CHECKS = [
    *[(bpins.test_closed_form_matches_torch_input_gradient, (s,)) for s in bpins.SHAPES],
    (bpins.test_linear_closed_form_matches_matmul, ()),
    (bpins.test_bruteforce_tiny, (0,)),
    (bpins.test_linear_equals_forward_with_transposed_codes, ()),
    (bpins.test_points_agree_with_full, ()),
]

CHECKS = [
    (pins.test_term_matches_exact_rational_floor, ()),
    (pins.test_term_reading_examples, ()),
    (pins.test_conv_bruteforce_tiny, (0,)),
    (pins.test_linear_bruteforce_tiny, ()),
    *[(pins.test_conv_closed_form_exact_shifts, (s,)) for s in pins.CLOSED_SHAPES],
    (pins.test_linear_closed_form_exact_shifts, ()),
    (pins.test_single_term_equals_numpy_right_shift, ()),
    *[(pins.test_one_sided_rounding_bound, (p,)) for p in ("pos", "neg", "mixed")],
    (pins.test_zero_codes_contribute_nothing, ()),
    (pins.test_sign_flip_negates_sum, ()),
    (pins.test_linear_equals_1x1_conv, ()),
    (pins.test_wraparound_extremes, ()),
    (pins.test_pack_layout_bitstream, ()),
    (pins.test_pack_literal_words, ()),
]


def load_mutant(tmp_path, name):
    old, new = MUTATIONS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site for {name} not unique"
    d = tmp_path / name
    d.mkdir()
    src = d / "oracle.c"
    src.write_text(text.replace(old, new))
    shutil.copy(os.path.join(ROOT, "oracle", "__init__.py"), d / "__init__.py")
    spec = importlib.util.spec_from_file_location(f"oracle_{name}", d / "__init__.py")
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod.build(force=True)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(tmp_path, monkeypatch, name):
    mod = load_mutant(tmp_path, name)
    monkeypatch.setattr(pins, "oracle", mod)
    monkeypatch.setattr(cpins, "oracle", mod)
    monkeypatch.setattr(lpins, "oracle", mod)
    monkeypatch.setattr(bpins, "oracle", mod)
    monkeypatch.setattr(kpins, "oracle", mod)
    failed = []
    for fn, args in CHECKS + CONVERT_CHECKS + LAYER_CHECKS + BACKWARD_CHECKS + BITS_CHECKS:
        try:
            fn(*args)
        except AssertionError:
            failed.append(fn.__name__)
    assert failed, f"no pin caught the mutation {name}"


def test_unmutated_copy_passes(tmp_path, monkeypatch):
    d = tmp_path / "clean"
    d.mkdir()
    shutil.copy(SRC, d / "oracle.c")
    shutil.copy(os.path.join(ROOT, "oracle", "__init__.py"), d / "__init__.py")
    spec = importlib.util.spec_from_file_location("oracle_clean", d / "__init__.py")
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod.build(force=True)
    monkeypatch.setattr(pins, "oracle", mod)
    monkeypatch.setattr(cpins, "oracle", mod)
    monkeypatch.setattr(lpins, "oracle", mod)
    monkeypatch.setattr(bpins, "oracle", mod)
    monkeypatch.setattr(kpins, "oracle", mod)
    for fn, args in CHECKS + CONVERT_CHECKS + LAYER_CHECKS + BACKWARD_CHECKS + BITS_CHECKS:
        fn(*args)
