"""The FlashSCA oracle's pins catch plausible mistakes.

Each mutant is a copy of flashsca_oracle.c with one plausible mistake
planted (a wrong anchor of a point, a dropped half-pixel, swapped offset
components, a missing softmax, a wrong level start, a wrong mask
convention ...).  It is compiled on the CPU, together with the unmodified
Eq. 1 oracle, into a temporary library and run through the pins; every
mutant must fail at least one of them.
"""
import ctypes
import subprocess

import pytest

import oracle
import test_oracle_sca_backward_pins as bpins
import test_oracle_sca_pins as pins
from oracle import build as obuild

MUTANTS = {
    "anchor_of_point_by_group": ("return k % Z;", "return k / (P / Z);"),
    "only_valid_anchors_hit_all": ("hit[n] |= reference_point(", "hit[n] = reference_point("),
    "depth_not_clamped": ("float dd = in_front ? d : p->depth_eps;", "float dd = d;"),
    "closed_image_interval": ("*un > 0.0f && *un < 1.0f", "*un >= 0.0f && *un <= 1.0f"),
    "mean_over_all_cameras": ("? (double)count : 1.0;", "? (double)p->N : 1.0;"),
    "no_softmax_normalization": ("attn[h * L * P + t] /= sum;", "attn[h * L * P + t] /= 1.0;"),
    "no_half_pixel": ("const float xim = sx - 0.5f;", "const float xim = sx;"),
    "offset_components_swapped": ("sx = sx + o[0];\n    sy = sy + o[1];",
                                  "sx = sx + o[1];\n    sy = sy + o[0];"),
    "level_start_not_advanced": ("                start += (int64_t)p->level_h[l] * p->level_w[l];\n            }\n        }\n    }\n    /* 4.",
                                 "                start += 0;\n            }\n        }\n    }\n    /* 4."),
    "value_rows_transposed": ("start + (int64_t)yt * Wl + xt", "start + (int64_t)xt * Hl + yt"),
    "head_channel_offset_dropped": ("const float *row = vcam + (size_t)cr.pix[t] * C + (size_t)h * D;",
                                    "const float *row = vcam + (size_t)cr.pix[t] * C + (size_t)0 * D;"),
    "bwd_value_head_offset_dropped": ("double *dst = gv + (size_t)cr.pix[c4] * C + (size_t)h * D;",
                                      "double *dst = gv + (size_t)cr.pix[c4] * C + (size_t)0 * D;"),
    "x_weights_swapped": ("(tx ? ax : 1.0 - ax)", "(tx ? 1.0 - ax : ax)"),
    "attention_of_head_zero": ("const double a = attn[(h * L + l) * P + k];",
                               "const double a = attn[(0 * L + l) * P + k];"),
    "offsets_of_first_query": ("offsets + ((size_t)b * Q + q) * H * L * P * 2;",
                               "offsets + ((size_t)b * Q + 0) * H * L * P * 2;"),
    "level_width_for_height": ("float sy = vn * (float)Hl;", "float sy = vn * (float)Wl;"),
    "x_y_swapped_in_centre": ("cell_centre(p, i, j, &x, &y);\n\n", "cell_centre(p, j, i, &x, &y);\n\n"),
    # backward
    "bwd_dx_uses_x_fraction": ("da[LP + t] += ge * ((1.0 - ay) * (v[1] - v[0]) + ay * (v[3] - v[2]));",
                               "da[LP + t] += ge * ((1.0 - ax) * (v[1] - v[0]) + ax * (v[3] - v[2]));"),
    "bwd_dy_sign": ("da[2 * LP + t] += ge * ((1.0 - ax) * (v[2] - v[0])",
                    "da[2 * LP + t] += ge * ((1.0 - ax) * (v[0] - v[2])"),
    "bwd_softmax_without_dot": ("grad_logits[o + t] = a[t] * (alpha * da[t] - dot);",
                                "grad_logits[o + t] = a[t] * (alpha * da[t]);"),
    "bwd_value_without_mean": ("const double wa = alpha * attn[(size_t)h * LP + l * P + k];",
                               "const double wa = attn[(size_t)h * LP + l * P + k];"),
    "bwd_value_all_to_first_camera": ("double *gv = grad_value + (size_t)bn * S * C;",
                                      "double *gv = grad_value + (size_t)(bn - n) * S * C;"),
    "bwd_offsets_without_attention": ("grad_offsets[(o + t) * 2 + 0] = alpha * a[t] * da[LP + t];",
                                      "grad_offsets[(o + t) * 2 + 0] = alpha * da[LP + t];"),
}


def _pin_suite():
    """Cheapest first: a mutant stops at the first pin that catches it."""
    return [
        ("hand_centre", pins.test_hand_point_offset_to_a_pixel_centre),
        ("hand_bilinear", pins.test_hand_point_bilinear_between_pixels),
        ("hand_invalid_anchor", pins.test_hand_invalid_anchor_of_a_hit_camera_still_samples),
        ("hand_k_mod_z", pins.test_hand_point_k_uses_anchor_k_mod_z),
        ("hand_mean", pins.test_hand_mean_over_hit_cameras_and_sum_mode),
        ("hand_open", pins.test_hand_image_interval_is_open),
        ("hand_behind", pins.test_hand_behind_camera_not_hit),
        ("hand_behind_anchor", pins.test_hand_anchor_behind_a_hit_camera_lands_far_away),
        ("hand_padding", pins.test_hand_locations_outside_the_map_are_zero_padded),
        ("hand_levels_heads", pins.test_hand_second_level_and_second_head),
        ("dense_small", lambda: pins.test_oracle_equals_dense_bevformer_path("small", "mean")),
        ("dense_p8", lambda: pins.test_oracle_equals_dense_bevformer_path("small_p8", "sum")),
        ("eq1", pins.test_reduces_to_eq1_for_one_point_at_the_anchor),
        ("linear", pins.test_linear_value_field_closed_form),
        ("bwd_invariants", bpins.test_invariants),
        ("bwd_adjoint", lambda: bpins.test_value_gradient_adjoint_identity("mean")),
        ("bwd_autograd", lambda: bpins.test_backward_equals_autograd_of_dense_path("small", "mean")),
        ("bwd_fd_logits", bpins.test_logits_gradient_is_a_finite_difference),
        ("bwd_fd_offsets", bpins.test_offsets_gradient_is_a_finite_difference),
    ]


def _build_mutant(tmp_path, name, old, new):
    src = open(obuild.SCA_SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", *obuild.CFLAGS, obuild.SRC, str(path), "-o", str(lib), "-lm"],
                   check=True, capture_output=True)
    return str(lib)


def test_unmutated_oracle_passes_suite():
    for _, fn in _pin_suite():
        fn()


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_sca_mutant(tmp_path, mutant):
    old, new = MUTANTS[mutant]
    path = _build_mutant(tmp_path, mutant, old, new)
    real = oracle.lib()
    mlib = ctypes.CDLL(path)
    for fn in ("oracle_sample_vt", "oracle_sample_cells", "oracle_project",
               "oracle_sample_vt_backward"):
        getattr(mlib, fn).argtypes = getattr(real, fn).argtypes
        getattr(mlib, fn).restype = getattr(real, fn).restype
    saved = oracle._LIB
    caught = []
    oracle._LIB = mlib
    try:
        for name, fn in _pin_suite():
            try:
                fn()
            except AssertionError:
                caught.append(name)
                break
    finally:
        oracle._LIB = saved
    assert caught, f"no pin catches mutant {mutant}"
    print(f"[mutant] {mutant} caught by {caught[0]}")
