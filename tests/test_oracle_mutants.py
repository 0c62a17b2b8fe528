"""The oracle's pins catch plausible mistakes.

Each mutant is a copy of the oracle's C source with one plausible mistake
planted (a dropped term, a wrong sign or index, a transposed operand, a
wrong convention).  It is compiled on the CPU into a temporary library and
run through the pin tests; every mutant must fail at least one pin.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
import test_oracle_backward_pins as bpins
import test_oracle_pins as pins
from oracle import build as obuild

MUTANTS = {
    "voxel_corner_not_centre": ("float fi = (float)i + 0.5f;", "float fi = (float)i;"),
    "align_corners_true": ("*xf = tx - 0.5f;", "*xf = tx;"),
    "negative_depth_accepted": ("if (!(d > p->depth_eps))", "if (!(d != 0.0f))"),
    "closed_image_box": ("u < (float)p->img_w", "u <= (float)p->img_w"),
    "mean_over_all_cameras": ("(double)den : 1.0;", "(double)p->N : 1.0;"),
    "x_weights_swapped": ("double wx = tx ? (double)ax : 1.0 - (double)ax;",
                          "double wx = tx ? 1.0 - (double)ax : (double)ax;"),
    "x_y_swapped_in_centre": ("voxel_centre(p, i, j, &x, &y);\n    for (int c = 0; c < C; ++c) { acc",
                              "voxel_centre(p, j, i, &x, &y);\n    for (int c = 0; c < C; ++c) { acc"),
    "wrong_matrix_entry": ("a = m[4] * x;", "a = m[1] * x;"),
    "dropped_height_term": ("float up = ((a + b) + c) + m[3];", "float up = (a + b) + m[3];"),
    "depth_offset_sign": ("float d = ((a + b) + c) + m[11];", "float d = ((a + b) + c) - m[11];"),
    "no_height_sum": ("acc[c] += num[c] / dd;", "acc[c] = num[c] / dd;"),
    "trunc_not_floor": ("float x0f = floorf(xf), y0f = floorf(yf);",
                        "float x0f = truncf(xf), y0f = truncf(yf);"),
    "den_counts_taps": ("den += 1;                 /* num_z", "den += 0;                 /* num_z"),
    "feature_row_col_swapped": ("* p->H + yt) * p->W + xt) * C;", "* p->H + xt % p->H) * p->W + yt) * C;"),
    # backward
    "bwd_no_valid_mean": ("? 1.0 / (double)seen : 1.0;", "? 1.0 : 1.0;"),
    "bwd_grad_cell_transposed": ("* p->X + i) * p->Y + j];",
                                 "* p->X + j % p->X) * p->Y + i % p->Y];"),
    "bwd_den_counts_all_cameras": ("seen += project(p, l2i", "seen += 1 + 0 * project(p, l2i"),
    "bwd_tap_row_col_swapped": ("const size_t q = (size_t)tys[t] * p->W + txs[t];",
                                "const size_t q = (size_t)(txs[t] % p->H) * p->W + tys[t] % p->W;"),
    "bwd_camera_of_first_batch": ("const float *m = l2i + (size_t)bn * 16;",
                                  "const float *m = l2i + (size_t)(bn % p->N) * 16;"),
    "bwd_weight_of_first_tap": ("const double term = tws[t] * norm * g;",
                                "const double term = tws[0] * norm * g;"),
}


def _pin_suite():
    """A fast subset of the pins, as (name, callable)."""
    return [
        ("brute_force", lambda: pins.test_oracle_equals_brute_force_ragged(1)),
        ("grid_sample", pins.test_single_camera_single_height_is_grid_sample),
        ("constant_mean", lambda: pins.test_constant_map_counts("mean")),
        ("planar", pins.test_planar_map_is_reproduced_exactly),
        ("axis", pins.test_hand_point_on_optical_axis_hits_principal_point),
        ("off_axis", pins.test_hand_point_off_axis_bilinear_weights),
        ("border", pins.test_hand_point_image_border_is_half_open),
        ("behind", pins.test_hand_point_behind_camera_is_rejected),
        ("mean_and_sum", pins.test_hand_points_valid_mean_over_cameras_and_sum_over_heights),
        ("additivity", pins.test_height_subset_additivity),
        ("bwd_jacobian", lambda: bpins.test_backward_is_transpose_of_brute_force_jacobian("mean")),
        ("bwd_adjoint", lambda: bpins.test_adjoint_identity_with_forward_oracle("sum", "ragged")),
        ("bwd_terms", bpins.test_term_counts_add_up_to_forward_taps),
    ]


def _build_mutant(tmp_path, name, old, new):
    src = open(obuild.SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", *obuild.CFLAGS, str(path), "-o", str(lib), "-lm"], check=True,
                   capture_output=True)
    return str(lib)


def test_unmutated_oracle_passes_suite():
    for name, fn in _pin_suite():
        fn()


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_mutant(tmp_path, mutant):
    old, new = MUTANTS[mutant]
    path = _build_mutant(tmp_path, mutant, old, new)
    real = oracle.lib()
    saved = oracle._LIB
    mlib = ctypes.CDLL(path)
    for fn in ("oracle_sample_vt", "oracle_sample_cells", "oracle_project",
               "oracle_sample_vt_backward"):
        getattr(mlib, fn).argtypes = getattr(real, fn).argtypes
        getattr(mlib, fn).restype = getattr(real, fn).restype
    caught = []
    oracle._LIB = mlib
    try:
        for name, fn in _pin_suite():
            try:
                fn()
            except AssertionError:
                caught.append(name)
    finally:
        oracle._LIB = saved
    assert caught, f"no pin catches mutant {mutant}"
