"""Pins of the FlashSCA oracle (BEVFormer spatial cross-attention, Sec. 4.5).

The oracle is checked against things other than itself:
  * BEVFormer's dense per-camera path (tests/sca_dense.py): the full
    sampling-location tensor, torch grid_sample and softmax, float64;
  * the reduction to Eq. 1: one head, one level, one point, one anchor and
    zero offsets make SCA the valid mean over cameras of a bilinear sample,
    which the Eq. 1 oracle (pinned in test_oracle_pins.py) computes;
  * a closed form: bilinear sampling reproduces a value map that is linear
    in the pixel position, so the output is an attention-weighted mean of
    linear functions of the sampling locations, computed here in float64;
  * hand-placed anchors with exactly known projections and pixel values,
    including the readings a random input cannot show (an invalid anchor of
    a hit camera still samples, the open image interval, behind-camera
    anchors);
  * invariants: softmax shift, camera permutation, linearity in the value,
    head independence, and sum versus mean over hit cameras.
"""
import numpy as np
import pytest

import oracle
import synth
from sca_dense import anchors_in_cameras, dense_sca, robust_queries


def _run(inst, reduce="mean"):
    return oracle.sca_instance(inst, reduce)


def _dense(inst, reduce="mean"):
    wl = inst.wl
    return dense_sca(inst.value, inst.lidar2img, inst.z, inst.offsets, inst.logits, wl.levels,
                     wl.heads, (wl.img_h, wl.img_w), wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min,
                     wl.dy, wl.depth_eps, reduce)


def _robust(inst):
    wl = inst.wl
    return robust_queries(inst.lidar2img, inst.z, wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy,
                          (wl.img_h, wl.img_w), wl.depth_eps)


# The oracle takes sampling locations in float32 (the paper's precision), the
# dense path in float64: the two differ by float32 rounding of the locations
# (a few 1e-5 pixels), which moves each bilinear term by at most that much
# times the value gradient.  Measured at BEVFormer-base shapes: at most
# 8.6e-4 S.  A mistake in the method moves the output by a sizeable part of S.
DENSE_TOL = 4e-3


def small_sca(seed=0, **kw):
    base = dict(name="small", cfg_id=200 + seed, B=2, N=6, img_h=256, img_w=704,
                levels=((20, 44), (10, 22), (5, 11)), C=12, heads=3, P=4, Z=2, dtype="f32",
                X=13, Y=11, x_min=-26.0, dx=4.0, y_min=-22.0, dy=4.0)
    base.update(kw)
    return synth.make_sca_workload(synth.ScaWorkload(**base))


@pytest.mark.parametrize("which", ["tiny", "small", "small_z1", "small_p8"])
@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_oracle_equals_dense_bevformer_path(which, reduce):
    inst = {"tiny": lambda: synth.make_sca_workload(synth.sca_config("sca_tiny")),
            "small": lambda: small_sca(1),
            "small_z1": lambda: small_sca(2, Z=1, P=3),
            "small_p8": lambda: small_sca(3, P=8, Z=4, levels=((24, 64), (12, 32)))}[which]()
    out, scale, terms, cnt = _run(inst, reduce)
    ref, hit, _ = _dense(inst, reduce)
    keep = _robust(inst)
    assert keep.mean() > 0.95
    assert hit.any(axis=1)[keep].sum() > 20 and cnt["taps"] > 100
    err = np.abs(out - ref)[keep]
    bad = err > DENSE_TOL * scale[keep] + 1e-12
    assert not bad.any(), f"{bad.sum()} elements off; max scaled {(err / (scale[keep] + 1e-30)).max()}"
    # queries no camera sees are exactly zero
    none = ~hit.any(axis=1)
    assert np.all(out[none] == 0.0) and np.all(terms[none] == 0)


def test_large_shapes_equal_dense_path_on_a_coarse_grid():
    """BEVFormer-base levels, heads and points on a 60x60 grid of queries."""
    wl = synth.sca_config("sca_base", X=60, Y=60, dx=102.4 / 60, dy=102.4 / 60, C=64)
    inst = synth.make_sca_workload(wl)
    out, scale, _, _ = _run(inst)
    ref, hit, _ = _dense(inst)
    keep = _robust(inst)
    err = np.abs(out - ref)[keep]
    assert hit.any(axis=1).mean() > 0.9
    assert np.all(err <= DENSE_TOL * scale[keep] + 1e-12)


def test_reduces_to_eq1_for_one_point_at_the_anchor():
    """heads=1, L=1, P=1, Z=1, zero offsets: SCA is Eq. 1 at one height."""
    fwl = synth.config("tiny").with_(Z=1, C=5, X=31, Y=29)
    finst = synth.make_workload(fwl)
    z = np.array([0.25], dtype=np.float32)
    Q = fwl.X * fwl.Y
    value = finst.features.reshape(fwl.B, fwl.N, fwl.H * fwl.W, fwl.C)
    offsets = np.zeros((fwl.B, Q, 1, 1, 1, 2), dtype=np.float32)
    logits = np.random.default_rng(5).standard_normal((fwl.B, Q, 1, 1, 1)).astype(np.float32)
    out, scale, _, cnt = oracle.sca_forward(value, finst.lidar2img, z, offsets, logits,
                                            [(fwl.H, fwl.W)], 1, (fwl.img_h, fwl.img_w), fwl.X,
                                            fwl.Y, fwl.x_min, fwl.dx, fwl.y_min, fwl.dy)
    eq1, eq1_scale, eq1_cnt = oracle.sample_vt(finst.features, finst.lidar2img, z,
                                               (fwl.img_h, fwl.img_w), fwl.X, fwl.Y, fwl.x_min,
                                               fwl.dx, fwl.y_min, fwl.dy)
    eq1 = eq1.transpose(0, 2, 3, 1).reshape(fwl.B, Q, fwl.C)
    keep = robust_queries(finst.lidar2img, z, fwl.X, fwl.Y, fwl.x_min, fwl.dx, fwl.y_min, fwl.dy,
                          (fwl.img_h, fwl.img_w))
    assert keep.mean() > 0.95 and cnt["hits"] > 100
    err = np.abs(out - eq1)[keep]
    # only the order of float32 roundings of the feature coordinate differs
    assert np.all(err <= 1e-3 * scale[keep] + 1e-12)


def _linear_value(levels, B, N, C, alpha, beta, gamma):
    parts = []
    for h, w in levels:
        yy, xx = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
        v = (alpha[None, None, None, :] * xx.reshape(1, 1, -1, 1)
             + beta[None, None, None, :] * yy.reshape(1, 1, -1, 1)
             + gamma[:, :, None, :])
        parts.append(np.broadcast_to(v, (B, N, h * w, C)))
    return np.concatenate(parts, axis=2).astype(np.float32)


def test_linear_value_field_closed_form():
    inst = small_sca(4, levels=((40, 100), (20, 50)), P=4, Z=2, heads=2, C=4, X=15, Y=15,
                     x_min=-30.0, dx=4.0, y_min=-30.0, dy=4.0)
    wl = inst.wl
    rng = np.random.default_rng(7)
    alpha = np.array([0.5, -0.25, 0.125, 1.0], dtype=np.float32)
    beta = np.array([0.25, 0.5, -1.0, 0.0], dtype=np.float32)
    gamma = rng.integers(-4, 5, size=(wl.B, wl.N, wl.C)).astype(np.float32)
    inst.value = _linear_value(wl.levels, wl.B, wl.N, wl.C, alpha, beta, gamma)
    inst.offsets = (0.25 * inst.offsets).astype(np.float32)
    out, _, _, _ = _run(inst)
    # closed form from float64 reference points
    ref, valid, _ = anchors_in_cameras(inst.lidar2img, inst.z, wl.X, wl.Y, wl.x_min, wl.dx,
                                       wl.y_min, wl.dy, (wl.img_h, wl.img_w))
    ref = ref.numpy()
    hit = valid.numpy().any(axis=-1)                                  # [B, N, Q]
    lg = inst.logits.astype(np.float64).reshape(wl.B, wl.Q, wl.heads, -1)
    a = np.exp(lg - lg.max(axis=-1, keepdims=True))
    a = (a / a.sum(axis=-1, keepdims=True)).reshape(wl.B, wl.Q, wl.heads, wl.L, wl.P)
    D = wl.C // wl.heads
    keep = _robust(inst)
    checked = 0
    for b in range(wl.B):
        for q in range(wl.Q):
            if not keep[b, q]:
                continue
            cams = np.nonzero(hit[b, :, q])[0]
            acc = np.zeros(wl.C)
            inside = True
            for n in cams:
                for m in range(wl.heads):
                    for l, (hl, wdt) in enumerate(wl.levels):
                        for k in range(wl.P):
                            r = ref[b, n, q, k % wl.Z]
                            o = inst.offsets[b, q, m, l, k].astype(np.float64)
                            xi = r[0] * wdt + o[0] - 0.5
                            yi = r[1] * hl + o[1] - 0.5
                            if not (0.01 < xi < wdt - 1.01 and 0.01 < yi < hl - 1.01):
                                inside = False
                            c = slice(m * D, (m + 1) * D)
                            acc[c] += a[b, q, m, l, k] * (alpha[c] * xi + beta[c] * yi
                                                          + gamma[b, n, c])
            if not inside or len(cams) == 0:
                continue
            acc /= len(cams)
            assert np.allclose(out[b, q], acc, rtol=0, atol=2e-4), (b, q, out[b, q], acc)
            checked += 1
    assert checked >= 30, checked


# ---------------------------------------------------------------------------
# Hand-placed anchors.  Camera n looks along +x (or -x) with fx = fy = 100 and
# principal point (cx_n, 40) in a 80 x 100 image:
#   (u', v', d) = (cx_n x - 100 s y, 40 x - 100 s z, x) with s = +1 (or -1).
# A query at (10, 0) with anchor z = 0 lands on (cx_n, 40), i.e. normalized
# (cx_n / 100, 0.5); every step is exact in float32.
# ---------------------------------------------------------------------------


def _cam(cx, sign=1.0):
    m = np.zeros((4, 4), dtype=np.float32)
    m[0] = [sign * cx, -100.0 * sign, 0.0, 0.0]
    m[1] = [sign * 40.0, 0.0, -100.0 * sign, 0.0]
    m[2] = [sign * 1.0, 0.0, 0.0, 0.0]
    m[3] = [0.0, 0.0, 0.0, 1.0]
    return m


def _hand(cams, z, offsets, logits, levels=((8, 10),), heads=1, C=2, x_centre=10.0,
          value=None, reduce="mean"):
    N = len(cams)
    l2i = np.stack(cams)[None]
    S = sum(h * w for h, w in levels)
    if value is None:
        # value[n, pixel, c] = 1000 n + 10 pixel + c: every tap identifiable
        value = (1000.0 * np.arange(N)[:, None, None] + 10.0 * np.arange(S)[None, :, None]
                 + np.arange(C)[None, None, :]).astype(np.float32)[None]
    off = np.asarray(offsets, dtype=np.float32).reshape(1, 1, heads, len(levels), -1, 2)
    lg = np.asarray(logits, dtype=np.float32).reshape(1, 1, heads, len(levels), -1)
    out, scale, terms, cnt = oracle.sca_forward(
        value, l2i, np.asarray(z, np.float32), off, lg, list(levels), heads, (80, 100), 1, 1,
        x_centre - 0.5, 1.0, -0.5, 1.0, reduce=reduce)
    return out[0, 0], cnt


NEG = -1e30  # softmax weight exactly zero in float64


def test_hand_point_offset_to_a_pixel_centre():
    # un = 0.5 -> x = 0.5 * 10 + 0.5 - 0.5 = 5; vn = 0.5 -> y = 0.5 * 8 + 0.5 - 0.5 = 4
    out, cnt = _hand([_cam(50.0)], [0.0, 100.0], [[0.5, 0.5], [0.0, 0.0]], [0.0, NEG])
    assert cnt["hits"] == 1
    assert np.array_equal(out, 10.0 * (4 * 10 + 5) + np.arange(2))


def test_hand_point_bilinear_between_pixels():
    # x = 5.25, y = 4.5: weights 0.375, 0.125, 0.375, 0.125 on (4,5) (4,6) (5,5) (5,6)
    out, _ = _hand([_cam(50.0)], [0.0, 100.0], [[0.75, 1.0], [0.0, 0.0]], [0.0, NEG])
    pix = lambda y, x: 10.0 * (y * 10 + x)
    expect = 0.375 * pix(4, 5) + 0.125 * pix(4, 6) + 0.375 * pix(5, 5) + 0.125 * pix(5, 6)
    assert np.allclose(out, expect + np.arange(2), rtol=0, atol=1e-9)


def test_hand_invalid_anchor_of_a_hit_camera_still_samples():
    # anchor 1 (z = 100) projects to v = -960 (vn = -12): invalid, but camera 0
    # is hit through anchor 0, so point 1 (anchor 1 mod 2) samples at
    # y = -12 * 8 + 99.5 - 0.5 = 3, x = 5.
    out, cnt = _hand([_cam(50.0)], [0.0, 100.0], [[0.0, 0.0], [0.5, 99.5]], [NEG, 0.0])
    assert cnt["hits"] == 1
    assert np.array_equal(out, 10.0 * (3 * 10 + 5) + np.arange(2))


def test_hand_point_k_uses_anchor_k_mod_z():
    # P = 4, Z = 2: points 0, 2 -> anchor 0; points 1, 3 -> anchor 1.
    offs = [[0.0, 0.0], [0.0, 0.0], [0.5, 0.5], [0.5, 99.5]]
    out2, _ = _hand([_cam(50.0)], [0.0, 100.0], offs, [NEG, NEG, 0.0, NEG])
    out3, _ = _hand([_cam(50.0)], [0.0, 100.0], offs, [NEG, NEG, NEG, 0.0])
    assert np.array_equal(out2, 10.0 * (4 * 10 + 5) + np.arange(2))
    assert np.array_equal(out3, 10.0 * (3 * 10 + 5) + np.arange(2))


def test_hand_mean_over_hit_cameras_and_sum_mode():
    cams = [_cam(50.0), _cam(30.0), _cam(50.0, sign=-1.0)]     # the third looks backwards
    offs = [[0.5, 0.5], [0.0, 0.0]]
    out, cnt = _hand(cams, [0.0, 100.0], offs, [0.0, NEG])
    # camera 1: un = 0.3 -> x = 3 + 0.5 - 0.5 = 3
    v0 = 10.0 * (4 * 10 + 5)
    v1 = 1000.0 + 10.0 * (4 * 10 + 3)
    assert cnt["hits"] == 2
    assert np.array_equal(out, (v0 + v1) / 2 + np.arange(2))
    out_s, _ = _hand(cams, [0.0, 100.0], offs, [0.0, NEG], reduce="sum")
    assert np.array_equal(out_s, v0 + v1 + 2 * np.arange(2))


def test_hand_image_interval_is_open():
    # principal point 0: the anchor lands on u = 0 exactly -> not inside
    out, cnt = _hand([_cam(0.0)], [0.0], [[5.5, 0.5]], [0.0])
    assert cnt["hits"] == 0 and np.all(out == 0.0)
    # principal point 100 (u = img_w): likewise
    out, cnt = _hand([_cam(100.0)], [0.0], [[-5.5, 0.5]], [0.0])
    assert cnt["hits"] == 0 and np.all(out == 0.0)
    # just inside
    out, cnt = _hand([_cam(99.0)], [0.0], [[-4.4, 0.5]], [0.0])
    assert cnt["hits"] == 1 and np.all(out != 0.0)


def test_hand_behind_camera_not_hit():
    out, cnt = _hand([_cam(50.0)], [0.0], [[0.5, 0.5]], [0.0], x_centre=-10.0)
    assert cnt["hits"] == 0 and np.all(out == 0.0)


def test_hand_anchor_behind_a_hit_camera_lands_far_away():
    # depth d = x + z: anchor 0 (z = 0) has d = 10 and hits the camera; anchor 1
    # (z = -20) has d = -10.  Dividing by the clamped depth (1e-5) sends it
    # millions of pixels away, so its point samples nothing.  (Dividing by the
    # raw depth would give un = -0.5, vn = -3, which these offsets bring back
    # onto pixel (4, 5).)
    cam = _cam(50.0)
    cam[2] = [1.0, 0.0, 1.0, 0.0]
    out, cnt = _hand([cam], [0.0, -20.0], [[0.0, 0.0], [10.5, 28.5]], [NEG, 0.0])
    assert cnt["hits"] == 1
    assert np.all(out == 0.0)
    # and the valid anchor's point, for contrast, samples pixel (4, 5)
    out, _ = _hand([cam], [0.0, -20.0], [[0.5, 0.5], [10.5, 28.5]], [0.0, NEG])
    assert np.array_equal(out, 10.0 * (4 * 10 + 5) + np.arange(2))


def test_hand_locations_outside_the_map_are_zero_padded():
    # x = 5 + 4.5 = 9.5: taps 9 (weight 0.5) and 10 (outside)
    out, _ = _hand([_cam(50.0)], [0.0], [[5.0, 0.5]], [0.0])
    assert np.allclose(out, 0.5 * 10.0 * (4 * 10 + 9) + 0.5 * np.arange(2), rtol=0, atol=1e-9)
    out, _ = _hand([_cam(50.0)], [0.0], [[60.0, 0.5]], [0.0])
    assert np.all(out == 0.0)


def test_hand_second_level_and_second_head():
    levels = ((8, 10), (4, 5))
    # head 0: weight on level 1 only; head 1: level 0 only
    offs = [[[0.0, 0.0]], [[0.0, 0.5]], [[0.5, 0.5]], [[0.0, 0.0]]]     # [heads, L, P=1, 2]
    lgs = [[NEG], [0.0], [0.0], [NEG]]
    out, _ = _hand([_cam(50.0)], [0.0], offs, lgs, levels=levels, heads=2, C=4)
    # level 1 (4 x 5): x = 0.5 * 5 + 0 - 0.5 = 2, y = 0.5 * 4 + 0.5 - 0.5 = 2 -> pixel 80 + 12
    # level 0: pixel 45
    assert np.array_equal(out[:2], 10.0 * (80 + 2 * 5 + 2) + np.arange(2))
    assert np.array_equal(out[2:], 10.0 * 45 + np.arange(2, 4))


# ---------------------------------------------------------------------------
# Invariants
# ---------------------------------------------------------------------------


def test_softmax_shift_invariance():
    inst = small_sca(5)
    out, scale, _, _ = _run(inst)
    shift = np.random.default_rng(3).uniform(-5, 5, size=inst.logits.shape[:3])
    inst.logits = (inst.logits + shift[..., None, None]).astype(np.float32)
    out2, _, _, _ = _run(inst)
    assert np.all(np.abs(out - out2) <= 1e-5 * scale + 1e-12)


def test_camera_permutation_invariance():
    inst = small_sca(6)
    out, scale, _, _ = _run(inst)
    perm = np.array([3, 0, 5, 1, 4, 2])
    inst.value = np.ascontiguousarray(inst.value[:, perm])
    inst.lidar2img = np.ascontiguousarray(inst.lidar2img[:, perm])
    out2, _, _, _ = _run(inst)
    assert np.all(np.abs(out - out2) <= 1e-12 * scale + 1e-300)


def test_linearity_in_value():
    inst = small_sca(7)
    # values on a 1/64 grid, so that 2 v1 - 3 v2 is exact in float32
    v1 = (np.round(inst.value * 64.0) / 64.0).astype(np.float32)
    v2 = (np.round(np.random.default_rng(9).standard_normal(v1.shape) * 64.0) / 64.0
          ).astype(np.float32)
    inst.value = v1
    o1, s1, _, _ = _run(inst)
    inst.value = v2
    o2, s2, _, _ = _run(inst)
    inst.value = (2.0 * v1 - 3.0 * v2).astype(np.float32)
    o3, _, _, _ = _run(inst)
    assert np.all(np.abs(o3 - (2.0 * o1 - 3.0 * o2)) <= 1e-12 * (2 * s1 + 3 * s2) + 1e-300)


def test_heads_are_independent():
    inst = small_sca(8)
    out, _, _, _ = _run(inst)
    D = inst.wl.C // inst.wl.heads
    inst.offsets[:, :, 1] += 2.5
    inst.logits[:, :, 1] *= -1.0
    out2, _, _, _ = _run(inst)
    assert np.array_equal(out[..., :D], out2[..., :D])
    assert np.array_equal(out[..., 2 * D:], out2[..., 2 * D:])
    assert not np.allclose(out[..., D:2 * D], out2[..., D:2 * D])


def test_sum_mode_is_mean_times_hit_count():
    inst = small_sca(9)
    wl = inst.wl
    om, sm, _, _ = _run(inst, "mean")
    os_, _, _, _ = _run(inst, "sum")
    _, _, _, hit = oracle.sca_reference_points(inst.lidar2img, inst.z, wl.B, wl.N,
                                               (wl.img_h, wl.img_w), wl.X, wl.Y, wl.x_min,
                                               wl.dx, wl.y_min, wl.dy)
    cnt = np.maximum(hit.sum(axis=-1), 1)[..., None]
    assert (cnt > 1).any()
    assert np.all(np.abs(os_ - om * cnt) <= 1e-12 * sm * cnt + 1e-300)


def test_terms_count_in_range_taps():
    inst = small_sca(10)
    _, _, terms, cnt = _run(inst)
    assert int(terms.sum()) == cnt["taps"] > 0
    wl = inst.wl
    assert terms.max() <= wl.N * wl.L * wl.P * 4


@pytest.mark.parametrize("which", ["tiny", "small", "wide_z"])
def test_reference_points_equal_the_dense_projection(which):
    """The oracle's reference points (step 1: every anchor projected into
    every camera, normalized by the image size) and their masks against the
    dense path's float64 projection, independent code.  Masks and hit
    cameras agree exactly on robust queries; the float32 coordinates agree
    within their rounding bound, including the depth-clamped points of
    anchors behind a camera (an invalid anchor of a hit camera still
    samples)."""
    inst = {"tiny": lambda: synth.make_sca_workload(synth.sca_config("sca_tiny")),
            "small": lambda: small_sca(11),
            "wide_z": lambda: small_sca(12, Z=4, P=8, z_lo=-9.0, z_hi=6.0)}[which]()
    wl = inst.wl
    un, vn, valid, hit = oracle.sca_reference_points(
        inst.lidar2img, inst.z, wl.B, wl.N, (wl.img_h, wl.img_w), wl.X, wl.Y, wl.x_min, wl.dx,
        wl.y_min, wl.dy, wl.depth_eps)
    eps32 = float(np.float32(wl.depth_eps))
    ref, dvalid, depth = anchors_in_cameras(inst.lidar2img, inst.z, wl.X, wl.Y, wl.x_min, wl.dx,
                                            wl.y_min, wl.dy, (wl.img_h, wl.img_w), eps32)
    # dense layout [B, N, Q, Z] -> the oracle's [B, Q, N, Z]
    ref = ref.numpy().transpose(0, 2, 1, 3, 4)
    dvalid = dvalid.numpy().transpose(0, 2, 1, 3)
    depth = depth.numpy().transpose(0, 2, 1, 3)
    keep = robust_queries(inst.lidar2img, inst.z, wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy,
                          (wl.img_h, wl.img_w), eps32)
    assert keep.mean() > 0.9
    assert np.array_equal(valid[keep], dvalid[keep])
    assert np.array_equal(hit[keep], dvalid.any(axis=-1)[keep])
    assert dvalid[keep].any() and not dvalid[keep].all() and (depth <= eps32).any()
    # rounding bound of the float32 recipe on robust queries (no depth near
    # the clamp): the cell centre carries 3 roundings and each of (u', v', d)
    # 3 more of its term magnitudes; the divides and the normalization one
    # each
    # cell centres are formed in float32 as well, so their magnitude terms
    # are |x_min| + (i + 1/2) |dx| (likewise y)
    m = np.asarray(inst.lidar2img, np.float64)
    xs = abs(wl.x_min) + (np.arange(wl.X) + 0.5) * abs(wl.dx)
    ys = abs(wl.y_min) + (np.arange(wl.Y) + 0.5) * abs(wl.dy)
    gx, gy = np.meshgrid(xs, ys, indexing="ij")
    pts = np.stack([gx.reshape(-1, 1).repeat(wl.Z, 1), gy.reshape(-1, 1).repeat(wl.Z, 1),
                    np.broadcast_to(np.asarray(inst.z, np.float64), (wl.X * wl.Y, wl.Z)),
                    np.ones((wl.X * wl.Y, wl.Z))], axis=-1)            # [Q, Z, 4]
    mag = np.einsum("bnrc,qzc->bqnzr", np.abs(m), np.abs(pts))          # [B, Q, N, Z, 4]
    dd = np.maximum(depth, eps32)
    e = 2.0 ** -24
    for k, (got, size) in enumerate(((un, wl.img_w), (vn, wl.img_h))):
        want = ref[..., k]
        bound = (6 * e * (mag[..., k] + np.abs(want * size) * mag[..., 2]) / dd / size
                 + 3 * e * np.abs(want))
        err = np.abs(got.astype(np.float64) - want)[keep]
        assert np.all(err <= bound[keep]), (which, k, float((err / bound[keep]).max()))
