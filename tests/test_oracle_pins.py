"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

The paper prints no worked example, so the oracle (Eq. 1 as a per-query
loop) is pinned by:
  * brute force: the staged tensorized evaluation of Alg. 1 (numpy,
    materializing Features3D) on tiny inputs;
  * a library special case: one camera and one height reduce to torch's
    grid_sample (bilinear, zero padding, align_corners=False);
  * closed forms: constant and planar feature maps, and hand-placed points
    whose projections are exact dyadic numbers worked out below;
  * invariants of Eq. 1: camera permutation, linearity, channel
    independence, height-subset additivity, batch independence, empty cells.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from brute_force import tensorized_sample_vt, run_instance as brute_instance


def small_workload(B=2, N=3, H=6, W=9, C=5, X=7, Y=5, Z=3, img=(48, 72), seed=7,
                   half_range=12.0):
    wl = synth.Workload(name="small", cfg_id=100 + seed, B=B, N=N, img_h=img[0], img_w=img[1],
                        H=H, W=W, C=C, dtype="f32", X=X, Y=Y, x_min=-half_range,
                        dx=2 * half_range / X, y_min=-half_range, dy=2 * half_range / Y,
                        z_lo=-3.0, z_hi=2.0, Z=Z)
    return synth.make_workload(wl)


def rel_err(a, b, s):
    s = np.maximum(s, 1e-300)
    return np.max(np.abs(a - b) / s)


# --------------------------------------------------------------------------
# brute force (Alg. 1)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_oracle_equals_tensorized_brute_force_tiny(reduce):
    inst = synth.make_workload(synth.config("tiny"))
    ref = brute_instance(inst, reduce)
    out, scale, cnt = oracle.run_instance(inst, reduce)
    assert cnt["valid_samples"] > 1000
    assert np.all(np.abs(out - ref) <= 1e-12 * scale + 1e-300)
    assert np.count_nonzero(out) > 0.5 * out.size


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_oracle_equals_brute_force_ragged(seed):
    inst = small_workload(seed=seed)
    ref = brute_instance(inst)
    out, scale, _ = oracle.run_instance(inst)
    assert np.all(np.abs(out - ref) <= 1e-12 * scale + 1e-300)


def test_oracle_equals_brute_force_16bit_values():
    wl = synth.config("tiny").with_(dtype="bf16", C=16, X=20, Y=24)
    inst = synth.make_workload(wl)
    # features are exact bf16 values
    import torch
    t = torch.from_numpy(inst.features)
    assert torch.equal(t.to(torch.bfloat16).to(torch.float32), t)
    ref = brute_instance(inst)
    out, scale, _ = oracle.run_instance(inst)
    assert np.all(np.abs(out - ref) <= 1e-12 * scale + 1e-300)


# --------------------------------------------------------------------------
# library special case: N = 1, Z = 1 is grid_sample
# --------------------------------------------------------------------------
def test_single_camera_single_height_is_grid_sample():
    import torch
    import torch.nn.functional as F

    wl = synth.config("tiny").with_(N=1, Z=1, X=40, Y=40, C=6, cfg_id=11)
    inst = synth.make_workload(wl)
    inst.z = np.array([-1.0], dtype=np.float32)
    out, scale, cnt = oracle.run_instance(inst)
    assert cnt["valid_samples"] > 50

    # independent float64 pinhole projection of the cell centres
    P = inst.lidar2img[0, 0].astype(np.float64)
    xs = wl.x_min + (np.arange(wl.X) + 0.5) * wl.dx
    ys = wl.y_min + (np.arange(wl.Y) + 0.5) * wl.dy
    gx, gy = np.meshgrid(xs, ys, indexing="ij")
    pts = np.stack([gx, gy, np.full_like(gx, -1.0), np.ones_like(gx)], -1)
    uvd = pts @ P[:3].T
    d = uvd[..., 2]
    with np.errstate(divide="ignore", invalid="ignore"):
        u = uvd[..., 0] / d
        v = uvd[..., 1] / d
    valid = (d > 1e-5) & (u >= 0) & (u < wl.img_w) & (v >= 0) & (v < wl.img_h)
    # keep away from mask edges where float32 and float64 may disagree
    margin = 1e-3
    safe = (~valid) | ((u > margin) & (u < wl.img_w - margin) & (v > margin) &
                       (v < wl.img_h - margin))
    grid = np.stack([2 * u / wl.img_w - 1, 2 * v / wl.img_h - 1], -1)
    grid = np.where(valid[..., None], grid, 0.0)
    inp = torch.from_numpy(inst.features[0, 0].astype(np.float64)).permute(2, 0, 1)[None]
    g = torch.from_numpy(grid)[None]  # (1, X, Y, 2)
    ref = F.grid_sample(inp, g, mode="bilinear", padding_mode="zeros", align_corners=False)
    ref = ref[0].numpy() * valid[None]
    assert valid.sum() > 50 and (~valid).sum() > 50
    err = np.abs(out[0] - ref)[:, safe]
    assert err.max() < 1e-4, err.max()
    # invalid cells are exactly zero
    assert np.all(out[0][:, ~valid] == 0.0)


# --------------------------------------------------------------------------
# closed forms
# --------------------------------------------------------------------------
def _counts(inst):
    wl = inst.wl
    mask, xf, yf = oracle.project(inst.lidar2img, inst.z, (wl.H, wl.W), (wl.img_h, wl.img_w),
                                  wl.B, wl.N, wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy)
    interior = mask & (xf >= 0) & (xf <= wl.W - 1) & (yf >= 0) & (yf <= wl.H - 1)
    # a valid sample with all four taps in range
    all_interior = np.all(~mask | interior, axis=(3, 4))  # (B, X, Y)
    den = mask.sum(axis=4)  # (B, X, Y, Z)
    return mask, xf, yf, den, all_interior


@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_constant_map_counts(reduce):
    inst = synth.make_workload(synth.config("tiny"))
    k = 0.75
    inst.features = np.full_like(inst.features, k)
    out, scale, _ = oracle.run_instance(inst, reduce)
    mask, xf, yf, den, all_int = _counts(inst)
    if reduce == "mean":
        bound = k * (den >= 1).sum(axis=3)  # k * #{z : den_z >= 1}
    else:
        bound = k * den.sum(axis=3)  # k * sum_z den_z
    bound = bound[:, None].astype(np.float64)  # (B,1,X,Y)
    cells = np.broadcast_to(all_int[:, None], out.shape)
    assert cells.sum() > 0.5 * out.size
    assert np.allclose(out[cells], np.broadcast_to(bound, out.shape)[cells], rtol=1e-13, atol=0)
    # the zero-padding border band only attenuates
    assert np.all(out >= -1e-15) and np.all(out <= np.broadcast_to(bound, out.shape) + 1e-12)
    assert np.any(out[~cells] < np.broadcast_to(bound, out.shape)[~cells] - 1e-6)


def test_planar_map_is_reproduced_exactly():
    inst = synth.make_workload(synth.config("tiny").with_(C=4))
    wl = inst.wl
    rng = np.random.default_rng(5)
    alpha, beta, gamma = rng.normal(size=(3, wl.C))
    delta = rng.normal(size=wl.N)
    yy, xx = np.meshgrid(np.arange(wl.H), np.arange(wl.W), indexing="ij")
    # values chosen so that the float32 feature map is exact: round the
    # coefficients to multiples of 1/64 (all products are then exact)
    alpha, beta, gamma, delta = [np.round(a * 64) / 64 for a in (alpha, beta, gamma, delta)]
    plane = alpha + beta * xx[..., None] + gamma * yy[..., None]  # (H, W, C)
    feat64 = plane[None, None] + delta[None, :, None, None, None]  # (1, N, H, W, C)
    feat = np.broadcast_to(feat64, inst.features.shape).astype(np.float32)
    assert np.array_equal(feat.astype(np.float64), np.broadcast_to(feat64, feat.shape))
    inst.features = np.ascontiguousarray(feat)
    out, scale, _ = oracle.run_instance(inst)
    mask, xf, yf, den, all_int = _counts(inst)
    # closed form: sum_z mean_n (alpha + beta x_f + gamma y_f + delta_n)
    xf64 = np.where(mask, xf, 0).astype(np.float64)
    yf64 = np.where(mask, yf, 0).astype(np.float64)
    exp = np.zeros(out.shape)
    for c in range(wl.C):
        val = (alpha[c] + beta[c] * xf64 + gamma[c] * yf64 + delta[None, None, None, None, :]) * mask
        per_z = val.sum(axis=4) / np.maximum(1, den)
        exp[:, c] = per_z.sum(axis=3)
    cells = np.broadcast_to(all_int[:, None], out.shape)
    assert cells.sum() > 0.5 * out.size
    assert np.all(np.abs(out - exp)[cells] <= 1e-11 * (1 + scale[cells]))


# Hand-placed points.  One camera at the origin looking along +x with
# f = 128 and principal point (32, 16) in a 64 x 32 image; feature map
# 8 x 16 (stride 4).  Its lidar2img is K [right; down; forward] =
#   [[32, -128, 0, 0], [16, 0, -128, 0], [1, 0, 0, 0]],
# so a point (x, y, z) lands at u = 32 - 128 y / x, v = 16 - 128 z / x.
IMG = (32, 64)
FEAT_HW = (8, 16)
L2I = np.array([[32, -128, 0, 0], [16, 0, -128, 0], [1, 0, 0, 0], [0, 0, 0, 1]], np.float32)


def _hand(features, x, y, zs, l2i=None, reduce="mean"):
    """Oracle on a 1x1 BEV grid whose only cell centre is (x, y)."""
    f = np.ascontiguousarray(features, dtype=np.float32)
    B, N = f.shape[:2]
    m = np.broadcast_to(L2I if l2i is None else l2i, (B, N, 4, 4)).astype(np.float32)
    out, scale, cnt = oracle.sample_vt(f, m, np.asarray(zs, np.float32), IMG, 1, 1,
                                       x - 0.5, 1.0, y - 0.5, 1.0, reduce=reduce)
    return out[:, :, 0, 0], cnt


def test_hand_point_on_optical_axis_hits_principal_point():
    # (4, 0, 0) -> (u, v) = (32, 16) -> (x_f, y_f) = (7.5, 3.5): the centre
    # of pixels (7, 3), (8, 3), (7, 4), (8, 4), each with weight 1/4.
    f = np.zeros((1, 1) + FEAT_HW + (2,), np.float32)
    f[0, 0, 3, 7] = [1, 10]
    f[0, 0, 3, 8] = [2, 20]
    f[0, 0, 4, 7] = [4, 40]
    f[0, 0, 4, 8] = [8, 80]
    out, cnt = _hand(f, 4.0, 0.0, [0.0])
    assert cnt == {"valid_samples": 1, "taps": 4}
    assert np.array_equal(out[0], [15 / 4, 150 / 4])


def test_hand_point_off_axis_bilinear_weights():
    # y = -25/64, z = 25/128 at depth 4:
    #   u = 32 + 128 * (25/64) / 4 = 44.5  -> x_f = 44.5/4 - 1/2 = 10.625
    #   v = 16 - 128 * (25/128) / 4 = 9.75 -> y_f = 9.75/4 - 1/2 = 1.9375
    # so x0 = 10, a_x = 0.625, y0 = 1, a_y = 0.9375.
    f = np.zeros((1, 1) + FEAT_HW + (1,), np.float32)
    f[0, 0, 1, 10, 0] = 1.0    # weight (1 - 0.625)(1 - 0.9375) = 0.0234375
    f[0, 0, 1, 11, 0] = 10.0   # weight 0.625 (1 - 0.9375)       = 0.0390625
    f[0, 0, 2, 10, 0] = 100.0  # weight (1 - 0.625) 0.9375       = 0.3515625
    f[0, 0, 2, 11, 0] = 1000.0  # weight 0.625 * 0.9375          = 0.5859375
    f[0, 0, 5, 5, 0] = 1e6     # never touched
    out, _ = _hand(f, 4.0, -25 / 64, [25 / 128])
    exp = 0.0234375 + 10 * 0.0390625 + 100 * 0.3515625 + 1000 * 0.5859375
    assert out[0, 0] == exp


def test_hand_point_image_border_is_half_open():
    f = np.ones((1, 1) + FEAT_HW + (1,), np.float32)
    # y = +1 at depth 4 -> u = 32 - 32 = 0: inside (left edge); x_f = -0.5,
    # so only tap x = 0 is in range, with weight 1/2 (zero padding).
    out, cnt = _hand(f, 4.0, 1.0, [0.0])
    assert cnt["valid_samples"] == 1 and cnt["taps"] == 2
    assert out[0, 0] == 0.5
    # y = -1 -> u = 64 = img_w: outside (half-open box), no sample at all
    out, cnt = _hand(f, 4.0, -1.0, [0.0])
    assert cnt["valid_samples"] == 0 and out[0, 0] == 0.0
    # same for v: z = 0.5 -> v = 16 - 16 = 0 (inside); z = -0.5 -> v = 32 (outside)
    out, cnt = _hand(f, 4.0, 0.0, [0.5])
    assert cnt["valid_samples"] == 1 and out[0, 0] == 0.5
    out, cnt = _hand(f, 4.0, 0.0, [-0.5])
    assert cnt["valid_samples"] == 0 and out[0, 0] == 0.0


def test_hand_point_behind_camera_is_rejected():
    # (-4, 0, 0): d = -4 < 0 while u'/d = 32 and v'/d = 16 fall inside the
    # image; positive depth is required, so nothing is sampled.
    f = np.ones((1, 1) + FEAT_HW + (3,), np.float32)
    out, cnt = _hand(f, -4.0, 0.0, [0.0])
    assert cnt["valid_samples"] == 0 and np.all(out == 0.0)
    # depth exactly zero is rejected as well (the point x = 0)
    out, cnt = _hand(f, 0.0, 0.0, [0.0])
    assert cnt["valid_samples"] == 0


def test_hand_points_valid_mean_over_cameras_and_sum_over_heights():
    # Three cameras: two copies of the forward camera (features 1 and 3 at
    # the principal-point pixels) and one looking backwards (never valid for
    # x > 0).  Per height the valid mean is (1 + 3) / 2 = 2; heights z = 0
    # and z = 0.5 both project inside the image, so Eq. 1 gives 2 + 2 = 4.
    back = np.array([[32, 128, 0, 0], [16, 0, -128, 0], [-1, 0, 0, 0], [0, 0, 0, 1]], np.float32)
    l2i = np.stack([L2I, L2I, back])[None]
    f = np.zeros((1, 3) + FEAT_HW + (1,), np.float32)
    f[0, 0] = 1.0
    f[0, 1] = 3.0
    f[0, 2] = 100.0
    out, cnt = _hand(f, 4.0, 0.0, [0.0, 0.25], l2i=l2i)
    assert cnt["valid_samples"] == 4
    assert out[0, 0] == 4.0
    # plain sum over cameras (den forced to 1): 2 * (1 + 3) = 8
    out, _ = _hand(f, 4.0, 0.0, [0.0, 0.25], l2i=l2i, reduce="sum")
    assert out[0, 0] == 8.0
    # a height that projects outside the image contributes 0 / max(1, 0) = 0
    out, cnt = _hand(f, 4.0, 0.0, [0.0, 0.25, 5.0], l2i=l2i)
    assert cnt["valid_samples"] == 4 and out[0, 0] == 4.0


# --------------------------------------------------------------------------
# invariants
# --------------------------------------------------------------------------
def test_camera_permutation_invariance():
    inst = small_workload(seed=4, N=4)
    out, scale, _ = oracle.run_instance(inst)
    perm = np.array([2, 0, 3, 1])
    inst.features = np.ascontiguousarray(inst.features[:, perm])
    inst.lidar2img = np.ascontiguousarray(inst.lidar2img[:, perm])
    out2, _, _ = oracle.run_instance(inst)
    assert np.all(np.abs(out - out2) <= 1e-13 * scale + 1e-300)


def test_linearity_and_channel_independence():
    inst = small_workload(seed=5)
    rng = np.random.default_rng(0)
    # multiples of 1/1024 below 8 in magnitude: a f + b g is exact in float32
    g = (np.round(rng.standard_normal(inst.features.shape) * 1024) / 1024).astype(np.float32)
    f = (np.round(inst.features * 1024) / 1024).astype(np.float32)
    inst.features = f
    a, b = 0.5, -2.0
    o_f, s_f, _ = oracle.run_instance(inst)
    inst.features = g
    o_g, s_g, _ = oracle.run_instance(inst)
    inst.features = (a * f + b * g).astype(np.float32)  # exact: a, b powers of two
    o_c, _, _ = oracle.run_instance(inst)
    assert np.all(np.abs(o_c - (a * o_f + b * o_g)) <= 1e-12 * (s_f + s_g) + 1e-300)
    # changing one channel changes only that output channel
    h = f.copy()
    h[..., 2] += 1.0
    inst.features = h
    o_h, _, _ = oracle.run_instance(inst)
    others = [c for c in range(f.shape[-1]) if c != 2]
    assert np.array_equal(o_h[:, others], o_f[:, others])
    assert not np.array_equal(o_h[:, 2], o_f[:, 2])


def test_height_subset_additivity():
    inst = small_workload(seed=6, Z=5)
    out, scale, _ = oracle.run_instance(inst)
    za, zb = inst.z[[0, 2, 4]], inst.z[[1, 3]]
    inst.z = za
    oa, _, _ = oracle.run_instance(inst)
    inst.z = zb
    ob, _, _ = oracle.run_instance(inst)
    assert np.all(np.abs(out - (oa + ob)) <= 1e-13 * scale + 1e-300)


def test_batch_independence():
    inst = small_workload(seed=8, B=3)
    out, scale, _ = oracle.run_instance(inst)
    for b in range(3):
        one = synth.Instance(wl=inst.wl.with_(B=1), features=inst.features[b:b + 1].copy(),
                             lidar2img=inst.lidar2img[b:b + 1].copy(), z=inst.z)
        o1, _, _ = oracle.run_instance(one)
        assert np.array_equal(o1[0], out[b])


def test_cells_nobody_sees_are_exactly_zero():
    inst = small_workload(seed=9)
    # tilt every camera to look straight up: (x, y, z) -> depth = z - 100 < 0
    up = np.array([[1, 0, 0, 0], [0, 1, 0, 0], [0, 0, 1, -100], [0, 0, 0, 1]], np.float32)
    inst.lidar2img = np.ascontiguousarray(np.broadcast_to(up, inst.lidar2img.shape))
    out, scale, cnt = oracle.run_instance(inst)
    assert cnt["valid_samples"] == 0
    assert np.all(out == 0.0) and not np.any(np.signbit(out))


def test_empty_shapes():
    inst = small_workload(seed=10)
    inst.z = inst.z[:0]
    out, scale, cnt = oracle.run_instance(inst)
    assert np.all(out == 0.0) and cnt["valid_samples"] == 0
    wl = inst.wl.with_(X=0)
    e = synth.Instance(wl=wl, features=inst.features, lidar2img=inst.lidar2img,
                       z=synth.z_centres(-3, 2, 3))
    out, _, _ = oracle.run_instance(e)
    assert out.shape == (2, 5, 0, 5)


def test_sampled_cells_match_full_evaluation():
    inst = synth.make_workload(synth.config("tiny"))
    out, scale, _ = oracle.run_instance(inst)
    cells = np.array([[0, 0, 0], [0, 49, 49], [0, 25, 10], [0, 7, 33]])
    o, s = oracle.cells_instance(inst, cells)
    for k, (b, i, j) in enumerate(cells):
        assert np.array_equal(o[k], out[b, :, i, j])
        assert np.array_equal(s[k], scale[b, :, i, j])
