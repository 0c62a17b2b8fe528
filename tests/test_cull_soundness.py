"""Soundness of the forward's camera culling test (CPU).

The packed projection phase drops a camera for a group of BEV cells when a
conservative test shows that no height of any cell's column can pass the
mask M_n (Sec. 3.1): depth above depth_eps and the projection inside the
image.  The kernel's test (``column_may_project`` in flashbev.hip) relies on
the homogeneous coordinates being linear along a column, with margins of
2^-14 of the terms' magnitudes.  This file restates that test in float32
numpy (every operation rounded to float32, as on the GPU) and checks it
against the oracle's own projection pass on random and adversarial camera
matrices: every (cell, camera) pair the test drops must have no valid
sample at any height.  The GPU parity tests then check the compiled kernel
end to end (tests/test_gpu_parity.py::test_arbitrary_camera_matrices).
"""
import numpy as np
import pytest

import oracle

F = np.float32


def may_project(m, x, y, zlo, zhi, zabs, img_w, img_h, eps):
    """Float32 restatement of the kernel's column test; m is [..., 12]
    (rows 0-2 of lidar2img), x and y broadcast against m[..., 0]."""
    k = F(2.0 ** -14)
    tiny = F(2.0 ** -100)
    m = m.astype(F)
    x, y = F(x), F(y)
    zlo, zhi, zabs, img_w, img_h, eps = (F(v) for v in (zlo, zhi, zabs, img_w, img_h, eps))
    with np.errstate(over="ignore", invalid="ignore"):
        bu = (m[..., 0] * x + m[..., 1] * y) + m[..., 3]
        bv = (m[..., 4] * x + m[..., 5] * y) + m[..., 7]
        bd = (m[..., 8] * x + m[..., 9] * y) + m[..., 11]
        Mu = ((np.abs(m[..., 0] * x) + np.abs(m[..., 1] * y)) + np.abs(m[..., 2]) * zabs) + np.abs(m[..., 3])
        Mv = ((np.abs(m[..., 4] * x) + np.abs(m[..., 5] * y)) + np.abs(m[..., 6]) * zabs) + np.abs(m[..., 7])
        Md = ((np.abs(m[..., 8] * x) + np.abs(m[..., 9] * y)) + np.abs(m[..., 10]) * zabs) + np.abs(m[..., 11])
        u0, u1 = bu + m[..., 2] * zlo, bu + m[..., 2] * zhi
        v0, v1 = bv + m[..., 6] * zlo, bv + m[..., 6] * zhi
        d0, d1 = bd + m[..., 10] * zlo, bd + m[..., 10] * zhi
        td = eps - k * Md
        behind = (d0 < td) & (d1 < td)
        tu, tv = k * Mu, k * Mv
        left = (u0 < -tu) & (u1 < -tu) & (Mu > tiny * Md)
        top = (v0 < -tv) & (v1 < -tv) & (Mv > tiny * Md)
        tr, tb = k * (Mu + img_w * Md), k * (Mv + img_h * Md)
        right = (u0 - img_w * d0 > tr) & (u1 - img_w * d1 > tr)
        bottom = (v0 - img_h * d0 > tb) & (v1 - img_h * d1 > tb)
    return ~(behind | left | top | right | bottom)


def random_matrices(rng, N, img_h, img_w):
    """Pinhole cameras in arbitrary orientations and places: any rotation,
    positions within +-20 m, focal lengths from 0.2 to 3 image widths and
    principal points anywhere from off-image to off-image."""
    out = np.zeros((N, 4, 4), np.float64)
    for n in range(N):
        q = rng.standard_normal(4)
        q /= np.linalg.norm(q)
        a, b, c, d = q
        R = np.array([[a * a + b * b - c * c - d * d, 2 * (b * c - a * d), 2 * (b * d + a * c)],
                      [2 * (b * c + a * d), a * a - b * b + c * c - d * d, 2 * (c * d - a * b)],
                      [2 * (b * d - a * c), 2 * (c * d + a * b), a * a - b * b - c * c + d * d]])
        t = rng.uniform(-20.0, 20.0, 3)
        fx, fy = rng.uniform(0.2, 3.0, 2) * img_w
        cx, cy = rng.uniform(-0.5, 1.5) * img_w, rng.uniform(-0.5, 1.5) * img_h
        K = np.array([[fx, 0, cx], [0, fy, cy], [0, 0, 1.0]])
        out[n, :3, :3] = K @ R
        out[n, :3, 3] = -K @ R @ t
        out[n, 3, 3] = 1.0
    return out.astype(np.float32)


def ring_matrices(N, img_h, img_w):
    """The benchmark's ring rig (no jitter): yaw n 360/N, 1.5 m high."""
    out = np.zeros((N, 4, 4), np.float64)
    K = np.array([[0.75 * img_w, 0, img_w / 2], [0, 0.75 * img_w, img_h / 2], [0, 0, 1.0]])
    axes = np.array([[0, -1, 0], [0, 0, -1], [1, 0, 0]], np.float64)  # ego -> camera (x fwd)
    for n in range(N):
        yaw = 2 * np.pi * n / N
        Rz = np.array([[np.cos(yaw), -np.sin(yaw), 0], [np.sin(yaw), np.cos(yaw), 0], [0, 0, 1]])
        R = axes @ Rz.T
        t = np.array([np.cos(yaw), np.sin(yaw), 1.5])
        out[n, :3, :3] = K @ R
        out[n, :3, 3] = -K @ R @ t
        out[n, 3, 3] = 1.0
    return out.astype(np.float32)


def check(l2i, z, X, Y, half, img_h, img_w, eps=1e-5):
    N = l2i.shape[0]
    dx = np.float32(2 * half / X)
    mask, _, _ = oracle.project(l2i[None], z, (8, 8), (img_h, img_w), 1, N, X, Y,
                                -half, float(dx), -half, float(dx), eps)
    seen = mask[0].any(axis=2)                                     # [X, Y, N]
    zz = np.asarray(z, np.float32)
    zlo, zhi = zz.min(), zz.max()
    zabs = max(abs(zlo), abs(zhi))
    # cell centres as the kernel forms them (float32, x_min + (i + 1/2) dx)
    i = np.arange(X, dtype=np.float32)
    xs = np.float32(-half) + (i + np.float32(0.5)) * dx
    ys = np.float32(-half) + (np.arange(Y, dtype=np.float32) + np.float32(0.5)) * dx
    m = l2i[:, :3, :].reshape(N, 12)
    keep = np.zeros((X, Y, N), bool)
    for a in range(X):
        for c in range(Y):
            keep[a, c] = may_project(m, xs[a], ys[c], zlo, zhi, zabs, float(img_w),
                                     float(img_h), eps)
    dropped_but_seen = seen & ~keep
    assert not dropped_but_seen.any(), np.argwhere(dropped_but_seen)[:5]
    return keep.mean(), seen.mean()


@pytest.mark.parametrize("seed", range(40))
def test_random_matrices_never_drop_a_seen_column(seed):
    rng = np.random.default_rng([8100, seed])
    img_h, img_w = (256, 704) if seed % 2 else (900, 1600)
    N = int(rng.integers(1, 9))
    Z = int(rng.integers(1, 40))
    z = np.sort(rng.uniform(-30.0, 30.0, Z)).astype(np.float32)
    if seed % 3 == 0:
        z = z[::-1].copy()          # heights in any order
    check(random_matrices(rng, N, img_h, img_w), z, 24, 20, float(rng.uniform(5.0, 80.0)),
          img_h, img_w)


def test_ring_rig_culls_most_pairs_and_never_a_seen_one():
    z = ((np.arange(8) + 0.5) * 1.0 - 5.0).astype(np.float32)
    kept, seen = check(ring_matrices(6, 256, 704), z, 40, 40, 50.0, 256, 704)
    # each cell's column is within the view of about two of the six cameras
    assert seen <= kept < 0.5, (kept, seen)


def test_degenerate_rows_and_boundary_columns():
    # a camera whose u row is zero (u' = 0: u = +0 or -0, both pass u >= 0),
    # one looking straight down, and one at the grid's own height
    l2i = np.zeros((3, 4, 4), np.float32)
    l2i[0, 0] = [0, 0, 0, 0]
    l2i[0, 1] = [0, 500, 0, 128]
    l2i[0, 2] = [1, 0, 0, 0]
    l2i[1, 0] = [500, 0, 352, 0]
    l2i[1, 1] = [0, 500, 128, 0]
    l2i[1, 2] = [0, 0, -1, 10]
    l2i[2, :3] = np.array([[352, -500, 0, 0], [128, 0, -500, 0], [1, 0, 0, 0]], np.float32)
    l2i[:, 3, 3] = 1
    z = np.array([-5.0, -1.0, 0.0, 2.0], np.float32)
    check(l2i, z, 30, 30, 30.0, 256, 704)
