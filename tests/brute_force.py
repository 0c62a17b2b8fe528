"""Tensorized Sampling-VT in numpy: the staged evaluation of Alg. 1.

Test infrastructure.  Written independently of the C oracle, it follows the
six stages of the paper's tensorized baseline (Sec. 3.2.1, Alg. 1) and
materializes every intermediate the paper lists:

  1. voxel grid                      (B, X, Y, Z, 3)
  2. projected coordinates           (B, N, X, Y, Z, 3)
  3. Features3D                      (B, N, C, X, Y, Z)
  4. validity mask and masked Features3D
  5. valid camera mean G             (B, C, X, Y, Z)
  6. height sum                      (B, C, X, Y)

Coordinates use the same float32 recipe as the oracle (each product and sum
rounded on its own, IEEE float32 division); sampling and reductions are
float64.  Memory grows as B*N*C*X*Y*Z, so only tiny shapes are evaluated.
"""
from __future__ import annotations

import numpy as np

f32 = np.float32


def tensorized_sample_vt(features, lidar2img, z, img_hw, X, Y, x_min, dx, y_min, dy,
                         depth_eps=1e-5, reduce="mean"):
    feat = np.asarray(features, dtype=np.float32)
    P = np.asarray(lidar2img, dtype=np.float32)
    zz = np.asarray(z, dtype=np.float32)
    B, N, H, W, C = feat.shape
    Z = zz.shape[0]
    img_h, img_w = img_hw

    # 1. voxel grid (B, X, Y, Z, 3): cell centres, float32
    xs = f32(x_min) + (np.arange(X, dtype=np.float32) + f32(0.5)) * f32(dx)
    ys = f32(y_min) + (np.arange(Y, dtype=np.float32) + f32(0.5)) * f32(dy)
    vox = np.empty((B, X, Y, Z, 3), dtype=np.float32)
    vox[..., 0] = xs[None, :, None, None]
    vox[..., 1] = ys[None, None, :, None]
    vox[..., 2] = zz[None, None, None, :]

    # 2. projection of every voxel into every camera (B, N, X, Y, Z, 3)
    proj = np.empty((B, N, X, Y, Z, 3), dtype=np.float32)
    vx = vox[:, None, ..., 0]
    vy = vox[:, None, ..., 1]
    vz = vox[:, None, ..., 2]
    for r in range(3):
        m = P[:, :, r, :].reshape(B, N, 1, 1, 1, 4)
        t0 = m[..., 0] * vx
        t1 = m[..., 1] * vy
        t2 = m[..., 2] * vz
        proj[..., r] = ((t0 + t1) + t2) + m[..., 3]
    d = proj[..., 2]
    positive = d > f32(depth_eps)
    safe_d = np.where(positive, d, f32(1.0))
    u = proj[..., 0] / safe_d
    v = proj[..., 1] / safe_d

    # 4 (mask part). M = positive depth and inside the image
    mask = positive & (u >= 0) & (u < f32(img_w)) & (v >= 0) & (v < f32(img_h))

    # 3. Features3D (B, N, C, X, Y, Z): bilinear samples, zero padding
    sx = f32(W) / f32(img_w)
    sy = f32(H) / f32(img_h)
    xf = u * sx - f32(0.5)
    yf = v * sy - f32(0.5)
    xf = np.where(mask, xf, f32(0.0))
    yf = np.where(mask, yf, f32(0.0))
    x0 = np.floor(xf)
    y0 = np.floor(yf)
    ax = (xf - x0).astype(np.float64)
    ay = (yf - y0).astype(np.float64)
    x0 = x0.astype(np.int64)
    y0 = y0.astype(np.int64)
    bi = np.arange(B).reshape(B, 1, 1, 1, 1)
    ni = np.arange(N).reshape(1, N, 1, 1, 1)
    feat64 = feat.astype(np.float64)
    features3d = np.zeros((B, N, C, X, Y, Z), dtype=np.float64)
    for ty in (0, 1):
        for tx in (0, 1):
            xt = x0 + tx
            yt = y0 + ty
            inr = (xt >= 0) & (xt < W) & (yt >= 0) & (yt < H)
            w = (ax if tx else 1.0 - ax) * (ay if ty else 1.0 - ay)
            w = np.where(inr, w, 0.0)
            g = feat64[bi, ni, np.clip(yt, 0, H - 1), np.clip(xt, 0, W - 1)]  # (B,N,X,Y,Z,C)
            features3d += np.moveaxis(g * w[..., None], -1, 2)

    # 4. masked Features3D
    masked = features3d * mask[:, :, None].astype(np.float64)

    # 5. valid camera mean G = num_z / max(1, den_z), (B, C, X, Y, Z)
    num = masked.sum(axis=1)
    den = mask.sum(axis=1).astype(np.float64)  # (B, X, Y, Z)
    if reduce == "mean":
        G = num / np.maximum(1.0, den)[:, None]
    else:
        G = num

    # 6. height sum
    return G.sum(axis=-1)


def run_instance(inst, reduce="mean"):
    wl = inst.wl
    return tensorized_sample_vt(inst.features, inst.lidar2img, inst.z, (wl.img_h, wl.img_w),
                                wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy, wl.depth_eps,
                                reduce)
