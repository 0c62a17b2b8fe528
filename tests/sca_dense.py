"""BEVFormer's dense per-camera SCA path, in plain PyTorch float64 on the CPU.

An independent formulation used to pin the FlashSCA oracle.  It follows the
structure the paper's baseline mirrors (Sec. 4.5): project every pillar
anchor into every camera, build the full sampling-location tensor
[B, N, Q, heads, L, P, 2] (the tensor FlashSCA never materializes), sample
each level with ``torch.nn.functional.grid_sample`` (bilinear, zero padding,
align_corners=False), weight by the softmax over (level, point), keep the
cameras a query hits and divide by their number.  Everything is float64:
projections, masks, locations, sampling and sums.  It shares no code with
the oracle.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def anchors_in_cameras(lidar2img, z, X, Y, x_min, dx, y_min, dy, img_hw, eps=1e-5):
    """Normalized reference points and masks in float64.

    Returns ``(ref [B, N, Q, Z, 2], valid [B, N, Q, Z], depth [B, N, Q, Z])``
    with query q = i * Y + j.
    """
    m = torch.from_numpy(np.asarray(lidar2img, dtype=np.float64))
    zz = torch.from_numpy(np.asarray(z, dtype=np.float64))
    xs = x_min + (torch.arange(X, dtype=torch.float64) + 0.5) * dx
    ys = y_min + (torch.arange(Y, dtype=torch.float64) + 0.5) * dy
    gx, gy = torch.meshgrid(xs, ys, indexing="ij")                  # [X, Y]
    Z = zz.numel()
    pts = torch.stack([gx.reshape(-1, 1).expand(-1, Z), gy.reshape(-1, 1).expand(-1, Z),
                       zz.view(1, Z).expand(X * Y, Z), torch.ones(X * Y, Z, dtype=torch.float64)],
                      dim=-1)                                         # [Q, Z, 4]
    cam = torch.einsum("bnrc,qzc->bnqzr", m, pts)                   # [B, N, Q, Z, 4]
    depth = cam[..., 2]
    uv = cam[..., :2] / torch.clamp(depth, min=eps)[..., None]
    img_h, img_w = img_hw
    ref = torch.stack([uv[..., 0] / img_w, uv[..., 1] / img_h], dim=-1)
    valid = ((depth > eps) & (ref[..., 0] > 0) & (ref[..., 0] < 1) & (ref[..., 1] > 0)
             & (ref[..., 1] < 1))
    return ref, valid, depth


def dense_sca(value, lidar2img, z, offsets, logits, levels, heads, img_hw, X, Y, x_min, dx,
              y_min, dy, eps=1e-5, reduce="mean"):
    """out [B, Q, C] float64 numpy, plus the hit mask [B, N, Q] and reference points."""
    v = torch.from_numpy(np.asarray(value, dtype=np.float64))
    off = torch.from_numpy(np.asarray(offsets, dtype=np.float64))
    lg = torch.from_numpy(np.asarray(logits, dtype=np.float64))
    B, N, S, C = v.shape
    D = C // heads
    L = len(levels)
    P = lg.shape[-1]
    Z = len(z)
    Q = X * Y
    ref, valid, _ = anchors_in_cameras(lidar2img, z, X, Y, x_min, dx, y_min, dy, img_hw, eps)
    hit = valid.any(dim=-1)                                          # [B, N, Q]
    count = hit.sum(dim=1).clamp(min=1).to(torch.float64)           # [B, Q]
    # sampling locations of every camera: [B, N, Q, heads, L, P/Z, Z, 2] -> P
    norm = torch.tensor([[w, h] for h, w in levels], dtype=torch.float64)  # [L, 2]
    off_n = off.view(B, 1, Q, heads, L, P // Z, Z, 2) / norm.view(1, 1, 1, 1, L, 1, 1, 2)
    loc = ref.view(B, N, Q, 1, 1, 1, Z, 2) + off_n
    loc = loc.reshape(B, N, Q, heads, L, P, 2)
    attn = torch.softmax(lg.view(B, Q, heads, L * P), dim=-1).view(B, Q, heads, L, P)
    out = torch.zeros(B, Q, C, dtype=torch.float64)
    start = 0
    for l, (hl, wl) in enumerate(levels):
        for n in range(N):
            vl = v[:, n, start:start + hl * wl, :].reshape(B, hl, wl, heads, D)
            vl = vl.permute(0, 3, 4, 1, 2).reshape(B * heads, D, hl, wl)
            grid = 2.0 * loc[:, n, :, :, l] - 1.0                    # [B, Q, heads, P, 2]
            grid = grid.permute(0, 2, 1, 3, 4).reshape(B * heads, Q, P, 2)
            samp = F.grid_sample(vl, grid, mode="bilinear", padding_mode="zeros",
                                 align_corners=False)                  # [B*heads, D, Q, P]
            w = attn[:, :, :, l, :].permute(0, 2, 1, 3).reshape(B * heads, 1, Q, P)
            contrib = (samp * w).sum(dim=-1).view(B, heads, D, Q).permute(0, 3, 1, 2)
            out += contrib.reshape(B, Q, C) * hit[:, n, :, None]
        start += hl * wl
    if reduce == "mean":
        out = out / count[..., None]
    return out.numpy(), hit.numpy(), ref.numpy()


def robust_queries(lidar2img, z, X, Y, x_min, dx, y_min, dy, img_hw, eps=1e-5, margin=1e-5):
    """[B, Q] bool: queries none of whose anchors lies within ``margin``
    (relative) of an image border or of the depth threshold, in any camera.
    Their hit decisions cannot depend on float32 versus float64 rounding."""
    ref, _, depth = anchors_in_cameras(lidar2img, z, X, Y, x_min, dx, y_min, dy, img_hw, eps)
    near = (depth - eps).abs() < margin * (1.0 + depth.abs())
    for k in range(2):
        r = ref[..., k]
        near |= (depth > eps) & ((r.abs() < margin) | ((r - 1.0).abs() < margin))
    return ~(near.any(dim=-1).any(dim=1)).numpy()                   # [B, Q]


def dense_sca_grads(value, lidar2img, z, offsets, logits, grad_out, levels, heads, img_hw, X, Y,
                    x_min, dx, y_min, dy, eps=1e-5, reduce="mean"):
    """Gradients of the dense path (torch autograd through grid_sample and
    softmax, float64) with respect to value, offsets and logits, for output
    gradient ``grad_out``; also the float64 sampling locations in level
    pixels [B, N, Q, heads, L, P, 2] and the hit mask [B, N, Q]."""
    v = torch.from_numpy(np.asarray(value, dtype=np.float64)).requires_grad_(True)
    off = torch.from_numpy(np.asarray(offsets, dtype=np.float64)).requires_grad_(True)
    lg = torch.from_numpy(np.asarray(logits, dtype=np.float64)).requires_grad_(True)
    g = torch.from_numpy(np.asarray(grad_out, dtype=np.float64))
    B, N, S, C = v.shape
    D = C // heads
    L = len(levels)
    P = lg.shape[-1]
    Z = len(z)
    Q = X * Y
    ref, valid, _ = anchors_in_cameras(lidar2img, z, X, Y, x_min, dx, y_min, dy, img_hw, eps)
    hit = valid.any(dim=-1)
    count = hit.sum(dim=1).clamp(min=1).to(torch.float64)
    norm = torch.tensor([[w, h] for h, w in levels], dtype=torch.float64)
    off_n = off.view(B, 1, Q, heads, L, P // Z, Z, 2) / norm.view(1, 1, 1, 1, L, 1, 1, 2)
    loc = (ref.view(B, N, Q, 1, 1, 1, Z, 2) + off_n).reshape(B, N, Q, heads, L, P, 2)
    attn = torch.softmax(lg.view(B, Q, heads, L * P), dim=-1).view(B, Q, heads, L, P)
    out = torch.zeros(B, Q, C, dtype=torch.float64)
    start = 0
    for l, (hl, wl) in enumerate(levels):
        for n in range(N):
            vl = v[:, n, start:start + hl * wl, :].reshape(B, hl, wl, heads, D)
            vl = vl.permute(0, 3, 4, 1, 2).reshape(B * heads, D, hl, wl)
            grid = (2.0 * loc[:, n, :, :, l] - 1.0).permute(0, 2, 1, 3, 4).reshape(B * heads, Q, P, 2)
            samp = F.grid_sample(vl, grid, mode="bilinear", padding_mode="zeros",
                                 align_corners=False)
            w = attn[:, :, :, l, :].permute(0, 2, 1, 3).reshape(B * heads, 1, Q, P)
            contrib = (samp * w).sum(dim=-1).view(B, heads, D, Q).permute(0, 3, 1, 2)
            out = out + contrib.reshape(B, Q, C) * hit[:, n, :, None]
        start += hl * wl
    if reduce == "mean":
        out = out / count[..., None]
    (out * g).sum().backward()
    pix = loc.detach() * norm.view(1, 1, 1, 1, L, 1, 2) - 0.5
    return (v.grad.numpy(), off.grad.numpy(), lg.grad.numpy(), pix.numpy(), hit.numpy())
