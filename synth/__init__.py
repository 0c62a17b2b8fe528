"""Seeded synthetic workloads for the fused Sampling-VT operator.

This module only *generates inputs*: camera rigs (``lidar2img`` matrices),
feature maps, BEV grid specifications and height-bin centres.  It contains
none of the operator's arithmetic (no projection, masking, sampling or
reduction), so both the CPU oracle and the GPU path can consume its output
without sharing any of the method's code.

The paper benchmarks a SimpleBEV-style setting on nuScenes (Sec. 4.1): six
ring cameras, a 100 m x 100 m BEV grid of 0.5 m cells and Z height bins.
nuScenes is not used here; seeded synthetic rigs with the same geometry and
standard-normal features of the same shapes stand in for it.

Rig convention (a reading of the paper, which does not fix one):
  * ego / lidar frame: x forward, y left, z up (metres);
  * camera n sits on a ring of radius ``ring_radius`` at yaw n*360/N degrees,
    ``mount_height`` metres above the ground plane, looking outwards;
  * camera frame: OpenCV (x right, y down, z along the optical axis);
  * pinhole intrinsics fx = fy = 0.75 * image width, principal point at the
    image centre;
  * roll, pitch and yaw each jittered by U(-2, 2) degrees and the position by
    U(-0.05, 0.05) m per axis, drawn from the seed;
  * ``lidar2img = [[K R, -K R t], [0, 0, 0, 1]]`` (4x4, float32, row-major),
    so that (u', v', d) = lidar2img[:3] @ (x, y, z, 1) and the pixel is
    (u'/d, v'/d).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "Workload",
    "CONFIGS",
    "config",
    "z_centres",
    "make_rig",
    "make_features",
    "make_workload",
    "DTYPES",
    "ScaWorkload",
    "SCA_CONFIGS",
    "sca_config",
    "pillar_anchors",
    "make_sca_workload",
]

# Feature element types understood by the operator.
DTYPES = ("f32", "f16", "bf16")


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic problem instance description (shapes and grid)."""

    name: str
    cfg_id: int
    B: int
    N: int
    img_h: int
    img_w: int
    H: int  # feature-map height
    W: int  # feature-map width
    C: int
    dtype: str
    X: int
    Y: int
    x_min: float
    dx: float
    y_min: float
    dy: float
    z_lo: float
    z_hi: float
    Z: int
    ring_radius: float = 1.0
    mount_height: float = 1.5
    jitter_deg: float = 2.0
    jitter_m: float = 0.05
    depth_eps: float = 1e-5

    @property
    def samples(self) -> int:
        """Projected (point, camera) samples per call: B*X*Y*Z*N."""
        return self.B * self.X * self.Y * self.Z * self.N

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def z_centres(z_lo: float, z_hi: float, Z: int) -> np.ndarray:
    """Centres of Z equal height bins spanning [z_lo, z_hi] (float32)."""
    k = np.arange(Z, dtype=np.float64)
    return (z_lo + (k + 0.5) * (z_hi - z_lo) / Z).astype(np.float32)


def _cfg(name, cfg_id, B, N, img_hw, stride, C, dtype, XY, half_range, Z,
         z_lo=-5.0, z_hi=3.0) -> Workload:
    img_h, img_w = img_hw
    X = Y = XY
    d = 2.0 * half_range / XY
    return Workload(name=name, cfg_id=cfg_id, B=B, N=N, img_h=img_h, img_w=img_w,
                    H=img_h // stride, W=img_w // stride, C=C, dtype=dtype,
                    X=X, Y=Y, x_min=-half_range, dx=d, y_min=-half_range, dy=d,
                    z_lo=z_lo, z_hi=z_hi, Z=Z)


# The five benchmark workloads, plus the paper's own reference setting
# (Sec. 4.1: 448x800 images, stride 8 -> 56x100 maps, C=128, 200x200 over
# +-50 m, Z=8 over [-5, 5] m; N=6 as on nuScenes).
CONFIGS: Dict[str, Workload] = {
    "tiny": _cfg("tiny", 1, 1, 6, (256, 704), 16, 32, "f32", 50, 25.0, 4),
    "rep": _cfg("rep", 2, 1, 6, (256, 704), 8, 80, "f32", 200, 50.0, 8),
    "half_batch": _cfg("half_batch", 3, 4, 6, (256, 704), 8, 128, "bf16", 200, 50.0, 8),
    "long_range": _cfg("long_range", 4, 1, 6, (900, 1600), 8, 64, "f16", 400, 100.0, 16),
    "z_sweep": _cfg("z_sweep", 5, 2, 8, (256, 704), 8, 64, "bf16", 512, 64.0, 8),
    "paper_ref": _cfg("paper_ref", 6, 1, 6, (448, 800), 8, 128, "f32", 200, 50.0, 8,
                      z_lo=-5.0, z_hi=5.0),
}
Z_SWEEP = (4, 8, 16, 32, 64)


def config(name: str, **overrides) -> Workload:
    """Look up a named workload; ``overrides`` replace fields (e.g. Z=32)."""
    wl = CONFIGS[name]
    return wl.with_(**overrides) if overrides else wl


def _rot_x(a):
    c, s = math.cos(a), math.sin(a)
    return np.array([[1, 0, 0], [0, c, -s], [0, s, c]], dtype=np.float64)


def _rot_y(a):
    c, s = math.cos(a), math.sin(a)
    return np.array([[c, 0, s], [0, 1, 0], [-s, 0, c]], dtype=np.float64)


def _rot_z(a):
    c, s = math.cos(a), math.sin(a)
    return np.array([[c, -s, 0], [s, c, 0], [0, 0, 1]], dtype=np.float64)


def camera_matrix(yaw: float, position: Sequence[float], fx: float, fy: float,
                  cx: float, cy: float, jitter_rpy=(0.0, 0.0, 0.0)) -> np.ndarray:
    """4x4 float64 lidar2img for one pinhole camera looking along ``yaw``.

    ``jitter_rpy`` = (roll, pitch, yaw) in radians, applied in the camera
    frame (roll about the optical axis, pitch about camera x, yaw about
    camera y).
    """
    fwd = np.array([math.cos(yaw), math.sin(yaw), 0.0])
    up = np.array([0.0, 0.0, 1.0])
    right = np.cross(fwd, up)
    down = -up
    r_nom = np.stack([right, down, fwd])  # rows: camera axes in ego frame
    roll, pitch, yw = jitter_rpy
    r_jit = _rot_z(roll) @ _rot_x(pitch) @ _rot_y(yw)
    rot = r_jit @ r_nom
    t = np.asarray(position, dtype=np.float64)
    K = np.array([[fx, 0, cx], [0, fy, cy], [0, 0, 1]], dtype=np.float64)
    m = np.eye(4)
    m[:3, :3] = K @ rot
    m[:3, 3] = -(K @ rot @ t)
    return m


def make_rig(wl, seed: Optional[Sequence[int]] = None) -> np.ndarray:
    """Seeded ``lidar2img`` [B, N, 4, 4] float32 for a ring rig.

    Every batch element draws its own jitter (independent rigs per sample).
    ``wl`` is a :class:`Workload` or a :class:`ScaWorkload`.
    """
    rng = np.random.default_rng(list(seed) if seed is not None else [wl.cfg_id, 0])
    fx = fy = 0.75 * wl.img_w
    cx, cy = wl.img_w / 2.0, wl.img_h / 2.0
    deg = math.pi / 180.0
    out = np.empty((wl.B, wl.N, 4, 4), dtype=np.float32)
    for b in range(wl.B):
        for n in range(wl.N):
            yaw = 2.0 * math.pi * n / wl.N
            jit = rng.uniform(-wl.jitter_deg, wl.jitter_deg, size=3) * deg
            pos = np.array([wl.ring_radius * math.cos(yaw),
                            wl.ring_radius * math.sin(yaw), wl.mount_height])
            pos = pos + rng.uniform(-wl.jitter_m, wl.jitter_m, size=3)
            out[b, n] = camera_matrix(yaw, pos, fx, fy, cx, cy, tuple(jit)).astype(np.float32)
    return out


def make_features(wl: Workload, seed: Optional[Sequence[int]] = None) -> np.ndarray:
    """Seeded standard-normal features, NHWC [B, N, H, W, C], float32.

    For 16-bit workloads the values are rounded once to the storage type
    (round-to-nearest-even) and returned as the exact float32 upcast of the
    rounded values; use :func:`to_storage` to get the 16-bit tensor.
    """
    rng = np.random.default_rng(list(seed) if seed is not None else [wl.cfg_id, 1])
    f = rng.standard_normal((wl.B, wl.N, wl.H, wl.W, wl.C), dtype=np.float32)
    if wl.dtype == "f32":
        return f
    return round_to(f, wl.dtype)


def round_to(f32: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to ``dtype`` (RNE) and return the float32 upcast."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(f32, dtype=np.float32))
    if dtype == "f32":
        return t.numpy().copy()
    tdt = {"f16": torch.float16, "bf16": torch.bfloat16}[dtype]
    return t.to(tdt).to(torch.float32).numpy()


def to_storage(f32: np.ndarray, dtype: str):
    """torch CPU tensor in the storage dtype holding exactly ``f32``'s values."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(f32, dtype=np.float32))
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dtype]
    return t.to(tdt)


@dataclasses.dataclass
class Instance:
    """Concrete inputs for one workload."""

    wl: Workload
    features: np.ndarray  # [B,N,H,W,C] float32 (exact values of the storage dtype)
    lidar2img: np.ndarray  # [B,N,4,4] float32
    z: np.ndarray  # [Z] float32

    def grid(self) -> dict:
        wl = self.wl
        return dict(x_min=wl.x_min, dx=wl.dx, X=wl.X, y_min=wl.y_min, dy=wl.dy, Y=wl.Y,
                    depth_eps=wl.depth_eps)


def make_workload(wl: Workload, rig_seed=None, feat_seed=None) -> Instance:
    """Rig, features and height centres for ``wl``."""
    return Instance(wl=wl, features=make_features(wl, feat_seed),
                    lidar2img=make_rig(wl, rig_seed),
                    z=z_centres(wl.z_lo, wl.z_hi, wl.Z))


def all_parity_workloads() -> List[Workload]:
    """The five benchmark workloads, with every Z of the height sweep."""
    out = [CONFIGS["tiny"], CONFIGS["rep"], CONFIGS["half_batch"], CONFIGS["long_range"]]
    out += [CONFIGS["z_sweep"].with_(Z=z) for z in Z_SWEEP]
    return out


# ---------------------------------------------------------------------------
# FlashSCA (BEVFormer spatial cross-attention) inputs.
#
# The paper measures FlashSCA at BEVFormer-base defaults (Sec. 4.5, Table 7):
# N=6 cameras, C=256, 8 heads, L=4 levels, BEV 200x200, Z=4 anchors and
# P in {8, 16, 32} points.  BEVFormer-base takes 900x1600 images padded to
# 928x1600 and a feature pyramid of strides 8, 16, 32, 64 (116x200, 58x100,
# 29x50, 15x25); its BEV spans +-51.2 m (0.512 m cells) and its pillars
# [-5, 3] m.  No trained weights or nuScenes data are used: the value maps
# are standard normal (the output of a value projection), the attention
# logits standard normal, and the sampling offsets follow the initial
# pattern of BEVFormer's offset predictor (head m points along angle
# 2 pi m / heads, point k at distance k + 1 pixels, on the square of the
# direction's largest component) plus N(0, 1) pixel noise per component.
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class ScaWorkload:
    """One synthetic FlashSCA problem description."""

    name: str
    cfg_id: int
    B: int
    N: int
    img_h: int
    img_w: int
    levels: Tuple[Tuple[int, int], ...]  # (H_l, W_l) per level
    C: int
    heads: int
    P: int  # sampling points per (head, level)
    Z: int  # pillar anchors
    dtype: str
    X: int
    Y: int
    x_min: float
    dx: float
    y_min: float
    dy: float
    z_lo: float = -5.0
    z_hi: float = 3.0
    offset_noise: float = 1.0
    ring_radius: float = 1.0
    mount_height: float = 1.5
    jitter_deg: float = 2.0
    jitter_m: float = 0.05
    depth_eps: float = 1e-5

    @property
    def L(self) -> int:
        return len(self.levels)

    @property
    def Q(self) -> int:
        return self.X * self.Y

    @property
    def S(self) -> int:
        """Value pixels per camera over all levels."""
        return sum(h * w for h, w in self.levels)

    def with_(self, **kw) -> "ScaWorkload":
        return dataclasses.replace(self, **kw)


def pillar_anchors(z_lo: float, z_hi: float, Z: int) -> np.ndarray:
    """Z anchor heights spread evenly from 0.5 m above the bottom of the
    pillar [z_lo, z_hi] to 0.5 m below its top (float32), as BEVFormer
    places its pillar points."""
    if Z == 1:
        return np.array([0.5 * (z_lo + z_hi)], dtype=np.float32)
    k = np.arange(Z, dtype=np.float64)
    return (z_lo + 0.5 + k * ((z_hi - z_lo) - 1.0) / (Z - 1)).astype(np.float32)


_BEVFORMER_LEVELS = ((116, 200), (58, 100), (29, 50), (15, 25))


def _sca(name, cfg_id, B, N, img_hw, levels, C, heads, P, Z, dtype, XY, half_range, **kw):
    d = 2.0 * half_range / XY
    return ScaWorkload(name=name, cfg_id=cfg_id, B=B, N=N, img_h=img_hw[0], img_w=img_hw[1],
                       levels=tuple(levels), C=C, heads=heads, P=P, Z=Z, dtype=dtype, X=XY,
                       Y=XY, x_min=-half_range, dx=d, y_min=-half_range, dy=d, **kw)


SCA_CONFIGS: Dict[str, ScaWorkload] = {
    # several tiles and a ragged tail, small enough for pure-Python checks
    "sca_tiny": _sca("sca_tiny", 101, 1, 6, (256, 704), ((16, 44), (8, 22)), 32, 4, 4, 2,
                     "f32", 23, 25.0),
    # BEVFormer-base defaults (Table 7), P = 8
    "sca_base": _sca("sca_base", 102, 1, 6, (900, 1600), _BEVFORMER_LEVELS, 256, 8, 8, 4,
                     "f32", 200, 51.2),
    # the same at half precision storage, two batch elements
    "sca_base_bf16": _sca("sca_base_bf16", 103, 2, 6, (900, 1600), _BEVFORMER_LEVELS, 256, 8,
                          8, 4, "bf16", 200, 51.2),
}
SCA_P_SWEEP = (8, 16, 32)


def sca_config(name: str, **overrides) -> ScaWorkload:
    wl = SCA_CONFIGS[name]
    return wl.with_(**overrides) if overrides else wl


@dataclasses.dataclass
class ScaInstance:
    """Concrete FlashSCA inputs."""

    wl: ScaWorkload
    value: np.ndarray  # [B, N, S, C] float32 (exact values of the storage dtype)
    lidar2img: np.ndarray  # [B, N, 4, 4] float32
    z: np.ndarray  # [Z] float32 anchor heights
    offsets: np.ndarray  # [B, Q, heads, L, P, 2] float32, level pixels (x, y)
    logits: np.ndarray  # [B, Q, heads, L, P] float32


def sca_offsets(wl: ScaWorkload, rng) -> np.ndarray:
    """Offsets in the initial pattern of BEVFormer's offset predictor, plus noise."""
    H, L, P = wl.heads, wl.L, wl.P
    theta = 2.0 * math.pi * np.arange(H) / H
    g = np.stack([np.cos(theta), np.sin(theta)], axis=-1)  # [H, 2]
    g = g / np.abs(g).max(axis=-1, keepdims=True)
    base = g[:, None, None, :] * (np.arange(P) + 1.0)[None, None, :, None]  # [H, 1, P, 2]
    base = np.broadcast_to(base, (H, L, P, 2))
    noise = rng.standard_normal((wl.B, wl.Q, H, L, P, 2)) * wl.offset_noise
    return (base[None, None] + noise).astype(np.float32)


def make_sca_workload(wl: ScaWorkload, seed: Optional[Sequence[int]] = None) -> ScaInstance:
    """Rig, value maps, anchors, offsets and logits for ``wl``."""
    base = list(seed) if seed is not None else [wl.cfg_id]
    rng = np.random.default_rng(base + [1])
    v = rng.standard_normal((wl.B, wl.N, wl.S, wl.C), dtype=np.float32)
    if wl.dtype != "f32":
        v = round_to(v, wl.dtype)
    rng2 = np.random.default_rng(base + [2])
    offsets = sca_offsets(wl, rng2)
    logits = rng2.standard_normal((wl.B, wl.Q, wl.heads, wl.L, wl.P), dtype=np.float32)
    return ScaInstance(wl=wl, value=v, lidar2img=make_rig(wl, base + [0]),
                       z=pillar_anchors(wl.z_lo, wl.z_hi, wl.Z), offsets=offsets,
                       logits=logits)
