"""CPU oracle for the fused Sampling-VT operator (Eq. 1 of the FlashBEV paper).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The GPU library never imports,
links or calls anything here, and nothing here imports the GPU library.

The arithmetic lives in ``flashbev_oracle.c`` (plain C, float64
accumulation); this module only marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

from . import build as _build

_LIB = None


class Problem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("N", ctypes.c_int32), ("H", ctypes.c_int32),
        ("W", ctypes.c_int32), ("C", ctypes.c_int32),
        ("img_h", ctypes.c_int32), ("img_w", ctypes.c_int32),
        ("X", ctypes.c_int32), ("Y", ctypes.c_int32), ("Z", ctypes.c_int32),
        ("x_min", ctypes.c_float), ("dx", ctypes.c_float),
        ("y_min", ctypes.c_float), ("dy", ctypes.c_float),
        ("depth_eps", ctypes.c_float), ("reduce", ctypes.c_int32),
    ]


class Counters(ctypes.Structure):
    _fields_ = [("valid_samples", ctypes.c_int64), ("taps", ctypes.c_int64)]


REDUCE = {"mean": 0, "sum": 1}


def lib():
    """Load ``liboracle.so``, building it first only if it is absent."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        P = ctypes.POINTER
        L.oracle_sample_vt.argtypes = [P(Problem), ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       P(Counters), ctypes.c_int]
        L.oracle_sample_vt.restype = ctypes.c_int
        L.oracle_sample_cells.argtypes = [P(Problem), ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        L.oracle_sample_cells.restype = ctypes.c_int
        L.oracle_project.argtypes = [P(Problem), ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.oracle_project.restype = ctypes.c_int
        L.oracle_sample_vt_backward.argtypes = [P(Problem), ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        L.oracle_sample_vt_backward.restype = ctypes.c_int
        _LIB = L
    return _LIB


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def problem(features: np.ndarray, img_hw: Tuple[int, int], X: int, Y: int, Z: int,
            x_min: float, dx: float, y_min: float, dy: float, depth_eps: float = 1e-5,
            reduce: str = "mean") -> Problem:
    B, N, H, W, C = features.shape
    return Problem(B, N, H, W, C, int(img_hw[0]), int(img_hw[1]), X, Y, Z,
                   float(x_min), float(dx), float(y_min), float(dy), float(depth_eps),
                   REDUCE[reduce])


def _prep(features, lidar2img, z):
    f = np.ascontiguousarray(features, dtype=np.float32)
    m = np.ascontiguousarray(lidar2img, dtype=np.float32)
    zz = np.ascontiguousarray(z, dtype=np.float32)
    assert f.ndim == 5 and m.shape == (f.shape[0], f.shape[1], 4, 4)
    return f, m, zz


def sample_vt(features: np.ndarray, lidar2img: np.ndarray, z: np.ndarray,
              img_hw: Tuple[int, int], X: int, Y: int, x_min: float, dx: float,
              y_min: float, dy: float, depth_eps: float = 1e-5, reduce: str = "mean",
              nthreads: int = 0):
    """Eq. 1 on the CPU.

    Returns ``(out, scale, counters)``: ``out`` and ``scale`` are float64
    ``[B, C, X, Y]``; ``scale`` is the per-element magnitude scale S (the sum
    of |weighted terms|) used for tolerances; ``counters`` is a dict with the
    number of valid samples and in-range taps.
    """
    f, m, zz = _prep(features, lidar2img, z)
    p = problem(f, img_hw, X, Y, len(zz), x_min, dx, y_min, dy, depth_eps, reduce)
    B, N, H, W, C = f.shape
    out = np.empty((B, C, X, Y), dtype=np.float64)
    scale = np.empty_like(out)
    cnt = Counters()
    rc = lib().oracle_sample_vt(ctypes.byref(p), _ptr(f), _ptr(m), _ptr(zz), _ptr(out),
                                _ptr(scale), ctypes.byref(cnt), int(nthreads))
    if rc:
        raise ValueError(f"oracle_sample_vt failed: {rc}")
    return out, scale, {"valid_samples": int(cnt.valid_samples), "taps": int(cnt.taps)}


def sample_cells(features, lidar2img, z, img_hw, X, Y, x_min, dx, y_min, dy, cells,
                 depth_eps: float = 1e-5, reduce: str = "mean", nthreads: int = 0):
    """Eq. 1 for selected cells; ``cells`` is [K, 3] (b, i, j).

    Returns ``(out, scale)`` as float64 [K, C].
    """
    f, m, zz = _prep(features, lidar2img, z)
    cl = np.ascontiguousarray(cells, dtype=np.int32).reshape(-1, 3)
    p = problem(f, img_hw, X, Y, len(zz), x_min, dx, y_min, dy, depth_eps, reduce)
    C = f.shape[4]
    out = np.empty((cl.shape[0], C), dtype=np.float64)
    scale = np.empty_like(out)
    rc = lib().oracle_sample_cells(ctypes.byref(p), _ptr(f), _ptr(m), _ptr(zz), _ptr(cl),
                                   int(cl.shape[0]), _ptr(out), _ptr(scale), int(nthreads))
    if rc:
        raise ValueError(f"oracle_sample_cells failed: {rc}")
    return out, scale


def project(lidar2img, z, feat_hw, img_hw, B, N, X, Y, x_min, dx, y_min, dy,
            depth_eps: float = 1e-5):
    """Projection-only pass: ``(mask, x_f, y_f)``, each [B, X, Y, Z, N]."""
    m = np.ascontiguousarray(lidar2img, dtype=np.float32)
    zz = np.ascontiguousarray(z, dtype=np.float32)
    H, W = feat_hw
    p = Problem(B, N, H, W, 1, int(img_hw[0]), int(img_hw[1]), X, Y, len(zz),
                float(x_min), float(dx), float(y_min), float(dy), float(depth_eps), 0)
    shape = (B, X, Y, len(zz), N)
    mask = np.empty(shape, dtype=np.uint8)
    xf = np.empty(shape, dtype=np.float32)
    yf = np.empty(shape, dtype=np.float32)
    rc = lib().oracle_project(ctypes.byref(p), _ptr(m), _ptr(zz), _ptr(mask), _ptr(xf), _ptr(yf))
    if rc:
        raise ValueError(f"oracle_project failed: {rc}")
    return mask.astype(bool), xf, yf


def run_instance(inst, reduce: str = "mean", nthreads: int = 0):
    """Oracle on a ``synth.Instance``."""
    wl = inst.wl
    return sample_vt(inst.features, inst.lidar2img, inst.z, (wl.img_h, wl.img_w), wl.X, wl.Y,
                     wl.x_min, wl.dx, wl.y_min, wl.dy, wl.depth_eps, reduce, nthreads)


def cells_instance(inst, cells, reduce: str = "mean", nthreads: int = 0):
    """Oracle on selected cells of a ``synth.Instance``."""
    wl = inst.wl
    return sample_cells(inst.features, inst.lidar2img, inst.z, (wl.img_h, wl.img_w), wl.X,
                        wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy, cells, wl.depth_eps, reduce,
                        nthreads)


def sample_vt_backward(grad_out: np.ndarray, lidar2img: np.ndarray, z: np.ndarray,
                       feat_shape, img_hw: Tuple[int, int], x_min: float, dx: float,
                       y_min: float, dy: float, depth_eps: float = 1e-5,
                       reduce: str = "mean", nthreads: int = 0):
    """Gradient of Eq. 1 with respect to the feature maps, on the CPU.

    ``grad_out`` is float32 ``[B, C, X, Y]``; ``feat_shape`` is
    ``(B, N, H, W, C)``.  Returns ``(grad_feat, scale, terms)``:
    ``grad_feat`` and ``scale`` are float64 ``[B, N, H, W, C]`` (``scale``
    is the sum of |terms| per element), ``terms`` is int32 ``[B, N, H, W]``,
    the number of (sample, tap) terms that reach each pixel.
    """
    g = np.ascontiguousarray(grad_out, dtype=np.float32)
    m = np.ascontiguousarray(lidar2img, dtype=np.float32)
    zz = np.ascontiguousarray(z, dtype=np.float32)
    B, N, H, W, C = (int(v) for v in feat_shape)
    assert g.ndim == 4 and g.shape[:2] == (B, C) and m.shape == (B, N, 4, 4)
    X, Y = g.shape[2], g.shape[3]
    p = Problem(B, N, H, W, C, int(img_hw[0]), int(img_hw[1]), X, Y, len(zz),
                float(x_min), float(dx), float(y_min), float(dy), float(depth_eps),
                REDUCE[reduce])
    grad_feat = np.empty((B, N, H, W, C), dtype=np.float64)
    scale = np.empty_like(grad_feat)
    terms = np.empty((B, N, H, W), dtype=np.int32)
    rc = lib().oracle_sample_vt_backward(ctypes.byref(p), _ptr(m), _ptr(zz), _ptr(g),
                                         _ptr(grad_feat), _ptr(scale), _ptr(terms),
                                         int(nthreads))
    if rc:
        raise ValueError(f"oracle_sample_vt_backward failed: {rc}")
    return grad_feat, scale, terms


def backward_instance(inst, grad_out, reduce: str = "mean", nthreads: int = 0):
    """Backward oracle on a ``synth.Instance`` with output gradient ``grad_out``."""
    wl = inst.wl
    return sample_vt_backward(grad_out, inst.lidar2img, inst.z, inst.features.shape,
                              (wl.img_h, wl.img_w), wl.x_min, wl.dx, wl.y_min, wl.dy,
                              wl.depth_eps, reduce, nthreads)
