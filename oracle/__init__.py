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


# ---------------------------------------------------------------------------
# FlashSCA (BEVFormer spatial cross-attention), flashsca_oracle.c
# ---------------------------------------------------------------------------

SCA_LMAX = 8


class ScaProblem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("N", ctypes.c_int32), ("C", ctypes.c_int32),
        ("heads", ctypes.c_int32), ("L", ctypes.c_int32), ("P", ctypes.c_int32),
        ("Z", ctypes.c_int32),
        ("level_h", ctypes.c_int32 * SCA_LMAX), ("level_w", ctypes.c_int32 * SCA_LMAX),
        ("img_h", ctypes.c_int32), ("img_w", ctypes.c_int32),
        ("X", ctypes.c_int32), ("Y", ctypes.c_int32),
        ("x_min", ctypes.c_float), ("dx", ctypes.c_float),
        ("y_min", ctypes.c_float), ("dy", ctypes.c_float),
        ("depth_eps", ctypes.c_float), ("reduce", ctypes.c_int32),
    ]


class ScaCounters(ctypes.Structure):
    _fields_ = [("hits", ctypes.c_int64), ("taps", ctypes.c_int64)]


def _sca_lib(path: Optional[str] = None):
    """The oracle library (or, for the mutant tests, another build of it)."""
    L = lib() if path is None else ctypes.CDLL(path)
    P = ctypes.POINTER
    L.sca_oracle_forward.argtypes = [P(ScaProblem)] + [ctypes.c_void_p] * 8 + [
        P(ScaCounters), ctypes.c_int]
    L.sca_oracle_forward.restype = ctypes.c_int
    L.sca_oracle_reference_points.argtypes = [P(ScaProblem)] + [ctypes.c_void_p] * 6
    L.sca_oracle_reference_points.restype = ctypes.c_int
    L.sca_oracle_backward.argtypes = [P(ScaProblem)] + [ctypes.c_void_p] * 14 + [ctypes.c_int]
    L.sca_oracle_backward.restype = ctypes.c_int
    return L


def sca_problem(B, N, C, heads, levels, P, Z, img_hw, X, Y, x_min, dx, y_min, dy,
                depth_eps=1e-5, reduce="mean") -> ScaProblem:
    L = len(levels)
    assert 1 <= L <= SCA_LMAX
    lh = (ctypes.c_int32 * SCA_LMAX)(*[int(h) for h, _ in levels], *([0] * (SCA_LMAX - L)))
    lw = (ctypes.c_int32 * SCA_LMAX)(*[int(w) for _, w in levels], *([0] * (SCA_LMAX - L)))
    return ScaProblem(B, N, C, heads, L, P, Z, lh, lw, int(img_hw[0]), int(img_hw[1]), X, Y,
                      float(x_min), float(dx), float(y_min), float(dy), float(depth_eps),
                      REDUCE[reduce])


def sca_forward(value, lidar2img, z, offsets, logits, levels, heads, img_hw, X, Y, x_min, dx,
                y_min, dy, depth_eps=1e-5, reduce="mean", nthreads=0, libpath=None):
    """FlashSCA forward on the CPU.

    ``value`` [B, N, S, C], ``offsets`` [B, X*Y, heads, L, P, 2], ``logits``
    [B, X*Y, heads, L, P] (all float32).  Returns ``(out, scale, terms,
    counters)``: ``out`` and ``scale`` float64 [B, X*Y, C], ``terms`` int32
    [B, X*Y, heads] (in-range taps per query and head), ``counters`` a dict
    with the (query, camera) hits and in-range taps.
    """
    v = np.ascontiguousarray(value, dtype=np.float32)
    m = np.ascontiguousarray(lidar2img, dtype=np.float32)
    zz = np.ascontiguousarray(z, dtype=np.float32)
    off = np.ascontiguousarray(offsets, dtype=np.float32)
    lg = np.ascontiguousarray(logits, dtype=np.float32)
    B, N, S, C = v.shape
    L = len(levels)
    P = lg.shape[-1]
    assert S == sum(h * w for h, w in levels)
    assert m.shape == (B, N, 4, 4)
    assert lg.shape == (B, X * Y, heads, L, P) and off.shape == lg.shape + (2,)
    p = sca_problem(B, N, C, heads, levels, P, len(zz), img_hw, X, Y, x_min, dx, y_min, dy,
                    depth_eps, reduce)
    out = np.empty((B, X * Y, C), dtype=np.float64)
    scale = np.empty_like(out)
    terms = np.empty((B, X * Y, heads), dtype=np.int32)
    cnt = ScaCounters()
    rc = _sca_lib(libpath).sca_oracle_forward(
        ctypes.byref(p), _ptr(v), _ptr(m), _ptr(zz), _ptr(off), _ptr(lg), _ptr(out),
        _ptr(scale), _ptr(terms), ctypes.byref(cnt), int(nthreads))
    if rc:
        raise ValueError(f"sca_oracle_forward failed: {rc}")
    return out, scale, terms, {"hits": int(cnt.hits), "taps": int(cnt.taps)}


def sca_reference_points(lidar2img, z, B, N, img_hw, X, Y, x_min, dx, y_min, dy,
                         depth_eps=1e-5, libpath=None):
    """Anchor reference points: ``(un, vn, valid, hit)``; the first three are
    [B, X*Y, N, Z], ``hit`` is [B, X*Y, N]."""
    m = np.ascontiguousarray(lidar2img, dtype=np.float32)
    zz = np.ascontiguousarray(z, dtype=np.float32)
    Z = len(zz)
    p = sca_problem(B, N, 1, 1, [(1, 1)], Z, Z, img_hw, X, Y, x_min, dx, y_min, dy, depth_eps)
    shape = (B, X * Y, N, Z)
    un = np.empty(shape, dtype=np.float32)
    vn = np.empty(shape, dtype=np.float32)
    valid = np.empty(shape, dtype=np.uint8)
    hit = np.empty(shape[:3], dtype=np.uint8)
    rc = _sca_lib(libpath).sca_oracle_reference_points(ctypes.byref(p), _ptr(m), _ptr(zz),
                                                       _ptr(un), _ptr(vn), _ptr(valid), _ptr(hit))
    if rc:
        raise ValueError(f"sca_oracle_reference_points failed: {rc}")
    return un, vn, valid.astype(bool), hit.astype(bool)


def sca_instance(inst, reduce="mean", nthreads=0, libpath=None):
    """FlashSCA oracle on a ``synth.ScaInstance``."""
    wl = inst.wl
    return sca_forward(inst.value, inst.lidar2img, inst.z, inst.offsets, inst.logits, wl.levels,
                       wl.heads, (wl.img_h, wl.img_w), wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min,
                       wl.dy, wl.depth_eps, reduce, nthreads, libpath)


def sca_backward(value, lidar2img, z, offsets, logits, grad_out, levels, heads, img_hw, X, Y,
                 x_min, dx, y_min, dy, depth_eps=1e-5, reduce="mean", nthreads=0, libpath=None,
                 with_scales=True, buffers=None):
    """Gradients of the FlashSCA forward with respect to the value maps, the
    offsets and the logits, for output gradient ``grad_out`` [B, X*Y, C].

    Returns a dict of float64 arrays: ``value`` [B, N, S, C] with
    ``value_scale`` and int32 ``value_terms`` [B, N, S, heads]; ``offsets``
    [B, X*Y, heads, L, P, 2] with ``offsets_scale``; ``logits``
    [B, X*Y, heads, L, P] with ``logits_scale``; int32 ``point_terms``
    [B, X*Y, heads, L, P] (in-range corners per point over hit cameras).
    ``with_scales=False`` skips the scales and term counts (None in the
    result); ``buffers`` may hold preallocated float64 ``value``,
    ``offsets`` and ``logits`` arrays of those shapes, which are reused.
    """
    v = np.ascontiguousarray(value, dtype=np.float32)
    m = np.ascontiguousarray(lidar2img, dtype=np.float32)
    zz = np.ascontiguousarray(z, dtype=np.float32)
    off = np.ascontiguousarray(offsets, dtype=np.float32)
    lg = np.ascontiguousarray(logits, dtype=np.float32)
    g = np.ascontiguousarray(grad_out, dtype=np.float32)
    B, N, S, C = v.shape
    L = len(levels)
    P = lg.shape[-1]
    Q = X * Y
    assert g.shape == (B, Q, C) and lg.shape == (B, Q, heads, L, P) and off.shape == lg.shape + (2,)
    p = sca_problem(B, N, C, heads, levels, P, len(zz), img_hw, X, Y, x_min, dx, y_min, dy,
                    depth_eps, reduce)
    shapes = {"value": (B, N, S, C), "offsets": (B, Q, heads, L, P, 2),
              "logits": (B, Q, heads, L, P)}
    r = {}
    for k, shp in shapes.items():
        buf = (buffers or {}).get(k)
        if buf is not None:
            assert buf.shape == shp and buf.dtype == np.float64 and buf.flags.c_contiguous
            r[k] = buf
        else:
            r[k] = np.empty(shp)
    if with_scales:
        r.update({"value_scale": np.empty((B, N, S, C)),
                  "value_terms": np.empty((B, N, S, heads), dtype=np.int32),
                  "offsets_scale": np.empty((B, Q, heads, L, P, 2)),
                  "logits_scale": np.empty((B, Q, heads, L, P)),
                  "point_terms": np.empty((B, Q, heads, L, P), dtype=np.int32)})
    else:
        r.update({k: None for k in ("value_scale", "value_terms", "offsets_scale",
                                    "logits_scale", "point_terms")})
    ptr = lambda a: _ptr(a) if a is not None else None
    rc = _sca_lib(libpath).sca_oracle_backward(
        ctypes.byref(p), _ptr(v), _ptr(m), _ptr(zz), _ptr(off), _ptr(lg), _ptr(g),
        _ptr(r["value"]), ptr(r["value_scale"]), ptr(r["value_terms"]), _ptr(r["offsets"]),
        ptr(r["offsets_scale"]), _ptr(r["logits"]), ptr(r["logits_scale"]),
        ptr(r["point_terms"]), int(nthreads))
    if rc:
        raise ValueError(f"sca_oracle_backward failed: {rc}")
    return r


def sca_backward_instance(inst, grad_out, reduce="mean", nthreads=0, libpath=None,
                          with_scales=True, buffers=None):
    """FlashSCA backward oracle on a ``synth.ScaInstance``."""
    wl = inst.wl
    return sca_backward(inst.value, inst.lidar2img, inst.z, inst.offsets, inst.logits, grad_out,
                        wl.levels, wl.heads, (wl.img_h, wl.img_w), wl.X, wl.Y, wl.x_min, wl.dx,
                        wl.y_min, wl.dy, wl.depth_eps, reduce, nthreads, libpath, with_scales,
                        buffers)
