"""Fused Sampling-VT (FlashBEV) and FlashSCA for AMD MI355X.

A thin Python binding over the C ABI of ``include/flashbev.h`` and
``include/flashsca.h`` (``libflashbev.so``).  It only marshals arguments: every step of the
operator runs in the library's HIP kernel.  PyTorch supplies device memory
and the current stream.  If the built library is missing the calls raise;
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional, Sequence, Tuple

__all__ = [
    "BevGrid", "sample_vt", "sample_vt_backward", "prepare_sample_vt", "prepare_sample_vt_backward",
    "sca_forward", "sca_forward_raw", "sca_launch_info", "prepare_sca_forward",
    "sca_backward", "sca_backward_launch_info", "prepare_sca_backward",
    "launch_info", "backward_launch_info", "status_string", "abi_version", "library_path",
    "FlashBevError", "DTYPE_CODES", "REDUCE_CODES", "STATUS",
    "sample_vt_autograd", "sca_autograd",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libflashbev.so")
_LIB = None

DTYPE_CODES = {"f32": 0, "f16": 1, "bf16": 2}
REDUCE_CODES = {"mean": 0, "sum": 1}
STATUS = {
    "OK": 0, "ERR_NULLPTR": -1, "ERR_SHAPE": -2, "ERR_DTYPE": -3, "ERR_ALIGN": -4,
    "ERR_UNSUPPORTED": -5, "ERR_ALIAS": -6, "ERR_VALUE": -7, "ERR_HIP": -8,
    "ERR_SCRATCH": -9,
}
ABI_VERSION = 2
ZMAX = 256
NMAX = 64
ROW_BYTES_MAX = 4096
SCRATCH_BYTES = 64 << 20


class FlashBevError(RuntimeError):
    def __init__(self, status: int, what: str = "flashbev_sample_vt"):
        self.status = status
        super().__init__(f"{what} failed: {status} ({status_string(status)})")


class Features(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("B", ctypes.c_int32), ("N", ctypes.c_int32), ("H", ctypes.c_int32),
                ("W", ctypes.c_int32), ("C", ctypes.c_int32),
                ("img_h", ctypes.c_int32), ("img_w", ctypes.c_int32)]


class GridSpec(ctypes.Structure):
    _fields_ = [("x_min", ctypes.c_float), ("dx", ctypes.c_float), ("X", ctypes.c_int32),
                ("y_min", ctypes.c_float), ("dy", ctypes.c_float), ("Y", ctypes.c_int32),
                ("depth_eps", ctypes.c_float), ("reduce", ctypes.c_int32)]


SCA_LMAX = 8
SCA_NMAX = 32
SCA_ZMAX = 32
SCA_LPMAX = 512
SCA_HEAD_BYTES_MAX = 1024


class ScaValue(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("B", ctypes.c_int32), ("N", ctypes.c_int32), ("C", ctypes.c_int32),
                ("heads", ctypes.c_int32), ("L", ctypes.c_int32),
                ("level_h", ctypes.c_int32 * SCA_LMAX), ("level_w", ctypes.c_int32 * SCA_LMAX),
                ("img_h", ctypes.c_int32), ("img_w", ctypes.c_int32)]


class ZBins(ctypes.Structure):
    _fields_ = [("z", ctypes.POINTER(ctypes.c_float)), ("Z", ctypes.c_int32)]


@dataclasses.dataclass(frozen=True)
class BevGrid:
    """BEV grid: X cells from x_min with pitch dx, Y cells from y_min with pitch dy."""

    x_min: float
    dx: float
    X: int
    y_min: float
    dy: float
    Y: int
    depth_eps: float = 1e-5


def library_path() -> str:
    return _LIB_PATH


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_LIB_PATH):
            raise FileNotFoundError(
                f"{_LIB_PATH} is not built; run `python -m paper_2607_10071_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER
        L.flashbev_sample_vt.argtypes = [P(Features), ctypes.c_void_p, P(GridSpec), P(ZBins),
                                         ctypes.c_void_p, ctypes.c_void_p]
        L.flashbev_sample_vt.restype = ctypes.c_int
        L.flashbev_status_string.argtypes = [ctypes.c_int]
        L.flashbev_status_string.restype = ctypes.c_char_p
        L.flashbev_abi_version.argtypes = []
        L.flashbev_abi_version.restype = ctypes.c_int
        L.flashbev_launch_info.argtypes = [P(Features), P(GridSpec), P(ZBins),
                                           P(ctypes.c_int64), P(ctypes.c_int32),
                                           P(ctypes.c_int32), P(ctypes.c_int32),
                                           P(ctypes.c_int32)]
        L.flashbev_launch_info.restype = ctypes.c_int
        L.flashbev_sample_vt_backward.argtypes = [P(Features), ctypes.c_void_p, P(GridSpec),
                                                  P(ZBins), ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_void_p]
        L.flashbev_sample_vt_backward.restype = ctypes.c_int
        L.flashbev_backward_launch_info.argtypes = [P(Features), P(GridSpec), P(ZBins),
                                                    P(ctypes.c_int64), P(ctypes.c_int32),
                                                    P(ctypes.c_int32), P(ctypes.c_int32),
                                                    P(ctypes.c_int32)]
        L.flashbev_backward_launch_info.restype = ctypes.c_int
        L.flashbev_backward_workspace_size.argtypes = [P(Features), P(GridSpec), P(ZBins),
                                                       P(ctypes.c_uint64)]
        L.flashbev_backward_workspace_size.restype = ctypes.c_int
        L.flashbev_sample_vt_backward_ws.argtypes = [P(Features), ctypes.c_void_p, P(GridSpec),
                                                     P(ZBins), ctypes.c_void_p, ctypes.c_void_p,
                                                     ctypes.c_void_p, ctypes.c_uint64,
                                                     ctypes.c_void_p]
        L.flashbev_sample_vt_backward_ws.restype = ctypes.c_int
        L.flashbev_sample_vt_backward_noalloc.argtypes = [P(Features), ctypes.c_void_p,
                                                          P(GridSpec), P(ZBins), ctypes.c_void_p,
                                                          ctypes.c_void_p, ctypes.c_void_p]
        L.flashbev_sample_vt_backward_noalloc.restype = ctypes.c_int
        L.flashsca_forward.argtypes = [P(ScaValue), ctypes.c_void_p, P(GridSpec), P(ZBins),
                                       ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p]
        L.flashsca_forward.restype = ctypes.c_int
        L.flashsca_launch_info.argtypes = [P(ScaValue), P(GridSpec), P(ZBins), ctypes.c_int32,
                                           P(ctypes.c_int64), P(ctypes.c_int32),
                                           P(ctypes.c_int32), P(ctypes.c_int32),
                                           P(ctypes.c_int32)]
        L.flashsca_launch_info.restype = ctypes.c_int
        L.flashsca_backward.argtypes = [P(ScaValue), ctypes.c_void_p, P(GridSpec), P(ZBins),
                                        ctypes.c_int32] + [ctypes.c_void_p] * 7
        L.flashsca_backward.restype = ctypes.c_int
        L.flashsca_backward_launch_info.argtypes = L.flashsca_launch_info.argtypes
        L.flashsca_backward_launch_info.restype = ctypes.c_int
        _LIB = L
    return _LIB


def status_string(status: int) -> str:
    return _lib().flashbev_status_string(int(status)).decode()


def abi_version() -> int:
    return int(_lib().flashbev_abi_version())


def _dtype_code(t) -> int:
    import torch

    m = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}
    if t.dtype not in m:
        raise TypeError(f"unsupported feature dtype {t.dtype}")
    return DTYPE_CODES[m[t.dtype]]


def _z_array(z_bins):
    import numpy as np

    if hasattr(z_bins, "detach"):
        z_bins = z_bins.detach().cpu().numpy()
    z = np.ascontiguousarray(np.asarray(z_bins, dtype=np.float32).reshape(-1))
    return z


def _structs(features_shape, dtype_code, data_ptr, img_hw, grid: BevGrid, z, reduce):
    B, N, H, W, C = features_shape
    f = Features(data_ptr, dtype_code, B, N, H, W, C, int(img_hw[0]), int(img_hw[1]))
    g = GridSpec(grid.x_min, grid.dx, grid.X, grid.y_min, grid.dy, grid.Y, grid.depth_eps,
                 REDUCE_CODES[reduce])
    zb = ZBins(z.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), len(z))
    return f, g, zb


def sample_vt(features, lidar2img, z_bins, grid: BevGrid, img_hw: Tuple[int, int],
              out=None, reduce: str = "mean", stream=None):
    """Fused Sampling-VT forward (Eq. 1) on the GPU.

    features   CUDA tensor [B, N, H, W, C] (float32, float16 or bfloat16),
               contiguous channel-last feature maps.
    lidar2img  CUDA float32 tensor [B, N, 4, 4].
    z_bins     heights in metres (host sequence, numpy array or tensor).
    grid       BevGrid.
    img_hw     (img_h, img_w) of the image lidar2img projects into.
    out        optional CUDA float32 tensor [B, C, X, Y] to write into.
    reduce     "mean" (Eq. 1, per-height valid mean) or "sum".
    stream     torch.cuda.Stream or raw hipStream_t int; defaults to the
               current stream.

    Returns ``out`` ([B, C, X, Y] float32).  The call is asynchronous.
    """
    import torch

    _check_forward(features, lidar2img, grid)
    B, N, H, W, C = features.shape
    if out is None:
        out = torch.empty((B, C, grid.X, grid.Y), dtype=torch.float32, device=features.device)
    _check_out(out, (B, C, grid.X, grid.Y), "out")
    z = _z_array(z_bins)
    f, g, zb = _structs(features.shape, _dtype_code(features), features.data_ptr(), img_hw,
                        grid, z, reduce)
    dev = _one_device(features, lidar2img, out)
    s = _stream_handle(stream, dev)
    with _on_device(dev):
        rc = _lib().flashbev_sample_vt(ctypes.byref(f), ctypes.c_void_p(lidar2img.data_ptr()),
                                       ctypes.byref(g), ctypes.byref(zb),
                                       ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(s))
    if rc != 0:
        raise FlashBevError(rc)
    return out


def _check_forward(features, lidar2img, grid: BevGrid) -> None:
    """The forward's tensor checks (sample_vt and prepare_sample_vt): the C
    call reads these tensors as raw device memory of the stated shape."""
    if features.dim() != 5:
        raise ValueError("features must be [B, N, H, W, C]")
    if not features.is_cuda or not lidar2img.is_cuda:
        raise ValueError("features and lidar2img must be device tensors")
    if not features.is_contiguous():
        raise ValueError("features must be contiguous (channel-last NHWC)")
    _dtype_code(features)
    _check_matrices(lidar2img, features.shape[0], features.shape[1])


def _check_matrices(lidar2img, B: int, N: int) -> None:
    import torch

    if lidar2img.dtype != torch.float32 or not lidar2img.is_contiguous():
        raise ValueError("lidar2img must be a contiguous float32 tensor")
    if tuple(lidar2img.shape) != (B, N, 4, 4):
        raise ValueError(f"lidar2img must be [{B}, {N}, 4, 4]")


def _check_out(t, shape, name: str) -> None:
    """A float32 contiguous device tensor of exactly ``shape``."""
    import torch

    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != torch.float32 or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be a contiguous float32 tensor "
                         f"[{', '.join(str(int(v)) for v in shape)}]")


def _check_backward(grad_out, lidar2img, grid: BevGrid, features_shape):
    """The backward's tensor checks (sample_vt_backward and
    prepare_sample_vt_backward); returns (B, N, H, W, C)."""
    if len(tuple(features_shape)) != 5:
        raise ValueError("features_shape must be (B, N, H, W, C)")
    B, N, H, W, C = (int(v) for v in features_shape)
    if not grad_out.is_cuda or not lidar2img.is_cuda:
        raise ValueError("grad_out and lidar2img must be device tensors")
    _check_out(grad_out, (B, C, grid.X, grid.Y), "grad_out")
    _check_matrices(lidar2img, B, N)
    return B, N, H, W, C


def _stream_handle(stream, device):
    import torch

    if stream is None:
        return torch.cuda.current_stream(device).cuda_stream
    if isinstance(stream, int):
        return stream
    if stream.device != device:
        raise ValueError(f"stream is on {stream.device}, the tensors on {device}")
    return stream.cuda_stream


def _one_device(*tensors):
    """The CUDA device the given tensors (None entries skipped) share."""
    devs = {t.device for t in tensors if t is not None}
    if len(devs) != 1:
        raise ValueError("all tensors of a call must be on one CUDA device, got "
                         + ", ".join(sorted(str(d) for d in devs)))
    return devs.pop()


def _on_device(device):
    """Makes ``device`` current around a C call: the entry points launch on the
    calling thread's current device."""
    import contextlib
    import torch

    if torch.cuda.current_device() == device.index:
        return contextlib.nullcontext()
    return torch.cuda.device(device)


BACKWARD_METHODS = ("gather", "scatter")


def backward_workspace_size(features_shape, features_dtype, z_bins, grid: BevGrid, img_hw,
                            reduce: str = "mean") -> int:
    """Workspace bytes of the gather-form backward for these arguments, or
    -1 when it does not serve them (the scatter form then does)."""
    z = _z_array(z_bins)
    f, g, zb = _structs(tuple(int(v) for v in features_shape), DTYPE_CODES[features_dtype], 0,
                        img_hw, grid, z, reduce)
    out = ctypes.c_uint64()
    rc = _lib().flashbev_backward_workspace_size(ctypes.byref(f), ctypes.byref(g),
                                                 ctypes.byref(zb), ctypes.byref(out))
    if rc == STATUS["ERR_UNSUPPORTED"]:
        # the scatter form's own checks decide whether any backward serves it
        backward_launch_info(features_shape, features_dtype, z, grid, img_hw, reduce)
        return -1
    if rc != 0:
        raise FlashBevError(rc, "flashbev_backward_workspace_size")
    return int(out.value)


def _dtype_name(features_dtype) -> str:
    import torch

    if isinstance(features_dtype, str):
        return features_dtype
    return {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[features_dtype]


def sample_vt_backward(grad_out, lidar2img, z_bins, grid: BevGrid, img_hw: Tuple[int, int],
                       features_shape, features_dtype="f32", grad_features=None,
                       reduce: str = "mean", stream=None, method: str = "gather",
                       workspace=None):
    """Gradient of the fused Sampling-VT forward with respect to the features.

    grad_out        CUDA float32 tensor [B, C, X, Y] (gradient w.r.t. ``out``).
    lidar2img       CUDA float32 tensor [B, N, 4, 4].
    features_shape  (B, N, H, W, C) of the features of the forward call.
    features_dtype  their dtype ("f32", "f16", "bf16" or a torch dtype).
    grad_features   optional CUDA float32 tensor [B, N, H, W, C] to write.
    method          "gather" (flashbev_sample_vt_backward_ws: every gradient
                    row written once, no atomics, bitwise reproducible; it
                    needs a device workspace, allocated here unless
                    ``workspace`` is given) or "scatter"
                    (flashbev_sample_vt_backward: float atomics, no
                    workspace).  "gather" falls back to "scatter" for
                    shapes it does not serve.

    Returns ``grad_features`` (float32, channel-last).  Asynchronous.
    """
    import torch

    if method not in BACKWARD_METHODS:
        raise ValueError(f"method must be one of {BACKWARD_METHODS}")
    B, N, H, W, C = _check_backward(grad_out, lidar2img, grid, features_shape)
    if grad_features is None:
        grad_features = torch.empty((B, N, H, W, C), dtype=torch.float32, device=grad_out.device)
    _check_out(grad_features, (B, N, H, W, C), "grad_features")
    features_dtype = _dtype_name(features_dtype)
    z = _z_array(z_bins)
    f, g, zb = _structs((B, N, H, W, C), DTYPE_CODES[features_dtype], 0, img_hw, grid, z, reduce)
    dev = _one_device(grad_out, lidar2img, grad_features)
    s = _stream_handle(stream, dev)
    if method == "gather":
        need = backward_workspace_size((B, N, H, W, C), features_dtype, z, grid, img_hw, reduce)
        if need < 0:
            method = "scatter"
        else:
            if workspace is None:
                workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=grad_out.device)
            elif not workspace.is_cuda or workspace.numel() * workspace.element_size() < need:
                raise ValueError(f"workspace must be a device tensor of at least {need} bytes")
            with _on_device(dev):
                rc = _lib().flashbev_sample_vt_backward_ws(
                    ctypes.byref(f), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
                    ctypes.byref(zb), ctypes.c_void_p(grad_out.data_ptr()),
                    ctypes.c_void_p(grad_features.data_ptr()),
                    ctypes.c_void_p(workspace.data_ptr()),
                    ctypes.c_uint64(workspace.numel() * workspace.element_size()),
                    ctypes.c_void_p(s))
            if rc != 0:
                raise FlashBevError(rc, "flashbev_sample_vt_backward_ws")
            return grad_features
    with _on_device(dev):
        rc = _lib().flashbev_sample_vt_backward(
            ctypes.byref(f), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
            ctypes.byref(zb), ctypes.c_void_p(grad_out.data_ptr()),
            ctypes.c_void_p(grad_features.data_ptr()), ctypes.c_void_p(s))
    if rc != 0:
        raise FlashBevError(rc, "flashbev_sample_vt_backward")
    return grad_features


def sample_vt_backward_raw(shape, dtype: str, lidar2img_ptr: int, z_bins, grid: BevGrid,
                           img_hw, grad_out_ptr: int, grad_features_ptr: int,
                           reduce: str = "mean", stream: int = 0) -> int:
    """The backward C entry point with raw device addresses; returns the status."""
    z = _z_array(z_bins)
    f, g, zb = _structs(shape, DTYPE_CODES[dtype], 0, img_hw, grid, z, reduce)
    return int(_lib().flashbev_sample_vt_backward(
        ctypes.byref(f), ctypes.c_void_p(lidar2img_ptr), ctypes.byref(g), ctypes.byref(zb),
        ctypes.c_void_p(grad_out_ptr), ctypes.c_void_p(grad_features_ptr),
        ctypes.c_void_p(stream)))


def sample_vt_backward_ws_raw(shape, dtype: str, lidar2img_ptr: int, z_bins, grid: BevGrid,
                              img_hw, grad_out_ptr: int, grad_features_ptr: int,
                              workspace_ptr: int, workspace_bytes: int, reduce: str = "mean",
                              stream: int = 0) -> int:
    """The gather-form backward's C entry point with raw device addresses;
    returns the status."""
    z = _z_array(z_bins)
    f, g, zb = _structs(shape, DTYPE_CODES[dtype], 0, img_hw, grid, z, reduce)
    return int(_lib().flashbev_sample_vt_backward_ws(
        ctypes.byref(f), ctypes.c_void_p(lidar2img_ptr), ctypes.byref(g), ctypes.byref(zb),
        ctypes.c_void_p(grad_out_ptr), ctypes.c_void_p(grad_features_ptr),
        ctypes.c_void_p(workspace_ptr), ctypes.c_uint64(workspace_bytes),
        ctypes.c_void_p(stream)))


def sample_vt_backward_noalloc(grad_out, lidar2img, z_bins, grid: BevGrid, img_hw,
                               features_shape, features_dtype, grad_features,
                               reduce: str = "mean", stream=None):
    """The gather-form backward on the library's static device scratch
    (flashbev_sample_vt_backward_noalloc): nothing is allocated, here or in
    the library, so ``grad_features`` is required.  Calls that can overlap on
    one GPU share its scratch and must be ordered by the caller.  Raises
    FlashBevError with status ERR_SCRATCH when the call needs more than
    SCRATCH_BYTES of workspace."""
    B, N, H, W, C = _check_backward(grad_out, lidar2img, grid, features_shape)
    _check_out(grad_features, (B, N, H, W, C), "grad_features")
    features_dtype = _dtype_name(features_dtype)
    z = _z_array(z_bins)
    f, g, zb = _structs((B, N, H, W, C), DTYPE_CODES[features_dtype], 0, img_hw, grid, z, reduce)
    dev = _one_device(grad_out, lidar2img, grad_features)
    s = _stream_handle(stream, dev)
    with _on_device(dev):
        rc = _lib().flashbev_sample_vt_backward_noalloc(
            ctypes.byref(f), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
            ctypes.byref(zb), ctypes.c_void_p(grad_out.data_ptr()),
            ctypes.c_void_p(grad_features.data_ptr()), ctypes.c_void_p(s))
    if rc != 0:
        raise FlashBevError(rc, "flashbev_sample_vt_backward_noalloc")
    return grad_features


def sample_vt_backward_noalloc_raw(shape, dtype: str, lidar2img_ptr: int, z_bins,
                                   grid: BevGrid, img_hw, grad_out_ptr: int,
                                   grad_features_ptr: int, reduce: str = "mean",
                                   stream: int = 0) -> int:
    """flashbev_sample_vt_backward_noalloc with raw device addresses; returns
    the status."""
    z = _z_array(z_bins)
    f, g, zb = _structs(shape, DTYPE_CODES[dtype], 0, img_hw, grid, z, reduce)
    return int(_lib().flashbev_sample_vt_backward_noalloc(
        ctypes.byref(f), ctypes.c_void_p(lidar2img_ptr), ctypes.byref(g), ctypes.byref(zb),
        ctypes.c_void_p(grad_out_ptr), ctypes.c_void_p(grad_features_ptr),
        ctypes.c_void_p(stream)))


def sample_vt_raw(features_ptr: int, dtype: str, shape, lidar2img_ptr: int, z_bins,
                  grid: BevGrid, img_hw, out_ptr: int, reduce: str = "mean",
                  stream: int = 0) -> int:
    """The C entry point with raw device addresses; returns the status code."""
    z = _z_array(z_bins)
    f, g, zb = _structs(shape, DTYPE_CODES[dtype], features_ptr, img_hw, grid, z, reduce)
    return int(_lib().flashbev_sample_vt(ctypes.byref(f), ctypes.c_void_p(lidar2img_ptr),
                                         ctypes.byref(g), ctypes.byref(zb),
                                         ctypes.c_void_p(out_ptr), ctypes.c_void_p(stream)))


def launch_info(shape, dtype: str, z_bins, grid: BevGrid, img_hw, reduce: str = "mean",
                data_ptr: int = 0) -> dict:
    """Launch geometry for these arguments (no HIP call)."""
    z = _z_array(z_bins)
    f, g, zb = _structs(shape, DTYPE_CODES[dtype], data_ptr, img_hw, grid, z, reduce)
    wg = ctypes.c_int64()
    thr = ctypes.c_int32()
    lds = ctypes.c_int32()
    cpw = ctypes.c_int32()
    lpc = ctypes.c_int32()
    rc = _lib().flashbev_launch_info(ctypes.byref(f), ctypes.byref(g), ctypes.byref(zb),
                                     ctypes.byref(wg), ctypes.byref(thr), ctypes.byref(lds),
                                     ctypes.byref(cpw), ctypes.byref(lpc))
    if rc != 0:
        raise FlashBevError(rc, "flashbev_launch_info")
    return {"workgroups": wg.value, "threads": thr.value, "lds_bytes": lds.value,
            "cells_per_wave": cpw.value, "lanes_per_cell": lpc.value}


def grid_of(wl) -> BevGrid:
    """BevGrid of a workload description with x_min/dx/X/y_min/dy/Y fields."""
    return BevGrid(wl.x_min, wl.dx, wl.X, wl.y_min, wl.dy, wl.Y, wl.depth_eps)


def backward_launch_info(shape, dtype: str, z_bins, grid: BevGrid, img_hw,
                         reduce: str = "mean") -> dict:
    """Launch geometry of the backward for these arguments (no HIP call)."""
    z = _z_array(z_bins)
    f, g, zb = _structs(shape, DTYPE_CODES[dtype], 0, img_hw, grid, z, reduce)
    wg = ctypes.c_int64()
    thr = ctypes.c_int32()
    lds = ctypes.c_int32()
    rows = ctypes.c_int32()
    lpc = ctypes.c_int32()
    rc = _lib().flashbev_backward_launch_info(ctypes.byref(f), ctypes.byref(g), ctypes.byref(zb),
                                              ctypes.byref(wg), ctypes.byref(thr),
                                              ctypes.byref(lds), ctypes.byref(rows),
                                              ctypes.byref(lpc))
    if rc != 0:
        raise FlashBevError(rc, "flashbev_backward_launch_info")
    return {"workgroups": wg.value, "threads": thr.value, "lds_bytes": lds.value,
            "rows_per_tile": rows.value, "lanes_per_cell": lpc.value}


class _Prepared:
    """A C entry point with its arguments marshalled once: calling it makes
    the call again with no Python-side allocation.  It keeps the tensors and
    structures it refers to alive."""

    def __init__(self, fn, args, keep, what, device):
        import torch

        self._fn = fn
        self._args = args
        self._keep = keep
        self._what = what
        self._dev = device.index
        self._cuda = torch.cuda

    def __call__(self) -> None:
        if self._cuda.current_device() == self._dev:
            rc = self._fn(*self._args)
        else:
            with self._cuda.device(self._dev):
                rc = self._fn(*self._args)
        if rc != 0:
            raise FlashBevError(rc, self._what)


def prepare_sample_vt(features, lidar2img, z_bins, grid: BevGrid, img_hw, out,
                      reduce: str = "mean", stream=None) -> _Prepared:
    """``sample_vt`` with every argument fixed: returns a callable that
    enqueues the same forward call again (same tensors, same stream)."""
    _check_forward(features, lidar2img, grid)
    B, N, H, W, C = features.shape
    _check_out(out, (B, C, grid.X, grid.Y), "out")
    z = _z_array(z_bins)
    f, g, zb = _structs(features.shape, _dtype_code(features), features.data_ptr(), img_hw,
                        grid, z, reduce)
    dev = _one_device(features, lidar2img, out)
    s = _stream_handle(stream, dev)
    args = (ctypes.byref(f), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
            ctypes.byref(zb), ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(s))
    return _Prepared(_lib().flashbev_sample_vt, args,
                     (features, lidar2img, out, z, f, g, zb), "flashbev_sample_vt", dev)


def prepare_sample_vt_backward(grad_out, lidar2img, z_bins, grid: BevGrid, img_hw,
                               features_shape, features_dtype, grad_features,
                               reduce: str = "mean", stream=None,
                               method: str = "gather") -> _Prepared:
    """``sample_vt_backward`` with every argument fixed (see prepare_sample_vt);
    the gather form's workspace is allocated once, here."""
    import torch

    if method not in BACKWARD_METHODS:
        raise ValueError(f"method must be one of {BACKWARD_METHODS}")
    B, N, H, W, C = _check_backward(grad_out, lidar2img, grid, features_shape)
    _check_out(grad_features, (B, N, H, W, C), "grad_features")
    features_dtype = _dtype_name(features_dtype)
    z = _z_array(z_bins)
    f, g, zb = _structs((B, N, H, W, C), DTYPE_CODES[features_dtype], 0, img_hw, grid, z, reduce)
    dev = _one_device(grad_out, lidar2img, grad_features)
    s = _stream_handle(stream, dev)
    if method == "gather":
        need = backward_workspace_size((B, N, H, W, C), features_dtype, z, grid, img_hw, reduce)
        if need >= 0:
            ws = torch.empty(max(need, 1), dtype=torch.uint8, device=grad_out.device)
            args = (ctypes.byref(f), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
                    ctypes.byref(zb), ctypes.c_void_p(grad_out.data_ptr()),
                    ctypes.c_void_p(grad_features.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                    ctypes.c_uint64(ws.numel()), ctypes.c_void_p(s))
            return _Prepared(_lib().flashbev_sample_vt_backward_ws, args,
                             (grad_out, lidar2img, grad_features, ws, z, f, g, zb),
                             "flashbev_sample_vt_backward_ws", dev)
    args = (ctypes.byref(f), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
            ctypes.byref(zb), ctypes.c_void_p(grad_out.data_ptr()),
            ctypes.c_void_p(grad_features.data_ptr()), ctypes.c_void_p(s))
    return _Prepared(_lib().flashbev_sample_vt_backward, args,
                     (grad_out, lidar2img, grad_features, z, f, g, zb),
                     "flashbev_sample_vt_backward", dev)


# ---------------------------------------------------------------------------
# FlashSCA (include/flashsca.h)
# ---------------------------------------------------------------------------


def _sca_structs(shape, dtype_code, data_ptr, heads, levels, img_hw, grid: BevGrid, z, reduce):
    B, N, S, C = (int(v) for v in shape)
    L = len(levels)
    if not 1 <= L <= SCA_LMAX:
        raise ValueError(f"between 1 and {SCA_LMAX} levels are supported")
    lh = (ctypes.c_int32 * SCA_LMAX)(*[int(h) for h, _ in levels], *([0] * (SCA_LMAX - L)))
    lw = (ctypes.c_int32 * SCA_LMAX)(*[int(w) for _, w in levels], *([0] * (SCA_LMAX - L)))
    v = ScaValue(data_ptr, dtype_code, B, N, C, int(heads), L, lh, lw, int(img_hw[0]),
                 int(img_hw[1]))
    g = GridSpec(grid.x_min, grid.dx, grid.X, grid.y_min, grid.dy, grid.Y, grid.depth_eps,
                 REDUCE_CODES[reduce])
    zb = ZBins(z.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), len(z))
    return v, g, zb


def _sca_check(value, lidar2img, offsets, logits, levels, heads, grid):
    import torch

    if value.dim() != 4:
        raise ValueError("value must be [B, N, S, C]")
    for name, t in (("value", value), ("lidar2img", lidar2img), ("offsets", offsets),
                    ("logits", logits)):
        if not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    for name, t in (("lidar2img", lidar2img), ("offsets", offsets), ("logits", logits)):
        if t.dtype != torch.float32:
            raise ValueError(f"{name} must be float32")
    B, N, S, C = value.shape
    if S != sum(int(h) * int(w) for h, w in levels):
        raise ValueError("value's S must equal the sum of the levels' H * W")
    if tuple(lidar2img.shape) != (B, N, 4, 4):
        raise ValueError(f"lidar2img must be [{B}, {N}, 4, 4]")
    Q = grid.X * grid.Y
    if logits.dim() != 5 or tuple(logits.shape[:4]) != (B, Q, heads, len(levels)):
        raise ValueError(f"logits must be [{B}, {Q}, {heads}, {len(levels)}, P]")
    P = int(logits.shape[4])
    if tuple(offsets.shape) != (B, Q, heads, len(levels), P, 2):
        raise ValueError(f"offsets must be [{B}, {Q}, {heads}, {len(levels)}, {P}, 2]")
    return B, N, S, C, Q, P


def sca_forward(value, lidar2img, anchors, grid: BevGrid, img_hw: Tuple[int, int], levels,
                heads: int, offsets, logits, out=None, reduce: str = "mean", stream=None):
    """FlashSCA forward (BEVFormer spatial cross-attention, Sec. 4.5) on the GPU.

    value      CUDA tensor [B, N, S, C] (float32, float16 or bfloat16): the
               value maps of all levels, concatenated, channel-last.
    lidar2img  CUDA float32 tensor [B, N, 4, 4].
    anchors    pillar heights in metres (host sequence, numpy array or tensor).
    grid       BevGrid of the queries (query q = i * Y + j).
    img_hw     (img_h, img_w) of the image lidar2img projects into.
    levels     sequence of (H_l, W_l).
    heads      number of attention heads (C % heads == 0).
    offsets    CUDA float32 tensor [B, X*Y, heads, L, P, 2], level pixels.
    logits     CUDA float32 tensor [B, X*Y, heads, L, P].
    out        optional CUDA float32 tensor [B, X*Y, C].
    reduce     "mean" over hit cameras (BEVFormer) or "sum".

    Returns ``out``.  Asynchronous on ``stream`` (default: the current one).
    """
    import torch

    B, N, S, C, Q, P = _sca_check(value, lidar2img, offsets, logits, levels, heads, grid)
    if out is None:
        out = torch.empty((B, Q, C), dtype=torch.float32, device=value.device)
    elif out.dtype != torch.float32 or not out.is_contiguous() or tuple(out.shape) != (B, Q, C):
        raise ValueError(f"out must be a contiguous float32 tensor [{B}, {Q}, {C}]")
    z = _z_array(anchors)
    v, g, zb = _sca_structs(value.shape, _dtype_code(value), value.data_ptr(), heads, levels,
                            img_hw, grid, z, reduce)
    dev = _one_device(value, lidar2img, offsets, logits, out)
    s = _stream_handle(stream, dev)
    with _on_device(dev):
        rc = _lib().flashsca_forward(ctypes.byref(v), ctypes.c_void_p(lidar2img.data_ptr()),
                                     ctypes.byref(g), ctypes.byref(zb), P,
                                     ctypes.c_void_p(offsets.data_ptr()),
                                     ctypes.c_void_p(logits.data_ptr()),
                                     ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(s))
    if rc != 0:
        raise FlashBevError(rc, "flashsca_forward")
    return out


def sca_forward_raw(value_ptr: int, dtype: str, shape, heads: int, levels, lidar2img_ptr: int,
                    anchors, grid: BevGrid, img_hw, P: int, offsets_ptr: int, logits_ptr: int,
                    out_ptr: int, reduce: str = "mean", stream: int = 0) -> int:
    """The FlashSCA C entry point with raw device addresses; returns the status."""
    z = _z_array(anchors)
    v, g, zb = _sca_structs(shape, DTYPE_CODES[dtype], value_ptr, heads, levels, img_hw, grid,
                            z, reduce)
    return int(_lib().flashsca_forward(ctypes.byref(v), ctypes.c_void_p(lidar2img_ptr),
                                       ctypes.byref(g), ctypes.byref(zb), int(P),
                                       ctypes.c_void_p(offsets_ptr), ctypes.c_void_p(logits_ptr),
                                       ctypes.c_void_p(out_ptr), ctypes.c_void_p(stream)))


def sca_launch_info(shape, dtype: str, heads: int, levels, anchors, grid: BevGrid, img_hw,
                    P: int, reduce: str = "mean", data_ptr: int = 0,
                    backward: bool = False) -> dict:
    """Launch geometry of the FlashSCA forward (or backward) for these
    arguments (no HIP call)."""
    z = _z_array(anchors)
    v, g, zb = _sca_structs(shape, DTYPE_CODES[dtype], data_ptr, heads, levels, img_hw, grid, z,
                            reduce)
    wg = ctypes.c_int64()
    thr = ctypes.c_int32()
    lds = ctypes.c_int32()
    lph = ctypes.c_int32()
    lw = ctypes.c_int32()
    fn = _lib().flashsca_backward_launch_info if backward else _lib().flashsca_launch_info
    rc = fn(ctypes.byref(v), ctypes.byref(g), ctypes.byref(zb), int(P), ctypes.byref(wg),
            ctypes.byref(thr), ctypes.byref(lds), ctypes.byref(lph), ctypes.byref(lw))
    if rc != 0:
        raise FlashBevError(rc, "flashsca_backward_launch_info" if backward
                            else "flashsca_launch_info")
    return {"workgroups": wg.value, "threads": thr.value, "lds_bytes": lds.value,
            "lanes_per_head": lph.value, "lane_bytes": lw.value}


def prepare_sca_forward(value, lidar2img, anchors, grid: BevGrid, img_hw, levels, heads: int,
                        offsets, logits, out, reduce: str = "mean", stream=None) -> _Prepared:
    """``sca_forward`` with every argument fixed: a callable that enqueues the
    same call again (same tensors, same stream)."""
    import torch

    B, N, S, C, Q, P = _sca_check(value, lidar2img, offsets, logits, levels, heads, grid)
    if out.dtype != torch.float32 or not out.is_contiguous() or tuple(out.shape) != (B, Q, C) \
            or not out.is_cuda:
        raise ValueError(f"out must be a contiguous float32 device tensor [{B}, {Q}, {C}]")
    z = _z_array(anchors)
    v, g, zb = _sca_structs(value.shape, _dtype_code(value), value.data_ptr(), heads, levels,
                            img_hw, grid, z, reduce)
    dev = _one_device(value, lidar2img, offsets, logits, out)
    s = _stream_handle(stream, dev)
    args = (ctypes.byref(v), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
            ctypes.byref(zb), ctypes.c_int32(P), ctypes.c_void_p(offsets.data_ptr()),
            ctypes.c_void_p(logits.data_ptr()), ctypes.c_void_p(out.data_ptr()),
            ctypes.c_void_p(s))
    return _Prepared(_lib().flashsca_forward, args,
                     (value, lidar2img, offsets, logits, out, z, v, g, zb), "flashsca_forward",
                     dev)


def _sca_bwd_outputs(value, Q, heads, L, P, grad_value, grad_offsets, grad_logits, want):
    import torch

    B, N, S, C = value.shape
    dev = value.device
    shapes = {"value": (B, N, S, C), "offsets": (B, Q, heads, L, P, 2),
              "logits": (B, Q, heads, L, P)}
    given = {"value": grad_value, "offsets": grad_offsets, "logits": grad_logits}
    out = {}
    for k in ("value", "offsets", "logits"):
        t = given[k]
        if t is None and k in want:
            t = torch.empty(shapes[k], dtype=torch.float32, device=dev)
        if t is not None and (t.dtype != torch.float32 or not t.is_contiguous() or not t.is_cuda
                              or tuple(t.shape) != shapes[k]):
            raise ValueError(f"grad_{k} must be a contiguous float32 device tensor {shapes[k]}")
        out[k] = t
    return out


def sca_backward(value, lidar2img, anchors, grid: BevGrid, img_hw, levels, heads: int, offsets,
                 logits, grad_out, grad_value=None, grad_offsets=None, grad_logits=None,
                 want=("value", "offsets", "logits"), reduce: str = "mean", stream=None):
    """FlashSCA backward on the GPU: gradients with respect to the value maps,
    the offsets and the logits for ``grad_out`` [B, X*Y, C] float32.

    Returns a dict with the float32 tensors ``value`` [B, N, S, C],
    ``offsets`` [B, X*Y, heads, L, P, 2] and ``logits`` [B, X*Y, heads, L, P]
    (None for gradients not in ``want`` and not passed in).  Asynchronous.
    """
    import torch

    B, N, S, C, Q, P = _sca_check(value, lidar2img, offsets, logits, levels, heads, grid)
    if not grad_out.is_cuda or grad_out.dtype != torch.float32 or not grad_out.is_contiguous() \
            or tuple(grad_out.shape) != (B, Q, C):
        raise ValueError(f"grad_out must be a contiguous float32 device tensor [{B}, {Q}, {C}]")
    outs = _sca_bwd_outputs(value, Q, heads, len(levels), P, grad_value, grad_offsets,
                            grad_logits, want)
    z = _z_array(anchors)
    v, g, zb = _sca_structs(value.shape, _dtype_code(value), value.data_ptr(), heads, levels,
                            img_hw, grid, z, reduce)
    dev = _one_device(value, lidar2img, offsets, logits, grad_out, *outs.values())
    s = _stream_handle(stream, dev)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    with _on_device(dev):
        rc = _lib().flashsca_backward(ctypes.byref(v), ctypes.c_void_p(lidar2img.data_ptr()),
                                      ctypes.byref(g), ctypes.byref(zb), P,
                                      ctypes.c_void_p(offsets.data_ptr()),
                                      ctypes.c_void_p(logits.data_ptr()),
                                      ctypes.c_void_p(grad_out.data_ptr()), ptr(outs["value"]),
                                      ptr(outs["offsets"]), ptr(outs["logits"]),
                                      ctypes.c_void_p(s))
    if rc != 0:
        raise FlashBevError(rc, "flashsca_backward")
    return outs


def prepare_sca_backward(value, lidar2img, anchors, grid: BevGrid, img_hw, levels, heads: int,
                         offsets, logits, grad_out, grad_value, grad_offsets, grad_logits,
                         reduce: str = "mean", stream=None) -> _Prepared:
    """``sca_backward`` with every argument fixed (outputs given; any may be
    None): a callable that enqueues the same call again."""
    B, N, S, C, Q, P = _sca_check(value, lidar2img, offsets, logits, levels, heads, grid)
    outs = _sca_bwd_outputs(value, Q, heads, len(levels), P, grad_value, grad_offsets,
                            grad_logits, ())
    z = _z_array(anchors)
    v, g, zb = _sca_structs(value.shape, _dtype_code(value), value.data_ptr(), heads, levels,
                            img_hw, grid, z, reduce)
    dev = _one_device(value, lidar2img, offsets, logits, grad_out, *outs.values())
    s = _stream_handle(stream, dev)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    args = (ctypes.byref(v), ctypes.c_void_p(lidar2img.data_ptr()), ctypes.byref(g),
            ctypes.byref(zb), ctypes.c_int32(P), ctypes.c_void_p(offsets.data_ptr()),
            ctypes.c_void_p(logits.data_ptr()), ctypes.c_void_p(grad_out.data_ptr()),
            ptr(outs["value"]), ptr(outs["offsets"]), ptr(outs["logits"]), ctypes.c_void_p(s))
    return _Prepared(_lib().flashsca_backward, args,
                     (value, lidar2img, offsets, logits, grad_out, outs, z, v, g, zb),
                     "flashsca_backward", dev)


# ---------------------------------------------------------------------------
# autograd: the two operators as differentiable torch functions
# ---------------------------------------------------------------------------
_AUTOGRAD = {}


def _autograd_functions():
    """The torch.autograd.Function classes, made on first use (torch is
    imported lazily).  Their forward and backward are the calls above."""
    if _AUTOGRAD:
        return _AUTOGRAD
    import torch

    class _SampleVT(torch.autograd.Function):
        @staticmethod
        def forward(ctx, features, lidar2img, z_bins, grid, img_hw, reduce, method):
            ctx.save_for_backward(lidar2img)
            ctx.meta = (tuple(features.shape), features.dtype, z_bins, grid, tuple(img_hw),
                        reduce, method)
            return sample_vt(features, lidar2img, z_bins, grid, img_hw, reduce=reduce)

        @staticmethod
        def backward(ctx, grad_out):
            (l2i,) = ctx.saved_tensors
            shape, dtype, z_bins, grid, img_hw, reduce, method = ctx.meta
            g = None
            if ctx.needs_input_grad[0]:
                g = sample_vt_backward(grad_out.float().contiguous(), l2i, z_bins, grid, img_hw,
                                       shape, _dtype_name(dtype), reduce=reduce, method=method)
                if g.dtype != dtype:
                    g = g.to(dtype)
            return g, None, None, None, None, None, None

    class _SCA(torch.autograd.Function):
        @staticmethod
        def forward(ctx, value, lidar2img, offsets, logits, anchors, grid, img_hw, levels, heads,
                    reduce):
            ctx.save_for_backward(value, lidar2img, offsets, logits)
            ctx.meta = (anchors, grid, tuple(img_hw), tuple(levels), heads, reduce)
            return sca_forward(value, lidar2img, anchors, grid, img_hw, levels, heads, offsets,
                               logits, reduce=reduce)

        @staticmethod
        def backward(ctx, grad_out):
            value, l2i, off, lg = ctx.saved_tensors
            anchors, grid, img_hw, levels, heads, reduce = ctx.meta
            want = tuple(k for k, i in (("value", 0), ("offsets", 2), ("logits", 3))
                         if ctx.needs_input_grad[i])
            if not want:
                return (None,) * 10
            r = sca_backward(value, l2i, anchors, grid, img_hw, levels, heads, off, lg,
                             grad_out.float().contiguous(), want=want, reduce=reduce)
            gv = r["value"]
            if gv is not None and gv.dtype != value.dtype:
                gv = gv.to(value.dtype)
            return gv, None, r["offsets"], r["logits"], None, None, None, None, None, None

    _AUTOGRAD["sample_vt"] = _SampleVT
    _AUTOGRAD["sca"] = _SCA
    return _AUTOGRAD


def sample_vt_autograd(features, lidar2img, z_bins, grid: BevGrid, img_hw: Tuple[int, int],
                       reduce: str = "mean", method: str = "gather"):
    """``sample_vt`` as a differentiable function: the gradient with respect to
    ``features`` is ``sample_vt_backward`` (``method``), cast to the features'
    dtype; the camera matrices get none (they are fixed inputs of Eq. 1)."""
    return _autograd_functions()["sample_vt"].apply(features, lidar2img, z_bins, grid, img_hw,
                                                    reduce, method)


def sca_autograd(value, lidar2img, anchors, grid: BevGrid, img_hw: Tuple[int, int], levels,
                 heads: int, offsets, logits, reduce: str = "mean"):
    """``sca_forward`` as a differentiable function: the gradients with respect
    to ``value`` (cast to its dtype), ``offsets`` and ``logits`` are
    ``sca_backward``'s, computed only for the inputs that need them; the
    camera matrices and anchors get none."""
    return _autograd_functions()["sca"].apply(value, lidar2img, offsets, logits, anchors, grid,
                                              img_hw, levels, heads, reduce)
