"""Binding of the memory-ceiling micro-benchmarks (include/flashbev_membench.h).

Measurement tools for bench.py: the gather ceiling (the access shape of the
fused gather on an L2- or L1-resident buffer), the HBM read ceiling and the
float atomic-add ceiling.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libflashbev_membench.so")
_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_LIB_PATH):
            raise FileNotFoundError(f"{_LIB_PATH} is not built")
        L = ctypes.CDLL(_LIB_PATH)
        L.flashbev_membench_gather.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                               ctypes.c_void_p]
        L.flashbev_membench_gather.restype = ctypes.c_int
        L.flashbev_membench_stream.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32,
                                               ctypes.c_void_p, ctypes.c_void_p]
        L.flashbev_membench_stream.restype = ctypes.c_int
        L.flashbev_membench_atomic.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_void_p]
        L.flashbev_membench_atomic.restype = ctypes.c_int
        _LIB = L
    return _LIB


def cells_per_wave(row_bytes: int) -> int:
    return min(8, 64 // (row_bytes // 16))


def gather_bytes(workgroups: int, row_bytes: int, iters: int) -> int:
    return workgroups * 4 * cells_per_wave(row_bytes) * iters * 4 * row_bytes


def gather(buf, row_bytes: int, row_pitch: int, iters: int, workgroups: int, sink, stream: int,
           loads_in_flight: int = 8, lds_bytes: int = 0) -> None:
    rc = _lib().flashbev_membench_gather(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                                         row_bytes, row_pitch, iters, loads_in_flight, lds_bytes,
                                         workgroups, ctypes.c_void_p(sink.data_ptr()),
                                         ctypes.c_void_p(stream))
    if rc:
        raise RuntimeError(f"flashbev_membench_gather failed: {rc}")


def stream_read(buf, workgroups: int, sink, stream: int) -> None:
    rc = _lib().flashbev_membench_stream(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                                         workgroups, ctypes.c_void_p(sink.data_ptr()),
                                         ctypes.c_void_p(stream))
    if rc:
        raise RuntimeError(f"flashbev_membench_stream failed: {rc}")


def atomic_ops(workgroups: int, iters: int) -> int:
    return workgroups * 256 * iters


def atomic_add(buf, iters: int, workgroups: int, stream: int) -> None:
    rc = _lib().flashbev_membench_atomic(ctypes.c_void_p(buf.data_ptr()), buf.numel(), iters,
                                         workgroups, ctypes.c_void_p(stream))
    if rc:
        raise RuntimeError(f"flashbev_membench_atomic failed: {rc}")
