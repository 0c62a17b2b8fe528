"""FlashSCA C ABI: argument checks and launch geometry (CPU only).

Every check of flashsca_forward runs before any HIP call, so the error paths
run here without a GPU.  Device pointers are fake addresses that the library
never dereferences because validation rejects the call first.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_10071_amd as fb
from paper_2607_10071_amd import GridSpec, ScaValue, ZBins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
S = fb.STATUS
VAL = 0x7F0000000000   # fake, 256-byte aligned device addresses
L2I = 0x7F1000000000
OFF = 0x7F2000000000
LOG = 0x7F3000000000
OUT = 0x7F4000000000
LEVELS = ((116, 200), (58, 100), (29, 50), (15, 25))


def call(B=1, N=6, C=256, heads=8, levels=LEVELS, dtype="f32", img=(900, 1600), X=200, Y=200,
         z=(-4.5, -2.1666667, 0.16666667, 2.5), P=8, reduce="mean", val=VAL, l2i=L2I, off=OFF,
         log=LOG, out=OUT, L=None, grid=None, zptr_null=False, Z=None, level_override=None):
    z = np.asarray(z, np.float32)
    nl = len(levels)
    lh = (ctypes.c_int32 * 8)(*[h for h, _ in levels], *([0] * (8 - nl)))
    lw = (ctypes.c_int32 * 8)(*[w for _, w in levels], *([0] * (8 - nl)))
    if level_override:
        i, h, w = level_override
        lh[i], lw[i] = h, w
    v = ScaValue(val, fb.DTYPE_CODES.get(dtype, dtype) if isinstance(dtype, str) else dtype,
                 B, N, C, heads, nl if L is None else L, lh, lw, img[0], img[1])
    g = grid or GridSpec(-51.2, 0.512, X, -51.2, 0.512, Y, 1e-5,
                         fb.REDUCE_CODES.get(reduce, reduce) if isinstance(reduce, str) else reduce)
    zb = ZBins(None if zptr_null else z.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
               len(z) if Z is None else Z)
    return fb._lib().flashsca_forward(ctypes.byref(v), ctypes.c_void_p(l2i), ctypes.byref(g),
                                      ctypes.byref(zb), P, ctypes.c_void_p(off),
                                      ctypes.c_void_p(log), ctypes.c_void_p(out),
                                      ctypes.c_void_p(0))


def test_header_constants_match_binding():
    src = open(os.path.join(ROOT, "include", "flashsca.h")).read()
    for k, v in (("FLASHSCA_LMAX", fb.SCA_LMAX), ("FLASHSCA_NMAX", fb.SCA_NMAX),
                 ("FLASHSCA_ZMAX", fb.SCA_ZMAX), ("FLASHSCA_LPMAX", fb.SCA_LPMAX),
                 ("FLASHSCA_HEAD_BYTES_MAX", fb.SCA_HEAD_BYTES_MAX)):
        assert re.search(rf"#define {k} {v}\b", src), k


def test_null_structs():
    lib = fb._lib()
    assert lib.flashsca_forward(None, None, None, None, 8, None, None, None, None) == S["ERR_NULLPTR"]
    assert lib.flashsca_launch_info(None, None, None, 8, None, None, None, None, None) == \
        S["ERR_NULLPTR"]


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), "ERR_DTYPE"),
    (dict(B=-1), "ERR_SHAPE"),
    (dict(N=-1), "ERR_SHAPE"),
    (dict(C=0), "ERR_SHAPE"),
    (dict(heads=0), "ERR_SHAPE"),
    (dict(C=255), "ERR_SHAPE"),                      # C % heads != 0
    (dict(L=0), "ERR_SHAPE"),
    (dict(L=9), "ERR_UNSUPPORTED"),
    (dict(level_override=(2, 0, 50)), "ERR_SHAPE"),
    (dict(img=(0, 1600)), "ERR_SHAPE"),
    (dict(X=-1), "ERR_SHAPE"),
    (dict(P=0), "ERR_SHAPE"),
    (dict(P=6), "ERR_SHAPE"),                        # P % Z != 0
    (dict(z=()), "ERR_SHAPE"),                       # no anchors
    (dict(z=np.zeros(33)), "ERR_UNSUPPORTED"),       # Z > ZMAX (P stays a multiple)
    (dict(N=33), "ERR_UNSUPPORTED"),
    (dict(P=132), "ERR_UNSUPPORTED"),                # L * P > 512
    (dict(C=2048, heads=4), "ERR_UNSUPPORTED"),      # 2 KiB head rows
    (dict(levels=((30000, 30000),)), "ERR_UNSUPPORTED"),  # one camera over 2 GiB
    (dict(zptr_null=True), "ERR_NULLPTR"),
    (dict(reduce=3), "ERR_VALUE"),
    (dict(grid=GridSpec(float("nan"), 0.5, 10, 0.0, 0.5, 10, 1e-5, 0)), "ERR_VALUE"),
    (dict(out=0), "ERR_NULLPTR"),
    (dict(off=0), "ERR_NULLPTR"),
    (dict(log=0), "ERR_NULLPTR"),
    (dict(val=0), "ERR_NULLPTR"),
    (dict(l2i=0), "ERR_NULLPTR"),
    (dict(val=VAL + 2), "ERR_ALIGN"),
    (dict(val=VAL + 2, dtype="bf16"), "ERR_ALIAS"),   # 2-byte aligned bf16 is fine; see below
    (dict(out=OUT + 2), "ERR_ALIGN"),
    (dict(off=OFF + 4), "ERR_ALIGN"),                # offsets travel as float2
    (dict(log=LOG + 1), "ERR_ALIGN"),
    (dict(l2i=L2I + 2), "ERR_ALIGN"),
    (dict(out=VAL + 4096), "ERR_ALIAS"),
    (dict(out=OFF), "ERR_ALIAS"),
    (dict(out=LOG + 64), "ERR_ALIAS"),
])
def test_argument_errors_before_any_hip_call(kw, status):
    if kw.get("dtype") == "bf16" and kw.get("val") == VAL + 2:
        # a bf16 value at a 2-byte aligned address passes alignment; make the
        # output overlap it so the call still fails before any HIP call
        kw = dict(kw, out=VAL + 64)
    if "z" in kw and len(kw["z"]) == 33:
        kw = dict(kw, P=33)
    assert call(**kw) == S[status], kw


def test_size_products_do_not_wrap():
    # B Q C = (2^31 - 1) * 10^8 * 256 output elements wraps 64 bits; with no
    # cameras there is no value tensor to reject it first
    assert call(B=2**31 - 1, N=0, X=10000, Y=10000) == S["ERR_UNSUPPORTED"]
    # eight levels near 2^31 pixels each: their sum no longer fits a camera
    big = tuple((46340, 46340) for _ in range(8))
    assert call(levels=big, C=8, heads=1) == S["ERR_UNSUPPORTED"]


def test_empty_outputs_enqueue_nothing():
    # B = 0 or an empty grid: OK without touching the (null) device pointers
    assert call(B=0, val=0, l2i=0, off=0, log=0, out=0) == S["OK"]
    assert call(X=0, val=0, l2i=0, off=0, log=0, out=0) == S["OK"]


def info(**kw):
    d = dict(shape=(1, 6, sum(h * w for h, w in LEVELS), 256), dtype="f32", heads=8,
             levels=LEVELS, anchors=[-4.5, -2.2, 0.2, 2.5],
             grid=fb.BevGrid(-51.2, 0.512, 200, -51.2, 0.512, 200), img_hw=(900, 1600), P=8)
    d.update(kw)
    return fb.sca_launch_info(**d)


def test_launch_geometry():
    # BEVFormer-base: 8 lanes of 16 bytes per head, 8 heads per wavefront,
    # 4 wavefronts (4 queries) per workgroup
    g = info()
    assert (g["lanes_per_head"], g["lane_bytes"], g["threads"]) == (8, 16, 256)
    assert g["workgroups"] == 200 * 200 // 4
    # bfloat16: 16-byte lanes, 4 per head, two queries per wavefront
    g = info(dtype="bf16")
    assert (g["lanes_per_head"], g["lane_bytes"]) == (4, 16)
    assert g["workgroups"] == 200 * 200 // 8
    # D = 64 float32: 16 lanes per head, 4 heads per wavefront
    g = info(shape=(1, 6, 30825, 512))
    assert (g["lanes_per_head"], g["lane_bytes"]) == (16, 16)
    assert g["workgroups"] == 200 * 200 * 8 // 16
    # D = 3 float32: three 4-byte lanes padded to four
    g = info(shape=(1, 6, 30825, 12), heads=4)
    assert (g["lanes_per_head"], g["lane_bytes"]) == (4, 4)
    # D = 8 float32 (32-byte head rows): four 8-byte lanes
    g = info(shape=(1, 6, 30825, 32), heads=4)
    assert (g["lanes_per_head"], g["lane_bytes"]) == (4, 8)
    # a value base that is only 4-byte aligned narrows the lanes
    g = fb.sca_launch_info((1, 6, 30825, 256), "f32", 8, LEVELS, [0.0],
                           fb.BevGrid(-51.2, 0.512, 200, -51.2, 0.512, 200), (900, 1600), 1,
                           data_ptr=VAL + 4)
    assert (g["lanes_per_head"], g["lane_bytes"]) == (32, 4)
    # LDS grows with L * P; past the budget the workgroup shrinks
    lds = [info(P=p)["lds_bytes"] for p in (8, 16, 32)]
    assert lds[0] < lds[1] < lds[2] <= 64 * 1024
    g = info(P=128, levels=LEVELS, anchors=[0.0, 1.0, 2.0, 3.0])
    assert g["threads"] < 256 and g["lds_bytes"] <= 64 * 1024


def test_binding_rejects_host_tensors():
    import torch
    with pytest.raises(ValueError):
        fb.sca_forward(torch.zeros(1, 6, 16, 8), torch.zeros(1, 6, 4, 4), [0.0],
                       fb.BevGrid(0, 1, 2, 0, 1, 2), (32, 32), ((4, 4),), 2,
                       torch.zeros(1, 4, 2, 1, 1, 2), torch.zeros(1, 4, 2, 1, 1))


GV = 0x7F5000000000
GO = 0x7F6000000000
GL = 0x7F7000000000
GOUT = 0x7F8000000000


def bcall(gv=GV, go=GO, gl=GL, gout=GOUT, **kw):
    """flashsca_backward with fake addresses (rejected before any HIP call
    in every case below)."""
    z = np.asarray(kw.pop("z", (-4.5, -2.1666667, 0.16666667, 2.5)), np.float32)
    lh = (ctypes.c_int32 * 8)(*[h for h, _ in LEVELS], *([0] * 4))
    lw = (ctypes.c_int32 * 8)(*[w for _, w in LEVELS], *([0] * 4))
    v = ScaValue(kw.pop("val", VAL), 0, 1, 6, 256, 8, 4, lh, lw, 900, 1600)
    g = GridSpec(-51.2, 0.512, 200, -51.2, 0.512, 200, 1e-5, 0)
    zb = ZBins(z.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), len(z))
    return fb._lib().flashsca_backward(ctypes.byref(v), ctypes.c_void_p(L2I), ctypes.byref(g),
                                       ctypes.byref(zb), 8, ctypes.c_void_p(kw.pop("off", OFF)),
                                       ctypes.c_void_p(LOG), ctypes.c_void_p(gout),
                                       ctypes.c_void_p(gv), ctypes.c_void_p(go),
                                       ctypes.c_void_p(gl), ctypes.c_void_p(0))


@pytest.mark.parametrize("kw,status", [
    (dict(gv=0, go=0, gl=0), "ERR_NULLPTR"),       # no gradient requested
    (dict(gout=0), "ERR_NULLPTR"),
    (dict(val=0), "ERR_NULLPTR"),
    (dict(go=GO + 4), "ERR_ALIGN"),                # offsets gradient travels as float2
    (dict(gl=GL + 2), "ERR_ALIGN"),
    (dict(gv=GV + 1), "ERR_ALIGN"),
    (dict(gv=VAL), "ERR_ALIAS"),                   # over the value maps
    (dict(go=LOG), "ERR_ALIAS"),                   # over the logits
    (dict(gl=GOUT), "ERR_ALIAS"),                  # over the output gradient
    (dict(gl=GO + 64), "ERR_ALIAS"),               # two outputs overlap
])
def test_backward_argument_errors_before_any_hip_call(kw, status):
    assert bcall(**kw) == S[status], kw


def test_backward_launch_geometry():
    d = dict(shape=(1, 6, sum(h * w for h, w in LEVELS), 256), dtype="f32", heads=8,
             levels=LEVELS, anchors=[-4.5, -2.2, 0.2, 2.5],
             grid=fb.BevGrid(-51.2, 0.512, 200, -51.2, 0.512, 200), img_hw=(900, 1600), P=8)
    f = fb.sca_launch_info(**d)
    b = fb.sca_launch_info(**d, backward=True)
    # same lanes; a backward tile holds 64 queries (8 wavefronts of 8) of one
    # head, twice the forward's workgroup, and the backward keeps
    # output-gradient rows, wider chunk records and a row-merge table in LDS
    # (within 80 KiB)
    assert (b["lanes_per_head"], b["lane_bytes"]) == (f["lanes_per_head"], f["lane_bytes"])
    assert (b["threads"], f["threads"]) == (512, 256)
    assert b["workgroups"] == (200 * 200 // 64) * 8
    assert f["lds_bytes"] < b["lds_bytes"] <= 80 * 1024
    # the backward keeps no per-point state in LDS: its size does not grow
    # with L * P, while the forward's attention weights do
    d2 = dict(d, shape=(1, 6, 30825, 32), heads=4, P=128)
    b2 = fb.sca_launch_info(**d2, backward=True)
    assert b2["lds_bytes"] == fb.sca_launch_info(**dict(d2, P=8), backward=True)["lds_bytes"]
    assert b2["threads"] == 512 and b2["lds_bytes"] <= 80 * 1024
    # the backward takes 8 lanes per head where it can: D = 8 float32 in
    # 4-byte lanes, 8 queries per wavefront, 64 per tile: Q / 64 tiles per head
    assert (b2["lanes_per_head"], b2["lane_bytes"]) == (8, 4)
    assert b2["workgroups"] == 200 * 200 // 64 * 4
    # bfloat16 BEVFormer-base: 8-byte lanes in the backward, 16-byte ones in
    # the forward
    bb = fb.sca_launch_info(**dict(d, dtype="bf16"), backward=True)
    fbf = fb.sca_launch_info(**dict(d, dtype="bf16"))
    assert (bb["lanes_per_head"], bb["lane_bytes"]) == (8, 8)
    assert (fbf["lanes_per_head"], fbf["lane_bytes"]) == (4, 16)
    # L * P = 512 with 16 slots per wavefront: the forward's attention
    # weights leave room for one wavefront within the 64 KiB budget
    f2 = fb.sca_launch_info(**d2)
    assert f2["threads"] == 64 and 32 * 1024 < f2["lds_bytes"] <= 64 * 1024
    # one head: still eight wavefronts, of 64 / lanes_per_head queries each,
    # one head per tile
    b3 = fb.sca_launch_info(**dict(d, shape=(1, 6, 30825, 32), heads=1), backward=True)
    assert b3["threads"] == 512 and b3["workgroups"] == -(-200 * 200 // (8 * 64 // b3["lanes_per_head"]))
