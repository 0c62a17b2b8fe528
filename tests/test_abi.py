"""C-ABI library: exported symbols and argument checks (CPU only).

Every argument check of flashbev_sample_vt runs before any HIP call, so the
error paths are exercised here without a GPU.  Device pointers below are
fake addresses that the library never dereferences because validation
rejects the call first.
"""
import ctypes
import math
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2607_10071_amd as fb
from paper_2607_10071_amd import Features, GridSpec, ZBins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashbev.h")


def declared_functions(header=HEADER):
    src = open(header).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(flash(?:bev|sca)_\w+)\s*\(", src)))


def exported(lib_path):
    out = subprocess.run(["nm", "-D", "--defined-only", lib_path],
                         capture_output=True, text=True, check=True).stdout
    return set(re.findall(r" T (flash(?:bev|sca)_\w+)", out))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert {"flashbev_sample_vt", "flashbev_status_string", "flashbev_abi_version",
            "flashbev_launch_info"} <= set(names)
    lib = ctypes.CDLL(fb.library_path())
    for n in names:
        assert hasattr(lib, n), n
    # everything declared is exported, and nothing else with the prefixes leaks
    sca = declared_functions(os.path.join(ROOT, "include", "flashsca.h"))
    assert exported(fb.library_path()) == set(names) | set(sca)


def test_every_header_maps_to_a_library_that_exports_it():
    from paper_2607_10071_amd import membench, phases
    libs = {"flashbev.h": [fb.library_path(), phases.LIB_PATH],
            "flashsca.h": [fb.library_path(), phases.LIB_PATH],
            "flashbev_membench.h": [membench._LIB_PATH],
            "flashbev_phases.h": [phases.LIB_PATH]}
    headers = sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))
    assert headers == sorted(libs)
    per_lib = {}
    for h in headers:
        names = declared_functions(os.path.join(ROOT, "include", h))
        assert names, h
        for lib in libs[h]:
            per_lib.setdefault(lib, set()).update(names)
    for lib, names in per_lib.items():
        ctypes.CDLL(lib)
        assert exported(lib) == names, lib


def test_abi_version_and_status_strings():
    assert fb.abi_version() == fb.ABI_VERSION
    for name, code in fb.STATUS.items():
        s = fb.status_string(code)
        assert s and s != "unknown status"
    assert fb.status_string(12345) == "unknown status"


def test_header_constants_match_binding():
    src = open(HEADER).read()
    for k, v in (("FLASHBEV_ZMAX", fb.ZMAX), ("FLASHBEV_NMAX", fb.NMAX),
                 ("FLASHBEV_ROW_BYTES_MAX", fb.ROW_BYTES_MAX), ("FLASHBEV_ABI_VERSION", fb.ABI_VERSION),
                 ("FLASHBEV_SCRATCH_BYTES", fb.SCRATCH_BYTES)):
        assert re.search(rf"#define {k} {v}\b", src), k
    for k, v in fb.STATUS.items():
        assert re.search(rf"FLASHBEV_{k} = {v}\b", src), k


FEAT = 0x7F0000000000  # fake, 256-byte aligned device addresses
L2I = 0x7F1000000000
OUT = 0x7F2000000000


def call(shape=(1, 6, 32, 88, 80), dtype="f32", img=(256, 704), X=200, Y=200, z=None,
         reduce="mean", feat=FEAT, l2i=L2I, out=OUT, grid=None, zptr_null=False, Z=None):
    z = np.linspace(-4.5, 2.5, 8).astype(np.float32) if z is None else np.asarray(z, np.float32)
    B, N, H, W, C = shape
    f = Features(feat, fb.DTYPE_CODES.get(dtype, dtype) if isinstance(dtype, str) else dtype,
                 B, N, H, W, C, img[0], img[1])
    g = grid or GridSpec(-50.0, 0.5, X, -50.0, 0.5, Y, 1e-5, fb.REDUCE_CODES.get(reduce, reduce)
                         if isinstance(reduce, str) else reduce)
    zb = ZBins(None if zptr_null else z.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
               len(z) if Z is None else Z)
    lib = fb._lib()
    return lib.flashbev_sample_vt(ctypes.byref(f), ctypes.c_void_p(l2i), ctypes.byref(g),
                                  ctypes.byref(zb), ctypes.c_void_p(out), ctypes.c_void_p(0))


S = fb.STATUS


def test_null_structs():
    lib = fb._lib()
    g = GridSpec(-50.0, 0.5, 4, -50.0, 0.5, 4, 1e-5, 0)
    z = np.zeros(2, np.float32)
    zb = ZBins(z.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), 2)
    f = Features(FEAT, 0, 1, 1, 2, 2, 4, 8, 8)
    assert lib.flashbev_sample_vt(None, ctypes.c_void_p(L2I), ctypes.byref(g), ctypes.byref(zb),
                                  ctypes.c_void_p(OUT), None) == S["ERR_NULLPTR"]
    assert lib.flashbev_sample_vt(ctypes.byref(f), ctypes.c_void_p(L2I), None, ctypes.byref(zb),
                                  ctypes.c_void_p(OUT), None) == S["ERR_NULLPTR"]
    assert lib.flashbev_sample_vt(ctypes.byref(f), ctypes.c_void_p(L2I), ctypes.byref(g), None,
                                  ctypes.c_void_p(OUT), None) == S["ERR_NULLPTR"]


@pytest.mark.parametrize("kw,status", [
    (dict(out=0), "ERR_NULLPTR"),
    (dict(feat=0), "ERR_NULLPTR"),
    (dict(l2i=0), "ERR_NULLPTR"),
    (dict(zptr_null=True), "ERR_NULLPTR"),
    (dict(dtype=7), "ERR_DTYPE"),
    (dict(dtype=-1), "ERR_DTYPE"),
    (dict(shape=(1, 6, 32, 88, 0)), "ERR_SHAPE"),
    (dict(shape=(-1, 6, 32, 88, 8)), "ERR_SHAPE"),
    (dict(shape=(1, -6, 32, 88, 8)), "ERR_SHAPE"),
    (dict(shape=(1, 6, 0, 88, 8)), "ERR_SHAPE"),
    (dict(shape=(1, 6, 32, 0, 8)), "ERR_SHAPE"),
    (dict(img=(0, 704)), "ERR_SHAPE"),
    (dict(img=(256, -1)), "ERR_SHAPE"),
    (dict(X=-1), "ERR_SHAPE"),
    (dict(Y=-3), "ERR_SHAPE"),
    (dict(Z=-1), "ERR_SHAPE"),
    (dict(z=np.zeros(257)), "ERR_UNSUPPORTED"),
    (dict(shape=(1, 65, 32, 88, 8)), "ERR_UNSUPPORTED"),
    (dict(shape=(1, 6, 32, 88, 1025)), "ERR_UNSUPPORTED"),
    (dict(shape=(1, 6, 32, 88, 2049), dtype="bf16"), "ERR_UNSUPPORTED"),
    (dict(shape=(64, 64, 128, 128, 64)), "ERR_UNSUPPORTED"),  # 17 GB of features
    (dict(shape=(1, 64, 128, 256, 256)), "ERR_UNSUPPORTED"),  # 2.1 GB of features
    (dict(X=50000, Y=50000), "ERR_UNSUPPORTED"),
    (dict(reduce=2), "ERR_VALUE"),
    (dict(grid=GridSpec(float("nan"), 0.5, 4, -1.0, 0.5, 4, 1e-5, 0)), "ERR_VALUE"),
    (dict(grid=GridSpec(-1.0, float("inf"), 4, -1.0, 0.5, 4, 1e-5, 0)), "ERR_VALUE"),
    (dict(grid=GridSpec(-1.0, 0.5, 4, -1.0, 0.5, 4, float("nan"), 0)), "ERR_VALUE"),
    (dict(feat=FEAT + 2), "ERR_ALIGN"),
    (dict(feat=FEAT + 1, dtype="bf16"), "ERR_ALIGN"),
    (dict(l2i=L2I + 2), "ERR_ALIGN"),
    (dict(out=OUT + 1), "ERR_ALIGN"),
    (dict(out=FEAT + 64), "ERR_ALIAS"),
    (dict(out=FEAT - 1024), "ERR_ALIAS"),
    (dict(out=L2I - 4), "ERR_ALIAS"),
])
def test_argument_errors_before_any_hip_call(kw, status):
    assert call(**kw) == S[status]


def test_size_products_do_not_wrap():
    # B N H W C s = 2^15 * 2^20 * 2^20 * 512 wraps 64 bits to 0: the call must
    # refuse it, not launch with an empty buffer and report success
    assert call(shape=(2**15, 1, 2**20, 2**20, 128), X=1, Y=1) == S["ERR_UNSUPPORTED"]
    # no features (N = 0) but B C X Y = 2^30 * 1024 * 2^30 output elements
    assert call(shape=(2**30, 0, 1, 1, 1024), X=2**15, Y=2**15) == S["ERR_UNSUPPORTED"]
    # the backward: B N H W C = 2^15 * 2^40 * 512 = 2^64 gradient elements
    z = np.linspace(-4.5, 2.5, 8).astype(np.float32)
    grid = fb.BevGrid(-50.0, 0.5, 1, -50.0, 0.5, 1)
    rc = fb.sample_vt_backward_raw((2**15, 1, 2**20, 2**20, 512), "f32", L2I, z, grid,
                                   (256, 704), OUT, FEAT)
    assert rc == S["ERR_UNSUPPORTED"]
    rc = fb.sample_vt_backward_raw((2**30, 0, 1, 1, 512), "f32", L2I, z,
                                   fb.BevGrid(-50.0, 0.5, 2**15, -50.0, 0.5, 2**15),
                                   (256, 704), OUT, FEAT)
    assert rc == S["ERR_UNSUPPORTED"]
    with pytest.raises(fb.FlashBevError):
        fb.launch_info((2**15, 1, 2**20, 2**20, 128), "f32", z, grid, (256, 704))


def test_empty_outputs_enqueue_nothing():
    # nothing to write: returns OK without touching HIP (this box has no GPU)
    assert call(X=0) == S["OK"]
    assert call(Y=0) == S["OK"]
    assert call(shape=(0, 6, 32, 88, 80)) == S["OK"]
    assert call(X=0, out=0, feat=0, l2i=0) == S["OK"]


def test_launch_info_geometry():
    for dtype, C, cpw, lpc in (("f32", 80, 3, 20), ("bf16", 128, 4, 16), ("f16", 64, 8, 8),
                               ("bf16", 64, 8, 8), ("f32", 32, 8, 8), ("f32", 4, 8, 1),
                               ("f32", 136, 3, 17), ("f32", 1024, 1, 64), ("bf16", 5, 8, 5)):
        info = fb.launch_info((1, 6, 32, 88, C), dtype, np.zeros(8), fb.BevGrid(-50, .5, 200, -50, .5, 200),
                              (256, 704))
        assert info["cells_per_wave"] == cpw and info["lanes_per_cell"] == lpc, (dtype, C, info)
        # 4 wavefronts per workgroup with full 8-cell groups, else 2
        waves = 4 if cpw == 8 else 2
        assert info["threads"] == 64 * waves
        # a tile is `waves` wavefronts x `rounds` groups of cpw cells: at
        # least 6 cells per wavefront, except one round where a wavefront
        # holds at most two cells or a lane several 16-byte vectors, or the
        # packed projection phase runs (groups of 4+ cells; N = 6, Z = 8)
        tiles = {math.ceil(40000 / (waves * r * cpw)): r for r in range(1, 9)}
        assert info["workgroups"] in tiles
        r = tiles[info["workgroups"]]
        vpl = math.ceil(C * (4 if dtype == "f32" else 2) / 16 / lpc)
        packed = cpw >= 4 and cpw * 6 <= 64
        if (cpw <= 2 or vpl >= 2 or packed) and 40000 <= waves * cpw * 262144:
            assert r == 1, (dtype, C, info)
        else:
            assert r * cpw >= 6, (dtype, C, info)
        assert info["lds_bytes"] <= 64 * 1024
    # a very large grid keeps several rounds per tile (fewer workgroups)
    info = fb.launch_info((1, 6, 56, 100, 128), "f32", np.zeros(8),
                          fb.BevGrid(-50, 0.0625, 1600, -50, 0.0625, 1600), (448, 800))
    assert info["workgroups"] == math.ceil(1600 * 1600 / (2 * 3 * info["cells_per_wave"]))
    with pytest.raises(fb.FlashBevError):
        fb.launch_info((1, 6, 32, 88, 80), "f32", np.zeros(300), fb.BevGrid(-50, .5, 200, -50, .5, 200),
                       (256, 704))


def test_binding_rejects_host_tensors():
    import torch
    f = torch.zeros(1, 1, 2, 2, 4)
    m = torch.zeros(1, 1, 4, 4)
    with pytest.raises(ValueError):
        fb.sample_vt(f, m, [0.0], fb.BevGrid(-1, 1, 2, -1, 1, 2), (8, 8))
    with pytest.raises(ValueError):
        fb.prepare_sample_vt(f, m, [0.0], fb.BevGrid(-1, 1, 2, -1, 1, 2), (8, 8),
                             torch.zeros(1, 4, 2, 2))
    with pytest.raises(ValueError):
        fb.sample_vt_backward(torch.zeros(1, 4, 2, 2), m, [0.0], fb.BevGrid(-1, 1, 2, -1, 1, 2),
                              (8, 8), (1, 1, 2, 2, 4))
    with pytest.raises(ValueError):
        fb.prepare_sample_vt_backward(torch.zeros(1, 4, 2, 2), m, [0.0],
                                      fb.BevGrid(-1, 1, 2, -1, 1, 2), (8, 8), (1, 1, 2, 2, 4),
                                      "f32", f)


class _OnDevice:
    """A host tensor that reports itself as a device tensor: the binding's
    checks read only its shape, dtype, layout and device flag, and each case
    below must be rejected by them before any pointer is taken."""

    def __init__(self, t):
        self._t = t
        self.is_cuda = True
        self.device = t.device

    def __getattr__(self, name):
        return getattr(self._t, name)

    def data_ptr(self):
        raise AssertionError("a malformed tensor reached the C call")


def test_prepared_calls_reject_malformed_tensors():
    import torch
    D = _OnDevice
    grid = fb.BevGrid(-1, 1, 2, -1, 1, 3)
    feats = D(torch.zeros(1, 2, 4, 4, 8))
    l2i = D(torch.zeros(1, 2, 4, 4))
    out = D(torch.zeros(1, 8, 2, 3))
    gout = D(torch.zeros(1, 8, 2, 3))
    gfeat = D(torch.zeros(1, 2, 4, 4, 8))
    bad_fwd = [
        ("features", D(torch.zeros(1, 2, 4, 8, 4).transpose(3, 4))),   # strided
        ("features", D(torch.zeros(1, 2, 4, 4, 8, dtype=torch.float64))),
        ("lidar2img", D(torch.zeros(1, 2, 3, 4))),
        ("lidar2img", D(torch.zeros(1, 2, 4, 4, dtype=torch.float64))),
        ("lidar2img", D(torch.zeros(1, 2, 4, 4).transpose(2, 3))),
        ("out", D(torch.zeros(1, 8, 3, 2))),
        ("out", D(torch.zeros(1, 8, 3, 2).transpose(2, 3))),
    ]
    for name, t in bad_fwd:
        kw = {"features": feats, "lidar2img": l2i, "out": out, name: t}
        for fn in (fb.prepare_sample_vt, fb.sample_vt):
            with pytest.raises((ValueError, TypeError)):
                fn(kw["features"], kw["lidar2img"], [0.0], grid, (8, 8), out=kw["out"])
    bad_bwd = [
        ("grad_out", D(torch.zeros(1, 8, 3, 2))),
        ("grad_out", D(torch.zeros(1, 8, 3, 2).transpose(2, 3))),
        ("grad_out", D(torch.zeros(1, 8, 2, 3, dtype=torch.float16))),
        ("lidar2img", D(torch.zeros(1, 2, 3, 4))),
        ("lidar2img", D(torch.zeros(1, 2, 4, 4, dtype=torch.float64))),
        ("grad_features", D(torch.zeros(1, 2, 4, 4, 4))),
        ("grad_features", D(torch.zeros(1, 2, 4, 8, 4).transpose(3, 4))),
    ]
    for name, t in bad_bwd:
        kw = {"grad_out": gout, "lidar2img": l2i, "grad_features": gfeat, name: t}
        with pytest.raises(ValueError):
            fb.prepare_sample_vt_backward(kw["grad_out"], kw["lidar2img"], [0.0], grid, (8, 8),
                                          (1, 2, 4, 4, 8), "f32", kw["grad_features"])
        with pytest.raises(ValueError):
            fb.sample_vt_backward(kw["grad_out"], kw["lidar2img"], [0.0], grid, (8, 8),
                                  (1, 2, 4, 4, 8), "f32", kw["grad_features"])


def test_binding_requires_one_device_per_call():
    import torch
    a, b = torch.zeros(2), torch.zeros(2, device="meta")
    assert fb._one_device(a, None, torch.ones(3)) == torch.device("cpu")
    with pytest.raises(ValueError, match="one CUDA device"):
        fb._one_device(a, b)
    with pytest.raises(ValueError):
        fb._one_device(None)


def test_backward_launch_info_geometry():
    """Tiled mode where pixel ids fit 20 bits and rows have at most 512
    channels: 8-wavefront workgroups within the tiled LDS budget (two per
    CU); direct mode otherwise."""
    grid = fb.BevGrid(-50, .5, 200, -50, .5, 200)
    for dtype, C, tiled in (("f32", 80, True), ("bf16", 128, True), ("f16", 64, True),
                            ("f32", 32, True), ("f32", 1, True), ("f32", 256, True),
                            ("bf16", 512, True), ("f32", 513, False), ("f32", 1024, False),
                            ("bf16", 2048, False)):
        info = fb.backward_launch_info((1, 6, 32, 88, C), dtype, np.zeros(8), grid, (256, 704))
        lpc = min(64, (C + 3) // 4)
        assert info["lanes_per_cell"] == lpc, (C, info)
        assert (info["rows_per_tile"] > 0) == tiled, (C, info)
        if tiled:
            assert info["rows_per_tile"] >= 16 and info["threads"] == 512
            assert info["lds_bytes"] <= 80 * 1024
            cpw = min(8, 64 // lpc)
            T = 8 * cpw
            ty = 4 if T % 4 == 0 else T
            assert info["workgroups"] == math.ceil(200 / (T // ty)) * math.ceil(200 / ty)
        else:
            assert info["lds_bytes"] <= 64 * 1024
    # more than 2^20 - 1 pixels per batch element: direct mode
    info = fb.backward_launch_info((1, 64, 128, 128, 16), "f32", np.zeros(4), grid, (512, 512))
    assert info["rows_per_tile"] == 0
    # nothing to scatter when the grid is empty; the fill still runs in the call
    info = fb.backward_launch_info((1, 6, 32, 88, 80), "f32", np.zeros(8),
                                   fb.BevGrid(-50, .5, 0, -50, .5, 200), (256, 704))
    assert info["workgroups"] == 0
    with pytest.raises(fb.FlashBevError):
        fb.backward_launch_info((1, 6, 32, 88, 80), "f32", np.zeros(300), grid, (256, 704))


@pytest.mark.parametrize("X,Y", [(1, 2**31 - 1), (2**31 - 1, 1), (2**31 - 64, 1), (1, 2**31 - 200)])
def test_backward_plan_on_extreme_grid_sides(X, Y):
    # a grid side near 2^31 must not overflow the tiled backward's tile count
    # (found by the property test: 1 x (2^31 - 1) gave a negative count)
    grid = fb.BevGrid(-50.0, 0.5, X, -50.0, 0.5, Y)
    try:
        info = fb.backward_launch_info((1, 1, 1, 1, 1), "f32", np.zeros(1, np.float32), grid, (1, 1))
    except fb.FlashBevError as e:
        assert e.status != 0
        return
    assert 0 < info["workgroups"] <= 2**31 - 1


WS = 0x7F3000000000  # fake workspace address


def test_gather_backward_workspace_size():
    """Gt (float32 B X Y C) then den_z (uint8 B X Y Z), each padded to 256
    bytes; -1 (the scatter form serves it) where Gt would reach 2^31 bytes."""
    grid = fb.BevGrid(-50, .5, 200, -50, .5, 200)
    z = np.linspace(-4.5, 2.5, 8).astype(np.float32)
    for B, C, Z in ((1, 80, 8), (4, 128, 8), (2, 64, 8), (1, 1, 1), (3, 7, 13)):
        zz = np.linspace(-4, 2, Z).astype(np.float32)
        got = fb.backward_workspace_size((B, 6, 32, 88, C), "f32", zz, grid, (256, 704))
        gt = B * 200 * 200 * C * 4
        den = B * 200 * 200 * Z
        assert got == -(-gt // 256) * 256 + -(-den // 256) * 256, (B, C, Z)
    big = fb.BevGrid(-50, .5, 4096, -50, .5, 4096)
    assert fb.backward_workspace_size((1, 6, 32, 88, 64), "f32", z, big, (256, 704)) == -1
    with pytest.raises(fb.FlashBevError):
        fb.backward_workspace_size((1, 6, 32, 88, 80), "f32", np.zeros(300), grid, (256, 704))


@pytest.mark.parametrize("kw,status", [
    (dict(ws=0), "ERR_NULLPTR"),
    (dict(ws=WS + 16), "ERR_ALIGN"),
    (dict(ws_bytes=-1), "ERR_VALUE"),
    (dict(ws=OUT), "ERR_ALIAS"),
    (dict(ws=FEAT - 256), "ERR_ALIAS"),
    (dict(ws=L2I), "ERR_ALIAS"),
    (dict(gout=0), "ERR_NULLPTR"),
    (dict(gout=OUT + 2), "ERR_ALIGN"),
    (dict(shape=(1, 6, 32, 88, 1025)), "ERR_UNSUPPORTED"),
    (dict(X=4096, Y=4096), "ERR_UNSUPPORTED"),
    (dict(reduce=2), "ERR_VALUE"),
])
def test_gather_backward_argument_errors(kw, status):
    """Every check of flashbev_sample_vt_backward_ws precedes its first HIP
    call; ws_bytes=-1 means one byte fewer than the workspace needs."""
    shape = kw.get("shape", (1, 6, 32, 88, 80))
    X, Y = kw.get("X", 200), kw.get("Y", 200)
    grid = fb.BevGrid(-50, .5, X, -50, .5, Y)
    z = np.linspace(-4.5, 2.5, 8).astype(np.float32)
    reduce = kw.get("reduce", "mean")
    try:
        need = fb.backward_workspace_size(shape, "f32", z, grid, (256, 704))
    except fb.FlashBevError:
        need = 0
    ws_bytes = kw.get("ws_bytes", need)
    if ws_bytes == -1:
        ws_bytes = need - 1
    if reduce == 2:
        f, g, zb = fb._structs(shape, 0, 0, (256, 704), grid, z, "mean")
        g.reduce = 2
        rc = fb._lib().flashbev_sample_vt_backward_ws(
            ctypes.byref(f), ctypes.c_void_p(L2I), ctypes.byref(g), ctypes.byref(zb),
            ctypes.c_void_p(OUT), ctypes.c_void_p(FEAT), ctypes.c_void_p(WS),
            ctypes.c_uint64(need), ctypes.c_void_p(0))
    else:
        rc = fb.sample_vt_backward_ws_raw(shape, "f32", L2I, z, grid, (256, 704),
                                          kw.get("gout", OUT), FEAT, kw.get("ws", WS),
                                          max(ws_bytes, 0))
    assert rc == S[status]


def test_gather_backward_empty_shapes_enqueue_nothing():
    grid = fb.BevGrid(-50, .5, 200, -50, .5, 200)
    z = np.linspace(-4.5, 2.5, 8).astype(np.float32)
    for shape in ((0, 6, 32, 88, 80), (1, 0, 32, 88, 80)):
        assert fb.sample_vt_backward_ws_raw(shape, "f32", L2I, z, grid, (256, 704), OUT, FEAT,
                                            0, 0) == S["OK"]


def test_noalloc_backward_checks_before_any_hip_call():
    """flashbev_sample_vt_backward_noalloc: argument errors, then the static
    scratch's limit, all before any HIP call (this box has no GPU)."""
    grid = fb.BevGrid(-50, .5, 200, -50, .5, 200)
    z = np.linspace(-4.5, 2.5, 8).astype(np.float32)
    shape = (1, 6, 32, 88, 80)
    raw = fb.sample_vt_backward_noalloc_raw
    assert raw(shape, "f32", L2I, z, grid, (256, 704), 0, FEAT) == S["ERR_NULLPTR"]
    assert raw(shape, "f32", L2I, z, grid, (256, 704), OUT + 2, FEAT) == S["ERR_ALIGN"]
    assert raw(shape, "f32", L2I, z, grid, (256, 704), OUT, OUT) == S["ERR_ALIAS"]
    assert raw((1, 6, 32, 88, 1025), "f32", L2I, z, grid, (256, 704), OUT, FEAT) == \
        S["ERR_UNSUPPORTED"]
    # 4 x 200 x 200 x 128 float32 rows of Gt: 82 MB, above the 64 MiB scratch
    need = fb.backward_workspace_size((4, 6, 32, 88, 128), "bf16", z, grid, (256, 704))
    assert need > fb.SCRATCH_BYTES
    assert raw((4, 6, 32, 88, 128), "bf16", L2I, z, grid, (256, 704), OUT, FEAT) == \
        S["ERR_SCRATCH"]
    # nothing to do: no HIP call either
    assert raw((0, 6, 32, 88, 80), "f32", L2I, z, grid, (256, 704), OUT, FEAT) == S["OK"]
    assert fb.status_string(S["ERR_SCRATCH"]) != "unknown status"


def test_autograd_wrappers_are_exported_and_refuse_host_tensors():
    # the differentiable wrappers marshal to the same C calls; on host
    # tensors they raise rather than compute anything
    import torch
    import paper_2607_10071_amd as fb
    assert "sample_vt_autograd" in fb.__all__ and "sca_autograd" in fb.__all__
    fns = fb._autograd_functions()
    assert issubclass(fns["sample_vt"], torch.autograd.Function)
    assert issubclass(fns["sca"], torch.autograd.Function)
    feats = torch.zeros((1, 1, 2, 2, 4), requires_grad=True)
    l2i = torch.eye(4).reshape(1, 1, 4, 4)
    grid = fb.BevGrid(x_min=-1.0, dx=1.0, X=2, y_min=-1.0, dy=1.0, Y=2)
    with pytest.raises(ValueError):
        fb.sample_vt_autograd(feats, l2i, [0.0], grid, (8, 8))
