"""GPU parity of the backward (gradient w.r.t. the feature maps) against the oracle.

Bar (per gradient element): |gpu - oracle| <= (K + 8) * 2^-24 * S, where S
is the oracle's sum of |terms| for that element and K the number of terms
reaching its pixel.  Derivation: each float32 term w * g carries at most
about seven roundings (the bilinear fractions, the weight products, the
approximate reciprocal of den_z, the product with g), and float32 atomic
addition of K terms in any order adds at most (K - 1) roundings of partial
sums no larger than S.  Elements no term reaches must be exactly zero.
The gather form (flashbev_sample_vt_backward_ws) sums each element's terms
in a fixed order with fused multiply-adds: K roundings of partial sums, the
same bar.  Every test runs both forms; the gather form must in addition be
bitwise reproducible.  All calls go through the C ABI via the thin binding.

The full-size workloads cover every path of the tiled scatter: long_range's
heavy tiles claim more distinct pixels in a pass than a tile has LDS rows
(those taps go to global atomics), and the height sweep up to Z = 64 runs up
to 16 passes per tile, so tiles flush their rows and start again mid-tile.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
METHODS = ("gather", "scatter")
_ORACLE = {}


@pytest.fixture(scope="module")
def fb():
    import paper_2607_10071_amd as m
    return m


def _grad_out(wl, seed=3):
    rng = np.random.default_rng([wl.cfg_id, 7, seed])
    return rng.standard_normal((wl.B, wl.C, wl.X, wl.Y)).astype(np.float32)


def oracle_backward(inst, g, reduce="mean"):
    """The oracle's gradient, computed once per instance for both forms."""
    key = (repr(inst.wl), float(np.sum(inst.lidar2img.astype(np.float64))), float(g.sum()),
           reduce)
    if key not in _ORACLE:
        _ORACLE.clear()
        _ORACLE[key] = oracle.backward_instance(inst, g, reduce)
    return _ORACLE[key]


def gpu_backward(fb, inst, g, device, reduce="mean", prefill=None, method="gather"):
    import torch
    wl = inst.wl
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(g).to(device)
    gf = None
    if prefill is not None:
        gf = torch.full(inst.features.shape, prefill, dtype=torch.float32, device=device)
    gf = fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                               inst.features.shape, wl.dtype, grad_features=gf, reduce=reduce,
                               method=method)
    torch.cuda.synchronize()
    return gf.cpu().numpy()


def assert_bwd_parity(gpu, ref, scale, terms, what=""):
    gpu = gpu.astype(np.float64)
    err = np.abs(gpu - ref)
    tol = (terms[..., None].astype(np.float64) + 8.0) * U * scale
    bad = err > tol
    nz = scale > 0
    worst = float((err[nz] / scale[nz]).max(initial=0.0))
    print(f"[parity-bwd] {what} max_abs={err.max(initial=0):.3e} max_scaled={worst:.3e} "
          f"max_terms={int(terms.max(initial=0))}", flush=True)
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} elements off (max scaled {worst:.3e})"
    assert np.all(gpu[~nz] == 0.0), f"{what}: untouched elements are not zero"


def check(fb, inst, device, reduce="mean", what="", prefill=None, method="gather"):
    print(f"[case] backward {method} {what} shape={inst.features.shape} X={inst.wl.X} "
          f"Y={inst.wl.Y} Z={len(inst.z)} reduce={reduce}", flush=True)
    g = _grad_out(inst.wl)
    gpu = gpu_backward(fb, inst, g, device, reduce, prefill, method)
    ref, scale, terms = oracle_backward(inst, g, reduce)
    assert gpu.shape == ref.shape
    assert_bwd_parity(gpu, ref, scale, terms, f"{method} {what}")
    wl = inst.wl
    served = fb.backward_workspace_size(inst.features.shape, wl.dtype, inst.z, fb.grid_of(wl),
                                        (wl.img_h, wl.img_w), reduce) >= 0
    if method == "gather" and served:
        again = gpu_backward(fb, inst, g, device, reduce, None, method)
        assert np.array_equal(gpu.view(np.uint32), again.view(np.uint32)), \
            f"{what}: the gather form is not bitwise reproducible"
    return gpu, ref, terms


@pytest.mark.parametrize("wl", synth.all_parity_workloads(), ids=lambda w: f"{w.name}-Z{w.Z}")
@pytest.mark.parametrize("method", METHODS)
def test_backward_workloads_full(fb, device, wl, method):
    inst = synth.make_workload(wl)
    _, _, terms = check(fb, inst, device, what=f"{wl.name} Z={wl.Z}", method=method)
    assert terms.sum() > 0


@pytest.mark.parametrize("C", [128, 256])
@pytest.mark.parametrize("method", METHODS)
def test_backward_paper_reference_setting(fb, device, C, method):
    """The paper's reference setting in full; C = 256 takes the tiled mode's
    wide-row path (channel blocks beyond two per lane)."""
    inst = synth.make_workload(synth.config("paper_ref", C=C))
    check(fb, inst, device, what=f"paper_ref C={C}", method=method)


@pytest.mark.parametrize("reduce", ["mean", "sum"])
@pytest.mark.parametrize("method", METHODS)
def test_backward_reduce_modes(fb, device, reduce, method):
    inst = synth.make_workload(synth.config("tiny"))
    check(fb, inst, device, reduce, what=f"tiny {reduce}", method=method)


@pytest.mark.parametrize("C,dtype", [(1, "f32"), (5, "f32"), (7, "bf16"), (36, "f16"),
                                     (128, "f32"), (129, "f32"), (192, "f32"), (256, "bf16"),
                                     (260, "f32"), (512, "f32"), (512, "f16"),
                                     (1024, "f32"), (2048, "bf16")])
@pytest.mark.parametrize("method", METHODS)
def test_backward_channel_counts(fb, device, C, dtype, method):
    wl = synth.config("tiny").with_(C=C, dtype=dtype, X=21, Y=19)
    check(fb, synth.make_workload(wl), device, what=f"C={C} {dtype}", method=method)


@pytest.mark.parametrize("X,Y", [(1, 1), (3, 50), (50, 3), (37, 41)])
@pytest.mark.parametrize("method", METHODS)
def test_backward_grid_shapes(fb, device, X, Y, method):
    wl = synth.config("tiny").with_(X=X, Y=Y)
    check(fb, synth.make_workload(wl), device, what=f"grid {X}x{Y}", method=method)


@pytest.mark.parametrize("method", METHODS)
def test_backward_overwrites_prefilled_gradient(fb, device, method):
    inst = synth.make_workload(synth.config("tiny"))
    check(fb, inst, device, what="prefilled NaN", prefill=float("nan"), method=method)


@pytest.mark.parametrize("method", METHODS)
def test_backward_degenerate_inputs(fb, device, method):
    import torch
    # no heights: the gradient is all zeros (the fill still runs)
    wl = synth.config("tiny").with_(Z=0)
    inst = synth.make_workload(wl)
    gpu = gpu_backward(fb, inst, _grad_out(wl), device, prefill=7.0, method=method)
    assert np.all(gpu == 0.0)
    # an empty grid: likewise
    wl = synth.config("tiny").with_(X=0)
    inst = synth.make_workload(wl)
    gpu = gpu_backward(fb, inst, _grad_out(wl), device, prefill=7.0, method=method)
    assert np.all(gpu == 0.0)
    # a 1x1 feature map (both tap steps are zero)
    wl = synth.config("tiny").with_(H=1, W=1)
    check(fb, synth.make_workload(wl), device, what="1x1 map", method=method)
    # an empty batch enqueues nothing
    wl = synth.config("tiny").with_(B=0)
    inst = synth.make_workload(wl)
    l2i = torch.zeros((0, wl.N, 4, 4), device=device)
    gt = torch.zeros((0, wl.C, wl.X, wl.Y), device=device)
    out = fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                (0, wl.N, wl.H, wl.W, wl.C), method=method)
    assert out.shape[0] == 0


def test_backward_unaligned_gradient_buffer(fb, device):
    import torch
    inst = synth.make_workload(synth.config("tiny").with_(X=23, Y=17))
    wl = inst.wl
    g = _grad_out(wl)
    n = int(np.prod(inst.features.shape))
    buf = torch.full((n + 1,), 3.0, dtype=torch.float32, device=device)
    view = buf[1:].view(inst.features.shape)           # 4-byte but not 16-byte aligned
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(g).to(device)
    rc = fb.sample_vt_backward_raw(inst.features.shape, wl.dtype, l2i.data_ptr(), inst.z,
                                   fb.grid_of(wl), (wl.img_h, wl.img_w), gt.data_ptr(),
                                   view.data_ptr())
    torch.cuda.synchronize()
    assert rc == 0
    ref, scale, terms = oracle_backward(inst, g)
    assert_bwd_parity(view.cpu().numpy(), ref, scale, terms, "scatter unaligned")
    assert buf[0].item() == 3.0
    # the gather form on the same unaligned gradient buffer
    need = fb.backward_workspace_size(inst.features.shape, wl.dtype, inst.z, fb.grid_of(wl),
                                      (wl.img_h, wl.img_w))
    ws = torch.empty(need, dtype=torch.uint8, device=device)
    buf.fill_(3.0)
    rc = fb.sample_vt_backward_ws_raw(inst.features.shape, wl.dtype, l2i.data_ptr(), inst.z,
                                      fb.grid_of(wl), (wl.img_h, wl.img_w), gt.data_ptr(),
                                      view.data_ptr(), ws.data_ptr(), need)
    torch.cuda.synchronize()
    assert rc == 0
    assert_bwd_parity(view.cpu().numpy(), ref, scale, terms, "gather unaligned")
    assert buf[0].item() == 3.0


@pytest.mark.parametrize("method", METHODS)
def test_backward_adjoint_of_gpu_forward(fb, device, method):
    """<fwd(F), G> = <F, bwd(G)> with both sides computed on the GPU."""
    import torch
    for name in ("rep", "half_batch"):
        wl = synth.config(name)
        inst = synth.make_workload(wl)
        ft = synth.to_storage(inst.features, wl.dtype).to(device)
        l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
        g = _grad_out(wl)
        out = fb.sample_vt(ft, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w))
        gf = fb.sample_vt_backward(torch.from_numpy(g).to(device), l2i, inst.z, fb.grid_of(wl),
                                   (wl.img_h, wl.img_w), inst.features.shape, wl.dtype,
                                   method=method)
        torch.cuda.synchronize()
        lhs = float(np.sum(out.cpu().numpy().astype(np.float64) * g))
        rhs = float(np.sum(inst.features.astype(np.float64) * gf.cpu().numpy()))
        _, oscale, _ = oracle.run_instance(inst)
        bound = float(np.sum(oscale * np.abs(g)))
        print(f"[adjoint] {method} {name} lhs={lhs:.6e} rhs={rhs:.6e} bound={bound:.3e}", flush=True)
        assert abs(lhs - rhs) <= 1e-5 * bound


@pytest.mark.parametrize("method", METHODS)
def test_backward_on_side_stream(fb, device, method):
    import torch
    inst = synth.make_workload(synth.config("tiny"))
    wl = inst.wl
    g = _grad_out(wl)
    s = torch.cuda.Stream(device)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(g).to(device)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        gf = fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                   inst.features.shape, stream=s, method=method)
    s.synchronize()
    ref, scale, terms = oracle_backward(inst, g)
    assert_bwd_parity(gf.cpu().numpy(), ref, scale, terms, f"{method} side stream")


def test_backward_allocates_nothing_beyond_its_output(fb, device):
    import torch
    wl = synth.config("rep")
    inst = synth.make_workload(wl)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(_grad_out(wl)).to(device)
    gf = torch.empty(inst.features.shape, dtype=torch.float32, device=device)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats(device)
    base = torch.cuda.memory_allocated(device)
    fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                          inst.features.shape, grad_features=gf, method="scatter")
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated(device) == base
    # the gather form with the caller's workspace
    need = fb.backward_workspace_size(inst.features.shape, wl.dtype, inst.z, fb.grid_of(wl),
                                      (wl.img_h, wl.img_w))
    ws = torch.empty(need, dtype=torch.uint8, device=device)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats(device)
    base = torch.cuda.memory_allocated(device)
    fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                          inst.features.shape, grad_features=gf, method="gather", workspace=ws)
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated(device) == base


@pytest.mark.parametrize("method", METHODS)
def test_prepared_backward_matches_plain_call(fb, device, method):
    import torch
    inst = synth.make_workload(synth.config("tiny"))
    wl = inst.wl
    g = _grad_out(wl)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(g).to(device)
    gf = torch.full(inst.features.shape, float("nan"), dtype=torch.float32, device=device)
    call = fb.prepare_sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                         inst.features.shape, wl.dtype, gf, method=method)
    call()
    call()
    torch.cuda.synchronize()
    ref, scale, terms = oracle_backward(inst, g)
    assert_bwd_parity(gf.cpu().numpy(), ref, scale, terms, f"{method} prepared")


def test_gather_backward_rejects_small_workspace(fb, device):
    import torch
    inst = synth.make_workload(synth.config("tiny"))
    wl = inst.wl
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(_grad_out(wl)).to(device)
    need = fb.backward_workspace_size(inst.features.shape, wl.dtype, inst.z, fb.grid_of(wl),
                                      (wl.img_h, wl.img_w))
    ws = torch.empty(need - 256, dtype=torch.uint8, device=device)
    with pytest.raises(ValueError):
        fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                              inst.features.shape, workspace=ws)


def test_gather_and_scatter_forms_agree(fb, device):
    """Both forms on the same inputs, against each other: each is within
    the bar of the oracle, so they differ by at most twice the bar."""
    for name in ("rep", "half_batch", "long_range"):
        wl = synth.config(name)
        inst = synth.make_workload(wl)
        g = _grad_out(wl)
        a = gpu_backward(fb, inst, g, device, method="gather").astype(np.float64)
        b = gpu_backward(fb, inst, g, device, method="scatter").astype(np.float64)
        _, scale, terms = oracle_backward(inst, g)
        tol = 2.0 * (terms[..., None] + 8.0) * U * scale
        print(f"[gather-vs-scatter] {name} max_abs={np.abs(a - b).max():.3e}", flush=True)
        assert np.all(np.abs(a - b) <= tol)
        # what no term reaches is zero in both
        assert np.all(a[scale == 0] == 0.0) and np.all(b[scale == 0] == 0.0)


@pytest.mark.parametrize("seed", range(8))
def test_backward_arbitrary_camera_matrices(fb, device, seed):
    """Cameras in any orientation and place, heights in any order over
    +-30 m, feature strides 4 to 16: the gather form's candidate regions
    must hold every sample that reaches a pixel (both forms against the
    oracle)."""
    from test_cull_soundness import random_matrices
    rng = np.random.default_rng([8400, seed])
    C, dtype = [(16, "f32"), (80, "f32"), (64, "bf16"), (8, "f16")][seed % 4]
    img_h, img_w = (256, 704) if seed % 2 else (900, 1600)
    stride = (4, 8, 16)[seed % 3]
    B, N, Z = int(rng.integers(1, 3)), int(rng.integers(1, 9)), int(rng.integers(1, 24))
    half = float(rng.uniform(5.0, 60.0))
    X, Y = int(rng.integers(8, 90)), int(rng.integers(8, 90))
    wl = synth.Workload(name="arbitrary", cfg_id=8400 + seed, B=B, N=N, img_h=img_h,
                        img_w=img_w, H=img_h // stride, W=img_w // stride, C=C, dtype=dtype,
                        X=X, Y=Y, x_min=-half, dx=2 * half / X, y_min=-half, dy=2 * half / Y,
                        z_lo=-5.0, z_hi=3.0, Z=Z)
    inst = synth.make_workload(wl)
    inst.lidar2img = np.stack([random_matrices(rng, N, img_h, img_w) for _ in range(B)])
    inst.z = rng.uniform(-30.0, 30.0, Z).astype(np.float32)
    for method in METHODS:
        check(fb, inst, device, what=f"arbitrary cameras {seed}", method=method)


def test_backward_degenerate_and_extreme_cameras(fb, device):
    """Zero rows, a camera looking straight down, one at the grid's height,
    one with entries near float32 overflow, one with a NaN entry and one
    whose u and v rows are scaled to 1e-36 (its samples are valid and land
    on pixel (0, 0); the gather form gives it no region and scans every
    cell)."""
    wl = synth.config("tiny").with_(N=6, X=60, Y=60, C=16, Z=4)
    inst = synth.make_workload(wl)
    m = np.zeros((6, 4, 4), np.float32)
    m[0, 1] = [0, 500, 0, 128]
    m[0, 2] = [1, 0, 0, 0]
    m[1, 0] = [500, 0, 352, 0]
    m[1, 1] = [0, 500, 128, 0]
    m[1, 2] = [0, 0, -1, 10]
    m[2, :3] = np.array([[352, -500, 0, 0], [128, 0, -500, 0], [1, 0, 0, 0]], np.float32)
    m[3, :3] = np.array([[3e37, 1, 0, 0], [0, 2e37, 0, 0], [1, 0, 0, 5]], np.float32)
    m[4, :3] = np.array([[352, -500, 0, 0], [128, 0, -500, np.nan], [1, 0, 0, 0]], np.float32)
    m[5] = m[2]
    m[5, :2] *= np.float32(1e-36)
    m[:, 3, 3] = 1
    inst.lidar2img = m[None]
    inst.z = np.array([-5.0, -1.0, 0.0, 2.0], np.float32)
    for method in METHODS:
        check(fb, inst, device, what="extreme cameras", method=method)
