"""GPU parity of the backward (gradient w.r.t. the feature maps) against the oracle.

Bar (per gradient element): |gpu - oracle| <= (K + 8) * 2^-24 * S, where S
is the oracle's sum of |terms| for that element and K the number of terms
reaching its pixel.  Derivation: each float32 term w * g carries at most
about seven roundings (the bilinear fractions, the weight products, the
approximate reciprocal of den_z, the product with g), and float32 atomic
addition of K terms in any order adds at most (K - 1) roundings of partial
sums no larger than S.  Elements no term reaches must be exactly zero.
All calls go through the C ABI via the thin binding.

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


@pytest.fixture(scope="module")
def fb():
    import paper_2607_10071_amd as m
    return m


def _grad_out(wl, seed=3):
    rng = np.random.default_rng([wl.cfg_id, 7, seed])
    return rng.standard_normal((wl.B, wl.C, wl.X, wl.Y)).astype(np.float32)


def gpu_backward(fb, inst, g, device, reduce="mean", prefill=None):
    import torch
    wl = inst.wl
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(g).to(device)
    gf = None
    if prefill is not None:
        gf = torch.full(inst.features.shape, prefill, dtype=torch.float32, device=device)
    gf = fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                               inst.features.shape, wl.dtype, grad_features=gf, reduce=reduce)
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


def check(fb, inst, device, reduce="mean", what="", prefill=None):
    print(f"[case] backward {what} shape={inst.features.shape} X={inst.wl.X} Y={inst.wl.Y} "
          f"Z={len(inst.z)} reduce={reduce}", flush=True)
    g = _grad_out(inst.wl)
    gpu = gpu_backward(fb, inst, g, device, reduce, prefill)
    ref, scale, terms = oracle.backward_instance(inst, g, reduce)
    assert gpu.shape == ref.shape
    assert_bwd_parity(gpu, ref, scale, terms, what)
    return gpu, ref, terms


@pytest.mark.parametrize("wl", synth.all_parity_workloads(), ids=lambda w: f"{w.name}-Z{w.Z}")
def test_backward_workloads_full(fb, device, wl):
    inst = synth.make_workload(wl)
    _, _, terms = check(fb, inst, device, what=f"{wl.name} Z={wl.Z}")
    assert terms.sum() > 0


@pytest.mark.parametrize("C", [128, 256])
def test_backward_paper_reference_setting(fb, device, C):
    """The paper's reference setting in full; C = 256 takes the tiled mode's
    wide-row path (channel blocks beyond two per lane)."""
    inst = synth.make_workload(synth.config("paper_ref", C=C))
    check(fb, inst, device, what=f"paper_ref C={C}")


@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_backward_reduce_modes(fb, device, reduce):
    inst = synth.make_workload(synth.config("tiny"))
    check(fb, inst, device, reduce, what=f"tiny {reduce}")


@pytest.mark.parametrize("C,dtype", [(1, "f32"), (5, "f32"), (7, "bf16"), (36, "f16"),
                                     (128, "f32"), (129, "f32"), (192, "f32"), (256, "bf16"),
                                     (260, "f32"), (512, "f32"), (512, "f16"),
                                     (1024, "f32"), (2048, "bf16")])
def test_backward_channel_counts(fb, device, C, dtype):
    wl = synth.config("tiny").with_(C=C, dtype=dtype, X=21, Y=19)
    check(fb, synth.make_workload(wl), device, what=f"C={C} {dtype}")


@pytest.mark.parametrize("X,Y", [(1, 1), (3, 50), (50, 3), (37, 41)])
def test_backward_grid_shapes(fb, device, X, Y):
    wl = synth.config("tiny").with_(X=X, Y=Y)
    check(fb, synth.make_workload(wl), device, what=f"grid {X}x{Y}")


def test_backward_overwrites_prefilled_gradient(fb, device):
    inst = synth.make_workload(synth.config("tiny"))
    check(fb, inst, device, what="prefilled NaN", prefill=float("nan"))


def test_backward_degenerate_inputs(fb, device):
    import torch
    # no heights: the gradient is all zeros (the fill still runs)
    wl = synth.config("tiny").with_(Z=0)
    inst = synth.make_workload(wl)
    gpu = gpu_backward(fb, inst, _grad_out(wl), device, prefill=7.0)
    assert np.all(gpu == 0.0)
    # a 1x1 feature map (both tap steps are zero)
    wl = synth.config("tiny").with_(H=1, W=1)
    check(fb, synth.make_workload(wl), device, what="1x1 map")
    # an empty batch enqueues nothing
    wl = synth.config("tiny").with_(B=0)
    inst = synth.make_workload(wl)
    l2i = torch.zeros((0, wl.N, 4, 4), device=device)
    gt = torch.zeros((0, wl.C, wl.X, wl.Y), device=device)
    out = fb.sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                (0, wl.N, wl.H, wl.W, wl.C))
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
    rc = fb.sample_vt_backward_raw(inst.features.shape, wl.dtype, l2i.data_ptr(), inst.z,
                                   fb.grid_of(wl), (wl.img_h, wl.img_w),
                                   torch.from_numpy(g).to(device).data_ptr(), view.data_ptr())
    torch.cuda.synchronize()
    assert rc == 0
    ref, scale, terms = oracle.backward_instance(inst, g)
    assert_bwd_parity(view.cpu().numpy(), ref, scale, terms, "unaligned")
    assert buf[0].item() == 3.0


def test_backward_adjoint_of_gpu_forward(fb, device):
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
                                   (wl.img_h, wl.img_w), inst.features.shape, wl.dtype)
        torch.cuda.synchronize()
        lhs = float(np.sum(out.cpu().numpy().astype(np.float64) * g))
        rhs = float(np.sum(inst.features.astype(np.float64) * gf.cpu().numpy()))
        _, oscale, _ = oracle.run_instance(inst)
        bound = float(np.sum(oscale * np.abs(g)))
        print(f"[adjoint] {name} lhs={lhs:.6e} rhs={rhs:.6e} bound={bound:.3e}", flush=True)
        assert abs(lhs - rhs) <= 1e-5 * bound


def test_backward_on_side_stream(fb, device):
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
                                   inst.features.shape, stream=s)
    s.synchronize()
    ref, scale, terms = oracle.backward_instance(inst, g)
    assert_bwd_parity(gf.cpu().numpy(), ref, scale, terms, "side stream")


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
                          inst.features.shape, grad_features=gf)
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated(device) == base


def test_prepared_backward_matches_plain_call(fb, device):
    import torch
    inst = synth.make_workload(synth.config("tiny"))
    wl = inst.wl
    g = _grad_out(wl)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    gt = torch.from_numpy(g).to(device)
    gf = torch.full(inst.features.shape, float("nan"), dtype=torch.float32, device=device)
    call = fb.prepare_sample_vt_backward(gt, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                         inst.features.shape, wl.dtype, gf)
    call()
    call()
    torch.cuda.synchronize()
    ref, scale, terms = oracle.backward_instance(inst, g)
    assert_bwd_parity(gf.cpu().numpy(), ref, scale, terms, "prepared")
