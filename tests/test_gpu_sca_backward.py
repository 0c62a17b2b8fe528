"""GPU parity of the FlashSCA backward against the CPU oracle.

Bars, per element, with u = 2^-24 and the oracle's magnitude scales S (sums
of |terms|):
  * value gradient: |gpu - oracle| <= (K + 16) u S, K = terms reaching the
    pixel's head slice.  Each term alpha a w G carries a few roundings and
    float32 atomic addition of K terms in any order at most K - 1 roundings
    of partial sums no larger than S.
  * offsets gradient: (T D + 32) u S, T = in-range corners of the point over
    the hit cameras, D channels per head: the dot products of tap rows with
    the output gradient (T D products, summed over lanes and then over the
    slot), the bilinear derivative's few roundings and the sum over cameras.
  * logits gradient: (sum_j T_j D + L P + 32) u S over the head's points: the
    softmax backward subtracts the attention-weighted sum of every point's
    d a_j.
Elements the oracle gives no term must be exactly zero.  All calls go
through the C ABI via the thin binding.
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


def _g(wl, seed=5):
    return np.random.default_rng([wl.cfg_id, 9, seed]).standard_normal(
        (wl.B, wl.Q, wl.C)).astype(np.float32)


def _dev(inst, device):
    import torch
    wl = inst.wl
    v = synth.to_storage(inst.value, wl.dtype).to(device)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    off = torch.from_numpy(np.ascontiguousarray(inst.offsets)).to(device)
    lg = torch.from_numpy(np.ascontiguousarray(inst.logits)).to(device)
    return v, l2i, off, lg


def gpu_bwd(fb, inst, g, device, reduce="mean", want=("value", "offsets", "logits"),
            prefill=None):
    import torch
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    kw = {}
    if prefill is not None:
        kw = dict(grad_value=torch.full((wl.B, wl.N, wl.S, wl.C), prefill, device=device),
                  grad_offsets=torch.full(tuple(off.shape), prefill, device=device),
                  grad_logits=torch.full(tuple(lg.shape), prefill, device=device))
    r = fb.sca_backward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels,
                        wl.heads, off, lg, torch.from_numpy(g).to(device), want=want,
                        reduce=reduce, **kw)
    torch.cuda.synchronize()
    return {k: (t.cpu().numpy() if t is not None else None) for k, t in r.items()}


def _check(name, gpu, ref, scale, K, what):
    err = np.abs(gpu.astype(np.float64) - ref)
    tol = (K + 0.0) * U * scale
    nz = scale > 0
    worst = float((err[nz] / scale[nz]).max(initial=0.0))
    print(f"[parity-sca-bwd] {what} {name} max_abs={err.max(initial=0):.3e} "
          f"max_scaled={worst:.3e}", flush=True)
    bad = err > tol
    assert not bad.any(), f"{what} {name}: {bad.sum()} of {bad.size} off (max scaled {worst:.3e})"
    assert np.all(gpu[~nz] == 0.0), f"{what} {name}: elements with no term are not zero"


def assert_bwd_parity(gpu, ref, wl, what=""):
    D = wl.C // wl.heads
    if gpu.get("value") is not None:
        K = np.repeat(ref["value_terms"], D, axis=-1).astype(np.float64) + 16.0
        _check("value", gpu["value"], ref["value"], ref["value_scale"], K, what)
    T = ref["point_terms"].astype(np.float64)
    if gpu.get("offsets") is not None:
        K = (T * D + 32.0)[..., None]
        _check("offsets", gpu["offsets"], ref["offsets"], ref["offsets_scale"], K, what)
    if gpu.get("logits") is not None:
        Th = T.reshape(T.shape[:3] + (-1,)).sum(axis=-1) * D + wl.L * wl.P + 32.0
        K = np.broadcast_to(Th[..., None, None], T.shape)
        _check("logits", gpu["logits"], ref["logits"], ref["logits_scale"], K, what)


def check(fb, inst, device, reduce="mean", what="", want=("value", "offsets", "logits"),
          prefill=None):
    wl = inst.wl
    print(f"[case] sca backward {what} value={inst.value.shape} {wl.dtype} heads={wl.heads} "
          f"P={wl.P} Z={wl.Z} X={wl.X} Y={wl.Y} reduce={reduce} want={want}", flush=True)
    g = _g(wl)
    gpu = gpu_bwd(fb, inst, g, device, reduce, want, prefill)
    ref = oracle.sca_backward_instance(inst, g, reduce)
    for k in ("value", "offsets", "logits"):
        if k not in want:
            assert gpu[k] is None
    assert_bwd_parity(gpu, ref, wl, what)
    return gpu, ref


def small(seed=0, **kw):
    base = dict(name="small", cfg_id=400 + seed, B=2, N=6, img_h=256, img_w=704,
                levels=((20, 44), (10, 22), (5, 11)), C=32, heads=4, P=4, Z=2, dtype="f32",
                X=13, Y=11, x_min=-26.0, dx=4.0, y_min=-22.0, dy=4.0)
    base.update(kw)
    return synth.make_sca_workload(synth.ScaWorkload(**base))


def test_sca_backward_tiny(fb, device):
    check(fb, synth.make_sca_workload(synth.sca_config("sca_tiny")), device, what="sca_tiny")


@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_sca_backward_reduce_modes(fb, device, reduce):
    check(fb, small(1), device, reduce, what=f"small {reduce}")


@pytest.mark.parametrize("C,heads,dtype", [
    (32, 4, "f32"), (256, 8, "f32"), (256, 8, "bf16"), (128, 8, "f16"), (512, 8, "f32"),
    (256, 1, "f32"), (12, 4, "f32"), (10, 2, "bf16"), (48, 3, "f16")])
def test_sca_backward_channel_and_head_shapes(fb, device, C, heads, dtype):
    check(fb, small(2, C=C, heads=heads, dtype=dtype, X=9, Y=7), device,
          what=f"C={C} heads={heads} {dtype}")


@pytest.mark.parametrize("C,heads,dtype", [(256, 8, "f32"), (512, 16, "f32"), (256, 8, "bf16")])
def test_sca_backward_head_to_xcd_order(fb, device, C, heads, dtype):
    # heads a multiple of 8 and more than 32 points per head: tiles follow the
    # head-to-XCD order (two head groups at 16 heads, both batch elements)
    check(fb, small(5, C=C, heads=heads, dtype=dtype, P=16, Z=4, X=23, Y=19), device,
          what=f"head order C={C} heads={heads} {dtype} P=16")


@pytest.mark.parametrize("C,heads,P", [(256, 8, 8), (256, 8, 16), (32, 4, 16)])
def test_sca_backward_azimuth_block_order(fb, device, C, heads, P):
    # a 32 x 48 grid of six whole 16 x 16 blocks: rank order at P = 8 (24
    # points per head), the azimuth order of the blocks at P = 16 (with the
    # head order at 8 heads, the band order at 4)
    check(fb, small(6, C=C, heads=heads, P=P, Z=4, X=32, Y=48, x_min=-30.0, dx=2.0, y_min=-45.0,
                    dy=2.0), device, what=f"azimuth order C={C} heads={heads} P={P}", prefill=np.nan)


@pytest.mark.parametrize("P,Z,L", [(1, 1, 1), (3, 1, 2), (8, 4, 4), (32, 4, 4), (64, 8, 8)])
def test_sca_backward_points_anchors_levels(fb, device, P, Z, L):
    levels = ((24, 64), (12, 32), (6, 16), (3, 8), (2, 4), (1, 2), (1, 1), (5, 3))[:L]
    check(fb, small(3, P=P, Z=Z, levels=levels, X=7, Y=9), device, what=f"P={P} Z={Z} L={L}")


@pytest.mark.parametrize("want", [("value",), ("offsets", "logits"), ("logits",)])
def test_sca_backward_partial_outputs(fb, device, want):
    check(fb, small(4), device, what=f"want={want}", want=want)


def test_sca_backward_overwrites_prefilled_outputs(fb, device):
    check(fb, small(5), device, what="prefilled NaN", prefill=float("nan"))


def test_sca_backward_degenerate_inputs(fb, device):
    inst = small(6)
    inst.offsets[:, : inst.wl.Q // 2] = 1e9
    inst.offsets[:, inst.wl.Q // 2:, :, :, ::2] = np.nan
    check(fb, inst, device, what="far and NaN offsets")
    check(fb, small(7, levels=((1, 1), (1, 1))), device, what="1x1 maps")
    # no cameras: all gradients zero
    inst = small(8, N=0)
    gpu = gpu_bwd(fb, inst, _g(inst.wl), device, prefill=3.0)
    assert gpu["value"].size == 0
    assert np.all(gpu["offsets"] == 0.0) and np.all(gpu["logits"] == 0.0)


@pytest.mark.parametrize("case", ["spread", "crowded"])
def test_sca_backward_row_merge_extremes(fb, device, case):
    """The value gradient's row merge at its extremes.  `spread`: offsets
    uniform over a 116 x 200 map, so nearly every in-range (point, slot, tap)
    row of a tile's chunk is a distinct pixel: about as many keys as rows in
    the table, with long probe runs.  `crowded`: one 4 x 4 map, so the rows of 32 queries x 8
    points x 4 taps pile onto 16 pixels per head and the member lists run
    long."""
    if case == "spread":
        inst = small(10, levels=((116, 200),), C=256, heads=8, P=8, Z=4, X=16, Y=16)
        rng = np.random.default_rng(10)
        inst.offsets[...] = rng.uniform(-150.0, 150.0, inst.offsets.shape).astype(np.float32)
    else:
        inst = small(11, levels=((4, 4),), C=256, heads=8, P=8, Z=4, X=16, Y=16)
    check(fb, inst, device, what=f"row merge {case}")


@pytest.mark.parametrize("name,P", [("sca_base", 8), ("sca_base", 16), ("sca_base", 32),
                                    ("sca_base_bf16", 8)])
def test_sca_backward_bevformer_base(fb, device, name, P):
    """Table 7's setting at every P the bench times (the row merge's keys and
    member lists grow with P), and the bfloat16 batch of two; every element
    of all three gradients checked against the oracle."""
    wl = synth.sca_config(name).with_(P=P)
    print(f"[case] {name} P={P} B={wl.B} dtype={wl.dtype}", flush=True)
    inst = synth.make_sca_workload(wl)
    check(fb, inst, device, what=f"{name} P={P}")


def test_sca_backward_adjoint_of_gpu_forward(fb, device):
    """<fwd(V), G> = <V, d value(G)>, both computed on the GPU."""
    import torch
    for name in ("sca_base", "sca_base_bf16"):
        wl = synth.sca_config(name)
        inst = synth.make_sca_workload(wl)
        v, l2i, off, lg = _dev(inst, device)
        g = _g(wl)
        out = fb.sca_forward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels,
                             wl.heads, off, lg)
        r = fb.sca_backward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels,
                            wl.heads, off, lg, torch.from_numpy(g).to(device), want=("value",))
        torch.cuda.synchronize()
        lhs = float(np.sum(out.cpu().numpy().astype(np.float64) * g))
        rhs = float(np.sum(inst.value.astype(np.float64) * r["value"].cpu().numpy()))
        _, oscale, _, _ = oracle.sca_instance(inst)
        bound = float(np.sum(oscale * np.abs(g)))
        print(f"[adjoint-sca] {name} lhs={lhs:.6e} rhs={rhs:.6e} bound={bound:.3e}", flush=True)
        assert abs(lhs - rhs) <= 1e-5 * bound


def test_sca_backward_on_side_stream(fb, device):
    import torch
    inst = small(9)
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    g = _g(wl)
    gt = torch.from_numpy(g).to(device)
    s = torch.cuda.Stream(device)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        r = fb.sca_backward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels,
                            wl.heads, off, lg, gt, stream=s)
    s.synchronize()
    gpu = {k: t.cpu().numpy() for k, t in r.items()}
    assert_bwd_parity(gpu, oracle.sca_backward_instance(inst, g), wl, "side stream")


def test_sca_backward_allocates_nothing_beyond_its_outputs(fb, device):
    import torch
    inst = small(10)
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    gt = torch.from_numpy(_g(wl)).to(device)
    gv = torch.empty((wl.B, wl.N, wl.S, wl.C), device=device)
    go = torch.empty(tuple(off.shape), device=device)
    gl = torch.empty(tuple(lg.shape), device=device)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats(device)
    base = torch.cuda.memory_allocated(device)
    fb.sca_backward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels, wl.heads,
                    off, lg, gt, grad_value=gv, grad_offsets=go, grad_logits=gl)
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated(device) == base


def test_prepared_sca_backward_matches_oracle(fb, device):
    import torch
    inst = small(11)
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    g = _g(wl)
    gt = torch.from_numpy(g).to(device)
    gv = torch.full((wl.B, wl.N, wl.S, wl.C), float("nan"), device=device)
    go = torch.full(tuple(off.shape), float("nan"), device=device)
    gl = torch.full(tuple(lg.shape), float("nan"), device=device)
    call = fb.prepare_sca_backward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                   wl.levels, wl.heads, off, lg, gt, gv, go, gl)
    call()
    call()
    torch.cuda.synchronize()
    gpu = {"value": gv.cpu().numpy(), "offsets": go.cpu().numpy(), "logits": gl.cpu().numpy()}
    assert_bwd_parity(gpu, oracle.sca_backward_instance(inst, g), wl, "prepared")


@pytest.mark.parametrize("what,kw", [
    ("32 cameras", dict(N=32, X=6, Y=5)),
    ("32 anchors", dict(Z=32, P=32, levels=((12, 32),), X=6, Y=5)),
    ("L*P = 512", dict(P=64, Z=8, levels=((24, 64), (12, 32), (6, 16), (3, 8), (2, 4), (1, 2),
                                         (1, 1), (5, 3)), X=4, Y=3)),
    ("1 KiB head rows", dict(C=256, heads=1, X=6, Y=5)),
    ("512-element bf16 heads", dict(C=1024, heads=2, dtype="bf16", X=5, Y=4)),
])
def test_sca_backward_limits(fb, device, what, kw):
    check(fb, small(12, **kw), device, what=what)
