"""GPU parity of the FlashSCA forward against the CPU oracle.

Bar (per output element): |gpu - oracle| <= (K + 16) * 2^-24 * S, where S
is the oracle's sum of |terms| for that element and K the number of in-range
taps summed into it (all hit cameras, levels and points of its head).  Each
float32 term a * w * v carries a few roundings (the softmax weight, about
four; the bilinear weight products, three; the product with the value, one),
and float32 accumulation of K terms adds at most K - 1 roundings of partial
sums no larger than S.  Elements no tap reaches must be exactly zero.  Hit
decisions and taps are integer outcomes taken in float32 by both sides with
the same recipe, so any disagreement there fails the bar.  All calls go
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


def _dev(inst, device):
    import torch
    wl = inst.wl
    v = synth.to_storage(inst.value, wl.dtype).to(device)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    off = torch.from_numpy(np.ascontiguousarray(inst.offsets)).to(device)
    lg = torch.from_numpy(np.ascontiguousarray(inst.logits)).to(device)
    return v, l2i, off, lg


def gpu_sca(fb, inst, device, reduce="mean", prefill=None):
    import torch
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    out = None
    if prefill is not None:
        out = torch.full((wl.B, wl.Q, wl.C), prefill, dtype=torch.float32, device=device)
    out = fb.sca_forward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels,
                         wl.heads, off, lg, out=out, reduce=reduce)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def assert_sca_parity(gpu, ref, scale, terms, heads, what=""):
    B, Q, C = ref.shape
    D = C // heads
    K = np.repeat(terms, D, axis=-1).astype(np.float64)           # [B, Q, C]
    err = np.abs(gpu.astype(np.float64) - ref)
    tol = (K + 16.0) * U * scale
    bad = err > tol
    nz = scale > 0
    worst = float((err[nz] / scale[nz]).max(initial=0.0))
    print(f"[parity-sca] {what} max_abs={err.max(initial=0):.3e} max_scaled={worst:.3e} "
          f"max_terms={int(terms.max(initial=0))}", flush=True)
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} elements off (max scaled {worst:.3e})"
    assert np.all(gpu[~nz] == 0.0), f"{what}: elements no tap reaches are not zero"


def check(fb, inst, device, reduce="mean", what="", prefill=None):
    wl = inst.wl
    print(f"[case] sca {what} value={inst.value.shape} {wl.dtype} heads={wl.heads} P={wl.P} "
          f"Z={wl.Z} X={wl.X} Y={wl.Y} reduce={reduce}", flush=True)
    gpu = gpu_sca(fb, inst, device, reduce, prefill)
    ref, scale, terms, cnt = oracle.sca_instance(inst, reduce)
    assert gpu.shape == ref.shape
    assert_sca_parity(gpu, ref, scale, terms, wl.heads, what)
    return gpu, ref, cnt


def small(seed=0, **kw):
    base = dict(name="small", cfg_id=300 + seed, B=2, N=6, img_h=256, img_w=704,
                levels=((20, 44), (10, 22), (5, 11)), C=32, heads=4, P=4, Z=2, dtype="f32",
                X=13, Y=11, x_min=-26.0, dx=4.0, y_min=-22.0, dy=4.0)
    base.update(kw)
    return synth.make_sca_workload(synth.ScaWorkload(**base))


def test_sca_tiny(fb, device):
    inst = synth.make_sca_workload(synth.sca_config("sca_tiny"))
    _, _, cnt = check(fb, inst, device, what="sca_tiny")
    assert cnt["hits"] > 100


@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_sca_reduce_modes(fb, device, reduce):
    check(fb, small(1), device, reduce, what=f"small {reduce}")


@pytest.mark.parametrize("C,heads,dtype", [
    (32, 4, "f32"),      # D=8: 4-byte lanes
    (256, 8, "f32"),     # D=32: 16-byte lanes (BEVFormer)
    (256, 8, "bf16"),    # D=32: 16-byte lanes, two queries per wavefront
    (128, 8, "f16"),     # D=16
    (512, 8, "f32"),     # D=64: 16 lanes per head
    (256, 1, "f32"),     # D=256: one head fills a wavefront
    (12, 4, "f32"),      # D=3: padded lanes
    (10, 2, "bf16"),     # D=5: 2-byte lanes
    (48, 3, "f16"),      # D=16, three heads
    (512, 16, "f32"),    # D=32, two head groups in the head-to-XCD order
])
def test_sca_channel_and_head_shapes(fb, device, C, heads, dtype):
    inst = small(2, C=C, heads=heads, dtype=dtype, X=9, Y=7)
    check(fb, inst, device, what=f"C={C} heads={heads} {dtype}")


@pytest.mark.parametrize("C,heads,dtype", [(256, 8, "f32"), (256, 8, "bf16"), (32, 4, "f32")])
def test_sca_azimuth_block_order(fb, device, C, heads, dtype):
    # a 32 x 48 grid of six whole 16 x 16 blocks and 144 points per head: the
    # query groups are visited in the azimuth order of the blocks (with the
    # head order at 8 heads, the band order at 4); every output element is
    # overwritten
    inst = small(6, C=C, heads=heads, dtype=dtype, X=32, Y=48, P=48, Z=4, x_min=-30.0, dx=2.0,
                 y_min=-45.0, dy=2.0)
    check(fb, inst, device, what=f"azimuth order C={C} heads={heads} {dtype}", prefill=np.nan)


@pytest.mark.parametrize("P", [8, 32])
def test_sca_launch_order_leaves_outputs_bitwise(fb, device, P):
    # BEVFormer-base (heads to XCDs; at P = 32 also the azimuth order of the
    # blocks) at B = 1 and the same batch element twice: the tile orders
    # decide only when a query is computed, so both copies equal the single
    # call bit for bit, and so do the backward's offset and logit gradients
    # (no atomics there)
    import torch
    inst = synth.make_sca_workload(synth.sca_config("sca_base", P=P))
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    grid, img = fb.grid_of(wl), (wl.img_h, wl.img_w)
    two = [t[:1].repeat(2, *([1] * (t.dim() - 1))).contiguous() for t in (v, l2i, off, lg)]
    one = fb.sca_forward(v, l2i, inst.z, grid, img, wl.levels, wl.heads, off, lg)
    dup = fb.sca_forward(*two[:2], inst.z, grid, img, wl.levels, wl.heads, *two[2:])
    g = torch.from_numpy(np.random.default_rng(P).standard_normal(
        (1, wl.Q, wl.C)).astype(np.float32)).to(device)
    want = ("offsets", "logits")
    b1 = fb.sca_backward(v, l2i, inst.z, grid, img, wl.levels, wl.heads, off, lg, g, want=want)
    b2 = fb.sca_backward(*two[:2], inst.z, grid, img, wl.levels, wl.heads, *two[2:],
                         g.repeat(2, 1, 1).contiguous(), want=want)
    torch.cuda.synchronize()
    for b in range(2):
        assert torch.equal(dup[b], one[0]), f"P={P}: forward copy {b} differs"
        for k in want:
            assert torch.equal(b2[k][b], b1[k][0]), f"P={P}: {k} gradient copy {b} differs"


@pytest.mark.parametrize("P,Z,L", [(1, 1, 1), (3, 1, 2), (8, 4, 4), (16, 4, 4), (32, 4, 4),
                                   (6, 3, 3), (64, 8, 8)])
def test_sca_points_anchors_levels(fb, device, P, Z, L):
    levels = ((24, 64), (12, 32), (6, 16), (3, 8), (2, 4), (1, 2), (1, 1), (5, 3))[:L]
    inst = small(3, P=P, Z=Z, levels=levels, X=7, Y=9)
    check(fb, inst, device, what=f"P={P} Z={Z} L={L}")


@pytest.mark.parametrize("X,Y", [(1, 1), (3, 50), (50, 3), (37, 41)])
def test_sca_grid_shapes(fb, device, X, Y):
    check(fb, small(4, X=X, Y=Y, dx=50.0 / X, dy=50.0 / Y, x_min=-25.0, y_min=-25.0), device,
          what=f"grid {X}x{Y}")


@pytest.mark.parametrize("P", synth.SCA_P_SWEEP)
def test_sca_bevformer_base(fb, device, P):
    """Table 7's setting in full, every output element checked."""
    inst = synth.make_sca_workload(synth.sca_config("sca_base", P=P))
    _, _, cnt = check(fb, inst, device, what=f"sca_base P={P}")
    assert cnt["hits"] > 40000


def test_sca_bevformer_base_bf16_two_batches(fb, device):
    inst = synth.make_sca_workload(synth.sca_config("sca_base_bf16"))
    check(fb, inst, device, what="sca_base_bf16")


def test_sca_overwrites_prefilled_output(fb, device):
    check(fb, small(5), device, what="prefilled NaN", prefill=float("nan"))


def test_sca_degenerate_inputs(fb, device):
    import torch
    # offsets far outside every map and non-finite offsets: hit cameras, no taps
    inst = small(6)
    inst.offsets[:, : inst.wl.Q // 2] = 1e9
    inst.offsets[:, inst.wl.Q // 2:, :, :, ::2] = np.nan
    check(fb, inst, device, what="far and NaN offsets")
    # a 1x1 map on every level
    check(fb, small(7, levels=((1, 1), (1, 1))), device, what="1x1 maps")
    # no cameras: every output is zero
    inst = small(8, N=0)
    gpu = gpu_sca(fb, inst, device, prefill=5.0)
    assert np.all(gpu == 0.0)
    # an empty batch enqueues nothing
    wl = synth.ScaWorkload(name="e", cfg_id=1, B=0, N=6, img_h=64, img_w=64, levels=((4, 4),),
                           C=8, heads=2, P=2, Z=2, dtype="f32", X=3, Y=3, x_min=0, dx=1,
                           y_min=0, dy=1)
    out = fb.sca_forward(torch.zeros((0, 6, 16, 8), device=device),
                         torch.zeros((0, 6, 4, 4), device=device), [0.0, 1.0], fb.grid_of(wl),
                         (64, 64), wl.levels, 2, torch.zeros((0, 9, 2, 1, 2, 2), device=device),
                         torch.zeros((0, 9, 2, 1, 2), device=device))
    assert out.shape == (0, 9, 8)


def test_sca_unaligned_value_buffer(fb, device):
    import torch
    inst = small(9, C=32, heads=4)
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    buf = torch.zeros(v.numel() + 1, dtype=torch.float32, device=device)
    view = buf[1:].view(v.shape)           # 4-byte but not 16-byte aligned
    view.copy_(v)
    out = torch.full((wl.B, wl.Q, wl.C), 7.0, dtype=torch.float32, device=device)
    rc = fb.sca_forward_raw(view.data_ptr(), "f32", tuple(v.shape), wl.heads, wl.levels,
                            l2i.data_ptr(), inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.P,
                            off.data_ptr(), lg.data_ptr(), out.data_ptr())
    torch.cuda.synchronize()
    assert rc == 0
    ref, scale, terms, _ = oracle.sca_instance(inst)
    assert_sca_parity(out.cpu().numpy(), ref, scale, terms, wl.heads, "unaligned value")


def test_sca_on_side_stream(fb, device):
    import torch
    inst = small(10)
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    s = torch.cuda.Stream(device)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        out = fb.sca_forward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels,
                             wl.heads, off, lg, stream=s)
    s.synchronize()
    ref, scale, terms, _ = oracle.sca_instance(inst)
    assert_sca_parity(out.cpu().numpy(), ref, scale, terms, wl.heads, "side stream")


def test_sca_allocates_nothing_beyond_its_output(fb, device):
    import torch
    inst = synth.make_sca_workload(synth.sca_config("sca_base", X=100, Y=100, dx=1.024,
                                                    dy=1.024))
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    out = torch.empty((wl.B, wl.Q, wl.C), dtype=torch.float32, device=device)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats(device)
    base = torch.cuda.memory_allocated(device)
    fb.sca_forward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels, wl.heads,
                   off, lg, out=out)
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated(device) == base


def test_prepared_sca_matches_oracle(fb, device):
    import torch
    inst = small(11)
    wl = inst.wl
    v, l2i, off, lg = _dev(inst, device)
    out = torch.full((wl.B, wl.Q, wl.C), float("nan"), dtype=torch.float32, device=device)
    call = fb.prepare_sca_forward(v, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                  wl.levels, wl.heads, off, lg, out)
    call()
    call()
    torch.cuda.synchronize()
    ref, scale, terms, _ = oracle.sca_instance(inst)
    assert_sca_parity(out.cpu().numpy(), ref, scale, terms, wl.heads, "prepared")


@pytest.mark.parametrize("what,kw", [
    ("32 cameras", dict(N=32, X=6, Y=5)),
    ("32 anchors", dict(Z=32, P=32, levels=((12, 32),), X=6, Y=5)),
    ("L*P = 512", dict(P=64, Z=8, levels=((24, 64), (12, 32), (6, 16), (3, 8), (2, 4), (1, 2),
                                         (1, 1), (5, 3)), X=4, Y=3)),
    ("1 KiB head rows", dict(C=256, heads=1, X=6, Y=5)),
    ("512-element bf16 heads", dict(C=1024, heads=2, dtype="bf16", X=5, Y=4)),
])
def test_sca_limits(fb, device, what, kw):
    check(fb, small(12, **kw), device, what=what)
