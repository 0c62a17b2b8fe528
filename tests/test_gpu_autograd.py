"""The differentiable wrappers (sample_vt_autograd, sca_autograd) on the GPU.

A loss through each wrapper must reproduce the operator's forward and, on
backward, the gradients of the explicit backward calls that the parity tests
check against the oracle: bitwise where the backward has no atomics (the
gather-form feature gradient, the FlashSCA offset and logit gradients), to a
few float32 roundings of the gradient's scale for the FlashSCA value
gradient, whose float atomics add in any order.
"""
import numpy as np
import pytest

import synth
import test_gpu_parity as tp
import test_gpu_sca as ts

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fb():
    import paper_2607_10071_amd as m
    return m


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sample_vt_autograd_matches_the_backward(fb, device, dtype):
    import torch
    inst = tp.small(B=2, C=40, dtype=dtype, X=23, Y=19, Z=5, cfg_id=901)
    wl = inst.wl
    ft, l2i = tp.to_dev(inst, device)
    grid, img = fb.grid_of(wl), (wl.img_h, wl.img_w)
    x = ft.clone().requires_grad_(True)
    l2i_g = l2i.clone().requires_grad_(True)
    out = fb.sample_vt_autograd(x, l2i_g, inst.z, grid, img)
    ref = fb.sample_vt(ft, l2i, inst.z, grid, img)
    g = torch.from_numpy(np.random.default_rng(5).standard_normal(
        tuple(out.shape)).astype(np.float32)).to(device)
    (out * g).sum().backward()
    want = fb.sample_vt_backward(g, l2i, inst.z, grid, img, tuple(ft.shape), dtype)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), ref)
    assert x.grad is not None and x.grad.dtype == ft.dtype
    assert torch.equal(x.grad, want.to(ft.dtype))
    assert l2i_g.grad is None   # the camera matrices are fixed inputs


def test_sca_autograd_matches_the_backward(fb, device):
    import torch
    inst = ts.small(31, C=64, heads=8, X=13, Y=11)
    wl = inst.wl
    v, l2i, off, lg = ts._dev(inst, device)
    grid, img = fb.grid_of(wl), (wl.img_h, wl.img_w)
    vv = v.clone().requires_grad_(True)
    oo = off.clone().requires_grad_(True)
    ll = lg.clone().requires_grad_(True)
    out = fb.sca_autograd(vv, l2i, inst.z, grid, img, wl.levels, wl.heads, oo, ll)
    ref = fb.sca_forward(v, l2i, inst.z, grid, img, wl.levels, wl.heads, off, lg)
    g = torch.from_numpy(np.random.default_rng(6).standard_normal(
        tuple(out.shape)).astype(np.float32)).to(device)
    (out * g).sum().backward()
    want = fb.sca_backward(v, l2i, inst.z, grid, img, wl.levels, wl.heads, off, lg, g)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), ref)
    assert torch.equal(oo.grad, want["offsets"])
    assert torch.equal(ll.grad, want["logits"])
    a, b = vv.grad.double(), want["value"].double()
    assert float((a - b).abs().max()) <= 1e-5 * max(float(b.abs().max()), 1e-30)


def test_sca_autograd_only_the_needed_gradients(fb, device):
    import torch
    inst = ts.small(32, C=32, heads=4, X=9, Y=7)
    wl = inst.wl
    v, l2i, off, lg = ts._dev(inst, device)
    grid, img = fb.grid_of(wl), (wl.img_h, wl.img_w)
    ll = lg.clone().requires_grad_(True)
    out = fb.sca_autograd(v, l2i, inst.z, grid, img, wl.levels, wl.heads, off, ll)
    out.sum().backward()
    want = fb.sca_backward(v, l2i, inst.z, grid, img, wl.levels, wl.heads, off, lg,
                           torch.ones_like(out), want=("logits",))
    torch.cuda.synchronize()
    assert torch.equal(ll.grad, want["logits"])
    assert v.grad is None and off.grad is None
