"""HIP graph capture of every compute entry point (torch.cuda.CUDAGraph).

The entry points allocate nothing and enqueue kernels only (the gradient
fills are kernels, not memsets), so a captured call can be replayed.  Each
test captures one call on the capture stream, then replays it several times.
Before every replay new inputs of the same shapes are copied into the
captured buffers; eager work and synchronizations run between replays.  Every
replay is checked against the oracle on that replay's inputs, under the bars
of the plain parity tests.
"""
import numpy as np
import pytest

import oracle
import synth
import test_gpu_backward as tb
import test_gpu_parity as tp
import test_gpu_sca as ts
import test_gpu_sca_backward as tsb

pytestmark = pytest.mark.gpu

REPLAYS = 3


@pytest.fixture(scope="module")
def fb():
    import paper_2607_10071_amd as m
    return m


def _eager_noise(device):
    """Unrelated eager work between replays."""
    import torch
    x = torch.randn(4096, device=device)
    return float((x * x).sum().item())


def _fbev_instances(n):
    return [tp.small(B=2, N=6, C=40, X=23, Y=19, Z=5, cfg_id=900 + k) for k in range(n)]


def test_forward_replays(fb, device):
    import torch
    insts = _fbev_instances(REPLAYS + 1)
    wl = insts[0].wl
    ft, l2i = tp.to_dev(insts[0], device)
    out = torch.empty((wl.B, wl.C, wl.X, wl.Y), dtype=torch.float32, device=device)
    grid, img = fb.grid_of(wl), (wl.img_h, wl.img_w)
    fb.sample_vt(ft, l2i, insts[0].z, grid, img, out=out)       # eager call first
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fb.sample_vt(ft, l2i, insts[0].z, grid, img, out=out)
    for k, inst in enumerate(insts[1:]):
        print(f"[case] forward graph replay {k} cfg_id={inst.wl.cfg_id}", flush=True)
        f2, m2 = tp.to_dev(inst, device)
        ft.copy_(f2)
        l2i.copy_(m2)
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        _eager_noise(device)
        torch.cuda.synchronize()
        ref, scale, _ = oracle.run_instance(inst)
        tp.assert_parity(out.cpu().numpy(), ref, scale, tp.RTOL[wl.dtype], f"graph replay {k}")


def test_prepared_forward_replays(fb, device):
    import torch
    insts = _fbev_instances(REPLAYS + 1)
    wl = insts[0].wl
    ft, l2i = tp.to_dev(insts[0], device)
    out = torch.empty((wl.B, wl.C, wl.X, wl.Y), dtype=torch.float32, device=device)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        # the stream is taken when the call is prepared: inside the capture
        call = fb.prepare_sample_vt(ft, l2i, insts[0].z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                    out)
        call()
    for k, inst in enumerate(insts[1:]):
        f2, m2 = tp.to_dev(inst, device)
        ft.copy_(f2)
        l2i.copy_(m2)
        torch.cuda.synchronize()
        graph.replay()
        _eager_noise(device)
        torch.cuda.synchronize()
        ref, scale, _ = oracle.run_instance(inst)
        tp.assert_parity(out.cpu().numpy(), ref, scale, tp.RTOL[wl.dtype], f"prepared replay {k}")


def test_backward_replays(fb, device):
    """The backward's two launches (fill, then the tiled scatter with its
    raised LDS limit) in one graph."""
    import torch
    insts = _fbev_instances(REPLAYS + 1)
    wl = insts[0].wl
    shape = insts[0].features.shape
    grid, img = fb.grid_of(wl), (wl.img_h, wl.img_w)
    _, l2i = tp.to_dev(insts[0], device)
    g = torch.from_numpy(tb._grad_out(wl)).to(device)
    gf = torch.empty(shape, dtype=torch.float32, device=device)
    fb.sample_vt_backward(g, l2i, insts[0].z, grid, img, shape, wl.dtype, grad_features=gf)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fb.sample_vt_backward(g, l2i, insts[0].z, grid, img, shape, wl.dtype, grad_features=gf)
    for k, inst in enumerate(insts[1:]):
        print(f"[case] backward graph replay {k} cfg_id={inst.wl.cfg_id}", flush=True)
        _, m2 = tp.to_dev(inst, device)
        gnew = tb._grad_out(inst.wl)
        l2i.copy_(m2)
        g.copy_(torch.from_numpy(gnew))
        gf.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        _eager_noise(device)
        torch.cuda.synchronize()
        ref, scale, terms = oracle.backward_instance(inst, gnew)
        tb.assert_bwd_parity(gf.cpu().numpy(), ref, scale, terms, f"graph replay {k}")


def _sca_instances(n, **kw):
    return [ts.small(20 + k, **kw) for k in range(n)]


def test_sca_forward_replays(fb, device):
    import torch
    insts = _sca_instances(REPLAYS + 1)
    wl = insts[0].wl
    v, l2i, off, lg = ts._dev(insts[0], device)
    out = torch.empty((wl.B, wl.Q, wl.C), dtype=torch.float32, device=device)
    args = (insts[0].z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels, wl.heads)
    fb.sca_forward(v, l2i, *args, off, lg, out=out)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fb.sca_forward(v, l2i, *args, off, lg, out=out)
    for k, inst in enumerate(insts[1:]):
        print(f"[case] sca graph replay {k} cfg_id={inst.wl.cfg_id}", flush=True)
        for dst, src in zip((v, l2i, off, lg), ts._dev(inst, device)):
            dst.copy_(src)
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        _eager_noise(device)
        torch.cuda.synchronize()
        ref, scale, terms, _ = oracle.sca_instance(inst)
        ts.assert_sca_parity(out.cpu().numpy(), ref, scale, terms, wl.heads, f"graph replay {k}")


@pytest.mark.parametrize("kw", [{}, dict(P=64, Z=8, levels=((24, 64), (12, 32), (6, 16), (3, 8),
                                                         (2, 4), (1, 2), (1, 1), (5, 3)),
                                         X=4, Y=3)],
                         ids=["default", "lds-above-64k"])
def test_sca_backward_replays(fb, device, kw):
    """The fill and the scatter kernel in one graph; the second case needs
    more than 64 KiB of LDS, so its launch raises the kernel's LDS limit."""
    import torch
    insts = _sca_instances(REPLAYS + 1, **kw)
    wl = insts[0].wl
    v, l2i, off, lg = ts._dev(insts[0], device)
    g = torch.from_numpy(tsb._g(wl)).to(device)
    outs = dict(grad_value=torch.empty((wl.B, wl.N, wl.S, wl.C), device=device),
                grad_offsets=torch.empty(tuple(off.shape), device=device),
                grad_logits=torch.empty(tuple(lg.shape), device=device))
    args = (insts[0].z, fb.grid_of(wl), (wl.img_h, wl.img_w), wl.levels, wl.heads)
    fb.sca_backward(v, l2i, *args, off, lg, g, **outs)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fb.sca_backward(v, l2i, *args, off, lg, g, **outs)
    for k, inst in enumerate(insts[1:]):
        print(f"[case] sca backward graph replay {k} cfg_id={inst.wl.cfg_id}", flush=True)
        for dst, src in zip((v, l2i, off, lg), ts._dev(inst, device)):
            dst.copy_(src)
        gnew = tsb._g(inst.wl)
        g.copy_(torch.from_numpy(gnew))
        for t in outs.values():
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        _eager_noise(device)
        torch.cuda.synchronize()
        gpu = {"value": outs["grad_value"].cpu().numpy(),
               "offsets": outs["grad_offsets"].cpu().numpy(),
               "logits": outs["grad_logits"].cpu().numpy()}
        ref = oracle.sca_backward_instance(inst, gnew)
        tsb.assert_bwd_parity(gpu, ref, wl, f"graph replay {k}")
