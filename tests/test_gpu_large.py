"""GPU parity of the forward at the scaling sweep's points (Sec. 4.4: height
bins, grid size and channels at the paper's reference setting).

The points the oracle finishes in seconds are checked element by element.
The two largest grids (1600 x 1600 and 3200 x 3200 cells, 1.3 and 5.2 GB
of output) are checked on every cell of their first and last tiles and on
4096 seeded random cells, each against the oracle's per-cell evaluation of
Eq. 1, and every output element must be finite.  These grids take the launch
plan's large-grid path: several rounds per tile (more than 256K one-round
tiles) and interleaved stripes of tiles per XCD (more than 2^30 gathered
bytes), which no smaller workload reaches.
"""
import math

import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

RTOL = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-3}


@pytest.fixture(scope="module")
def fb():
    import paper_2607_10071_amd as m
    return m


def ref_point(**kw):
    """The paper's reference setting with one axis changed; the grid keeps
    the +-50 m extent and refines the cells."""
    wl = synth.config("paper_ref")
    n = kw.pop("XY", None)
    if n is not None:
        kw.update(X=n, Y=n, dx=100.0 / n, dy=100.0 / n)
    return wl.with_(**kw)


def run_gpu(fb, inst, device):
    import torch
    wl = inst.wl
    ft = synth.to_storage(inst.features, wl.dtype).to(device)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    out = fb.sample_vt(ft, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w))
    torch.cuda.synchronize()
    del ft, l2i
    return out


@pytest.mark.parametrize("what,kw", [
    ("Z=4", dict(Z=4)), ("Z=16", dict(Z=16)), ("Z=64", dict(Z=64)), ("Z=256", dict(Z=256)),
    ("C=64", dict(C=64)), ("C=256", dict(C=256)), ("C=1024", dict(C=1024)),
    ("X=Y=800", dict(XY=800)),
])
def test_sweep_point_full(fb, device, what, kw):
    wl = ref_point(**kw)
    print(f"[case] paper_ref {what}: B={wl.B} C={wl.C} X={wl.X} Y={wl.Y} Z={wl.Z}", flush=True)
    inst = synth.make_workload(wl)
    g = run_gpu(fb, inst, device).cpu().numpy().astype(np.float64)
    r, s, _ = oracle.run_instance(inst)
    err = np.abs(g - r)
    bad = err > RTOL[wl.dtype] * s
    nz = s > 0
    print(f"[parity] paper_ref {what} max_scaled={float((err[nz] / s[nz]).max(initial=0)):.3e}",
          flush=True)
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} elements off"
    assert np.all(g[~nz] == 0.0)


def tile_cells(fb, wl, inst):
    """Cells per tile of the forward's launch plan (waves x rounds x cells
    per wavefront), recovered from the reported geometry."""
    info = fb.launch_info((wl.B, wl.N, wl.H, wl.W, wl.C), wl.dtype, inst.z, fb.grid_of(wl),
                          (wl.img_h, wl.img_w))
    waves = info["threads"] // 64
    XY = wl.X * wl.Y
    cand = [waves * r * info["cells_per_wave"] for r in range(1, 65)
            if wl.B * math.ceil(XY / (waves * r * info["cells_per_wave"])) == info["workgroups"]]
    assert cand, info
    return cand[0], info


@pytest.mark.parametrize("n", [1600, 3200])
def test_large_grid_sampled_cells(fb, device, n):
    import torch
    wl = ref_point(XY=n)
    inst = synth.make_workload(wl)
    T, info = tile_cells(fb, wl, inst)
    XY = wl.X * wl.Y
    # the large-grid path: several rounds per tile
    assert T > (info["threads"] // 64) * info["cells_per_wave"], (T, info)
    print(f"[case] paper_ref grid {n}x{n}: tile {T} cells, {info}", flush=True)
    out = run_gpu(fb, inst, device)
    assert bool(torch.isfinite(out).all())
    rng = np.random.default_rng([6, n])
    q = np.concatenate([np.arange(T), np.arange((math.ceil(XY / T) - 1) * T, XY),
                        rng.integers(0, XY, 4096)])
    cells = np.stack([np.zeros_like(q), q // wl.Y, q % wl.Y], axis=1).astype(np.int32)
    idx = torch.from_numpy(q).to(device)
    g = out[0].reshape(wl.C, XY).index_select(1, idx).t().cpu().numpy().astype(np.float64)
    del out
    torch.cuda.empty_cache()
    r, s = oracle.cells_instance(inst, cells)
    err = np.abs(g - r)
    nz = s > 0
    print(f"[parity] grid {n} cells={len(q)} max_scaled={float((err[nz] / s[nz]).max(initial=0)):.3e} "
          f"seen={int(nz.any(axis=1).sum())}", flush=True)
    assert nz.any(axis=1).sum() > len(q) // 10
    assert not (err > RTOL[wl.dtype] * s).any()
    assert np.all(g[~nz] == 0.0)
