"""The no-allocation backward (flashbev_sample_vt_backward_noalloc) against
the workspace entry point (flashbev_sample_vt_backward_ws) on the GPU.

Both run the same two kernels on the same inputs; the gather form sums in a
fixed order, so the two gradients must be bitwise equal.  Two no-allocation
calls in a row, the second on a smaller input, check that the second call
reads nothing left in the shared scratch by the first.  All calls go
through the C ABI via the thin binding.
"""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fb():
    import paper_2607_10071_amd as m
    return m


def _inputs(name, device, seed):
    import torch
    wl = synth.config(name)
    inst = synth.make_workload(wl)
    rng = np.random.default_rng([wl.cfg_id, 11, seed])
    g = rng.standard_normal((wl.B, wl.C, wl.X, wl.Y)).astype(np.float32)
    l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(device)
    return wl, inst, torch.from_numpy(g).to(device), l2i


def _with_workspace(fb, wl, inst, gout, l2i, device):
    import torch
    need = fb.backward_workspace_size(inst.features.shape, wl.dtype, inst.z, fb.grid_of(wl),
                                      (wl.img_h, wl.img_w))
    ws = torch.empty(need, dtype=torch.uint8, device=device)
    gf = torch.full(inst.features.shape, float("nan"), dtype=torch.float32, device=device)
    fb.sample_vt_backward(gout, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                          inst.features.shape, wl.dtype, grad_features=gf, method="gather",
                          workspace=ws)
    torch.cuda.synchronize()
    return gf.cpu().numpy()


def test_noalloc_matches_workspace_entry_point_twice(fb, device):
    import torch
    results = []
    for name, seed in (("rep", 0), ("tiny", 1)):   # the second input is smaller
        wl, inst, gout, l2i = _inputs(name, device, seed)
        print(f"[case] noalloc {name} shape={inst.features.shape}", flush=True)
        gf = torch.full(inst.features.shape, float("nan"), dtype=torch.float32, device=device)
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(device)
        base = torch.cuda.memory_allocated(device)
        fb.sample_vt_backward_noalloc(gout, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                      inst.features.shape, wl.dtype, gf)
        torch.cuda.synchronize()
        assert torch.cuda.max_memory_allocated(device) == base
        got = gf.cpu().numpy()
        ref = _with_workspace(fb, wl, inst, gout, l2i, device)
        assert np.isfinite(got).all()
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), name
        assert np.any(got != 0.0)
        results.append(got)
    assert results[0].shape != results[1].shape


def test_noalloc_rejects_work_beyond_the_scratch(fb, device):
    import torch
    wl, inst, gout, l2i = _inputs("half_batch", device, 2)
    gf = torch.zeros(inst.features.shape, dtype=torch.float32, device=device)
    with pytest.raises(fb.FlashBevError) as e:
        fb.sample_vt_backward_noalloc(gout, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                      inst.features.shape, wl.dtype, gf)
    assert e.value.status == fb.STATUS["ERR_SCRATCH"]
    torch.cuda.synchronize()
    assert float(gf.abs().sum()) == 0.0   # nothing was launched
