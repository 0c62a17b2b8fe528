"""Statelessness of the C ABI under concurrent callers (GPU).

The headers state that the library keeps no per-call state and that calls
may come from several threads on their own streams.  Here two host threads, each with
its own stream and its own inputs, issue forward, FlashSCA forward and
backward calls in a loop; every result must equal what the same call gives
alone (bitwise for the forwards, which have no atomics; within the parity
bar for the backward, whose float atomics may add in another order).  The
FlashSCA forward's run-to-run bitwise determinism is checked as well.
"""
import threading

import numpy as np
import pytest

import oracle
import synth
import test_gpu_backward as tb
import test_gpu_parity as tp
import test_gpu_sca as ts

pytestmark = pytest.mark.gpu

ITERS = 12


@pytest.fixture(scope="module")
def fb():
    import paper_2607_10071_amd as m
    return m


def test_sca_run_to_run_bitwise_determinism(fb, device):
    inst = ts.small(30, C=64, heads=8, X=17, Y=15)
    a = ts.gpu_sca(fb, inst, device)
    for _ in range(3):
        assert np.array_equal(ts.gpu_sca(fb, inst, device), a)


def _job(fb, device, seed):
    """Inputs, a call per operator on a private stream, and the results of
    the same calls made alone."""
    import torch
    inst = tp.small(B=1, N=6, C=48, X=29, Y=23, Z=6, cfg_id=700 + seed)
    wl = inst.wl
    ft, l2i = tp.to_dev(inst, device)
    g = torch.from_numpy(tb._grad_out(wl)).to(device)
    sca = ts.small(40 + seed, X=11, Y=13)
    sw = sca.wl
    v, m, off, lg = ts._dev(sca, device)
    st = torch.cuda.Stream(device)
    outs = {"fwd": torch.empty((wl.B, wl.C, wl.X, wl.Y), device=device),
            "bwd": torch.empty(tuple(inst.features.shape), device=device),
            "sca": torch.empty((sw.B, sw.Q, sw.C), device=device)}
    calls = {
        "fwd": fb.prepare_sample_vt(ft, l2i, inst.z, fb.grid_of(wl), (wl.img_h, wl.img_w),
                                    outs["fwd"], stream=st),
        "bwd": fb.prepare_sample_vt_backward(g, l2i, inst.z, fb.grid_of(wl),
                                             (wl.img_h, wl.img_w), inst.features.shape,
                                             wl.dtype, outs["bwd"], stream=st),
        "sca": fb.prepare_sca_forward(v, m, sca.z, fb.grid_of(sw), (sw.img_h, sw.img_w),
                                      sw.levels, sw.heads, off, lg, outs["sca"], stream=st),
    }
    alone = {}
    for k, call in calls.items():
        call()
        st.synchronize()
        alone[k] = outs[k].cpu().numpy().copy()
    return inst, sca, st, calls, outs, alone


def test_two_threads_on_their_own_streams(fb, device):
    import torch
    jobs = [_job(fb, device, s) for s in range(2)]
    torch.cuda.synchronize()
    errors = []

    def run(job):
        try:
            inst, sca, st, calls, outs, alone = job
            for _ in range(ITERS):
                for k in ("fwd", "sca", "bwd"):
                    calls[k]()
                st.synchronize()
                for k in ("fwd", "sca"):
                    if not np.array_equal(outs[k].cpu().numpy(), alone[k]):
                        errors.append(f"{k} differs from the call made alone")
                got = outs["bwd"].cpu().numpy()
                ref = alone["bwd"].astype(np.float64)
                if np.abs(got - ref).max(initial=0.0) > 1e-5 * np.abs(ref).max(initial=1.0):
                    errors.append("bwd differs from the call made alone")
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=run, args=(j,)) for j in jobs]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors[:5]
    # and the results made alone are the right ones
    for inst, sca, st, calls, outs, alone in jobs:
        ref, scale, _ = oracle.run_instance(inst)
        tp.assert_parity(alone["fwd"], ref, scale, tp.RTOL["f32"], "threads: forward")
        r2, s2, terms, _ = oracle.sca_instance(sca)
        ts.assert_sca_parity(alone["sca"], r2, s2, terms, sca.wl.heads, "threads: sca")
        rb, sb, tbs = oracle.backward_instance(inst, tb._grad_out(inst.wl))
        tb.assert_bwd_parity(alone["bwd"], rb, sb, tbs, "threads: backward")
