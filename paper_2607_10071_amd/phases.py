"""Phase breakdowns of the fused Sampling-VT forward and the FlashSCA backward (measurement tool).

    python -m paper_2607_10071_amd.phases [workload ...]     (default: rep half_batch)

Runs the forward of each named synthetic workload through
``libflashbev_phases.so``, the operator library built once more with the
forward's phase clock compiled in (``include/flashbev_phases.h``): 50
untimed calls, then ``--calls`` calls (default 5) that each record every
wavefront's clock.  Prints one JSON line per workload with, over the
wavefronts of all recorded calls, the mean and median time per wavefront
in each phase of the forward (Sec. 3.3, Alg. 2):

  staging     camera rows and heights into LDS, and the workgroup barrier
  projection  projection, mask M_n and compaction of the samples (with the
              camera-culling test; the packed pass sets up its samples too)
  setup       bilinear set-up of the compacted samples (per-cell passes)
  pad         padding of the groups' sample lists to the gather's unroll
  gather      the bilinear gather-reduce
  stash       the group's sums into the LDS output tile
  barrier     waiting at the workgroup barrier before the stores
  store       the single write of the output tile

with each phase's share of the summed wavefront time, the kernel span (first
start to last end), the wavefronts' lifetime and start spread, and the
forward's per-call time through both libraries (best of three runs of 200
back-to-back prepared calls: the clock's overhead) and whether the two
libraries' outputs are bitwise equal.
Clock ticks are 10 ns (the 100 MHz real-time counter).

    python -m paper_2607_10071_amd.phases --sca-backward P [P ...]

runs the FlashSCA backward at BEVFormer-base defaults for each point count P
through the same library (its phase clock, ``flashsca_phase_log``) and prints,
per P, the mean time per wavefront in each step of that kernel (projection,
set-up, chunk records, point gradients, merge-table inserts and the barrier
after them, the walk of the distinct rows with its float atomics and the
barrier after it, emptying the table, the tail), with the chunk-camera steps
per wavefront and the distinct rows per step.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_PATH = os.path.join(HERE, "libflashbev_phases.so")
SLOTS = 16
TICK_US = 0.01
PHASES = ("staging", "projection", "setup", "pad", "gather", "stash", "barrier", "store")


def phase_table(log: np.ndarray) -> dict:
    """Per-phase statistics from clock records [waves, 16] (int64 ticks)."""
    live = log[:, 0] > 0
    d = log[live].astype(np.float64)
    start, staged, barrier, end = d[:, 0], d[:, 1], d[:, 7], d[:, 8]
    per = {
        "staging": staged - start,
        "projection": d[:, 2],
        "setup": d[:, 3],
        "pad": d[:, 4],
        "gather": d[:, 5],
        "stash": d[:, 6],
        "barrier": barrier - (staged + d[:, 2:7].sum(axis=1)),
        "store": end - barrier,
    }
    life = end - start
    total = life.sum()
    out = {"waves": int(live.sum()),
           "rounds_per_wave": float(np.mean(d[:, 9])),
           "passes_per_wave": float(np.mean(d[:, 10])),
           "wave_lifetime_us": {"median": round(float(np.median(life)) * TICK_US, 3),
                                "mean": round(float(np.mean(life)) * TICK_US, 3),
                                "max": round(float(np.max(life)) * TICK_US, 3)},
           "phases_us_per_wave": {}}
    for k in PHASES:
        v = per[k]
        out["phases_us_per_wave"][k] = {"mean": round(float(np.mean(v)) * TICK_US, 3),
                                        "median": round(float(np.median(v)) * TICK_US, 3),
                                        "share": round(float(v.sum() / total), 4)}
    return out


def run(names, calls: int = 5, device: str = "cuda:0") -> list:
    import torch

    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import paper_2607_10071_amd as fb
    import synth

    dev = torch.device(device)
    plain_path, plain_lib = fb._LIB_PATH, fb._LIB
    results = []
    try:
        for name in names:
            wl = synth.config(name)
            inst = synth.make_workload(wl)
            feats = synth.to_storage(inst.features, wl.dtype).to(dev)
            l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(dev)
            out = torch.empty((wl.B, wl.C, wl.X, wl.Y), dtype=torch.float32, device=dev)
            grid = fb.grid_of(wl)
            img = (wl.img_h, wl.img_w)
            per_call, outs = {}, []
            for tag, path in (("plain", plain_path), ("clocked", LIB_PATH)):
                fb._LIB_PATH, fb._LIB = path, None
                stream = torch.cuda.current_stream(dev)
                call = fb.prepare_sample_vt(feats, l2i, inst.z, grid, img, out, stream=stream)
                best = float("inf")
                for _ in range(3):
                    for _ in range(50):
                        call()
                    a = torch.cuda.Event(enable_timing=True)
                    b = torch.cuda.Event(enable_timing=True)
                    a.record(stream)
                    for _ in range(200):
                        call()
                    b.record(stream)
                    torch.cuda.synchronize()
                    best = min(best, a.elapsed_time(b) / 200 * 1e3)
                per_call[tag] = round(best, 2)
                outs.append(out.cpu().numpy().view(np.uint32).copy())
                del call
            # the clocked library is loaded: record `calls` calls
            lib = fb._lib()
            lib.flashbev_phase_log.argtypes = [ctypes.c_void_p]
            lib.flashbev_phase_log.restype = ctypes.c_int
            info = fb.launch_info((wl.B, wl.N, wl.H, wl.W, wl.C), wl.dtype, inst.z, grid, img)
            waves = info["workgroups"] * (info["threads"] // 64)
            logs = []
            buf = torch.zeros(waves * SLOTS, dtype=torch.int64, device=dev)
            with fb._on_device(dev):
                for _ in range(calls):
                    buf.zero_()
                    torch.cuda.synchronize()
                    if lib.flashbev_phase_log(ctypes.c_void_p(buf.data_ptr())) != 0:
                        raise RuntimeError("flashbev_phase_log failed")
                    fb.sample_vt(feats, l2i, inst.z, grid, img, out=out)
                    torch.cuda.synchronize()
                    if lib.flashbev_phase_log(None) != 0:
                        raise RuntimeError("flashbev_phase_log failed")
                    logs.append(buf.cpu().numpy().reshape(waves, SLOTS).copy())
            spans, spreads = [], []
            for lg in logs:
                live = lg[:, 0] > 0
                spans.append((lg[live, 8].max() - lg[live, 0].min()) * TICK_US)
                spreads.append((lg[live, 0].max() - lg[live, 0].min()) * TICK_US)
            rec = {"workload": name,
                   "config": f"B={wl.B} N={wl.N} {wl.H}x{wl.W} C={wl.C} {wl.dtype} "
                             f"BEV {wl.X}x{wl.Y} Z={wl.Z}",
                   "launch": info, "calls_recorded": calls,
                   "forward_us_per_call": per_call,
                   "outputs_bitwise_equal": bool(np.array_equal(outs[0], outs[1])),
                   "kernel_span_us_median": round(float(np.median(spans)), 3),
                   "wave_start_spread_us_median": round(float(np.median(spreads)), 3),
                   **phase_table(np.concatenate(logs))}
            results.append(rec)
            print(json.dumps(rec), flush=True)
            del feats, l2i, out, buf
    finally:
        fb._LIB_PATH, fb._LIB = plain_path, plain_lib
    return results


SCA_STEPS = (("projection", 1), ("setup", 2), ("records", 3), ("point_gradients", 4),
             ("inserts", 5), ("insert_barrier", 6), ("walk_and_atomics", 7),
             ("walk_barrier", 8), ("clear", 9), ("tail", 12))


def sca_backward_table(log: np.ndarray) -> dict:
    """Per-step statistics of the FlashSCA backward from clock records
    [waves, 16] (int64)."""
    live = log[:, 0] > 0
    d = log[live].astype(np.float64)
    life = d[:, 13] - d[:, 0]
    total = sum(d[:, k].sum() for _, k in SCA_STEPS)
    steps = d[:, 10].sum()
    out = {"waves": int(live.sum()),
           "steps_per_wave": round(float(np.mean(d[:, 10])), 3),
           "distinct_rows_per_step": round(float(d[:, 11].sum() / max(steps, 1.0)), 1),
           "wave_lifetime_us": {"median": round(float(np.median(life)) * TICK_US, 3),
                                "mean": round(float(np.mean(life)) * TICK_US, 3),
                                "max": round(float(np.max(life)) * TICK_US, 3)},
           "steps_us_per_wave": {}}
    for name, k in SCA_STEPS:
        out["steps_us_per_wave"][name] = {"mean": round(float(np.mean(d[:, k])) * TICK_US, 3),
                                          "share": round(float(d[:, k].sum() / total), 4)}
    return out


def run_sca_backward(points, calls: int = 3, device: str = "cuda:0") -> list:
    import torch

    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import paper_2607_10071_amd as fb
    import synth

    dev = torch.device(device)
    plain_path, plain_lib = fb._LIB_PATH, fb._LIB
    results = []
    try:
        for P in points:
            wl = synth.sca_config("sca_base", P=P)
            inst = synth.make_sca_workload(wl)
            v = synth.to_storage(inst.value, wl.dtype).to(dev)
            l2i = torch.from_numpy(np.ascontiguousarray(inst.lidar2img)).to(dev)
            off = torch.from_numpy(np.ascontiguousarray(inst.offsets)).to(dev)
            lg = torch.from_numpy(np.ascontiguousarray(inst.logits)).to(dev)
            g = torch.from_numpy(np.random.default_rng([wl.cfg_id, 9, 5]).standard_normal(
                (wl.B, wl.Q, wl.C)).astype(np.float32)).to(dev)
            gv = torch.empty((wl.B, wl.N, wl.S, wl.C), dtype=torch.float32, device=dev)
            go = torch.empty(tuple(off.shape), dtype=torch.float32, device=dev)
            gl = torch.empty(tuple(lg.shape), dtype=torch.float32, device=dev)
            grid, img = fb.grid_of(wl), (wl.img_h, wl.img_w)
            per_call = {}
            for tag, path in (("plain", plain_path), ("clocked", LIB_PATH)):
                fb._LIB_PATH, fb._LIB = path, None
                stream = torch.cuda.current_stream(dev)
                call = fb.prepare_sca_backward(v, l2i, inst.z, grid, img, wl.levels, wl.heads,
                                               off, lg, g, gv, go, gl, stream=stream)
                best = float("inf")
                for _ in range(3):
                    for _ in range(5):
                        call()
                    a = torch.cuda.Event(enable_timing=True)
                    b = torch.cuda.Event(enable_timing=True)
                    a.record(stream)
                    for _ in range(20):
                        call()
                    b.record(stream)
                    torch.cuda.synchronize()
                    best = min(best, a.elapsed_time(b) / 20)
                per_call[tag] = round(best, 4)
                del call
            lib = fb._lib()   # the clocked library is loaded
            lib.flashsca_phase_log.argtypes = [ctypes.c_void_p]
            lib.flashsca_phase_log.restype = ctypes.c_int
            info = fb.sca_launch_info((wl.B, wl.N, wl.S, wl.C), wl.dtype, wl.heads, wl.levels,
                                      inst.z, grid, img, P, backward=True)
            waves = info["workgroups"] * (info["threads"] // 64)
            buf = torch.zeros(waves * SLOTS, dtype=torch.int64, device=dev)
            logs = []
            with fb._on_device(dev):
                for _ in range(calls):
                    buf.zero_()
                    torch.cuda.synchronize()
                    if lib.flashsca_phase_log(ctypes.c_void_p(buf.data_ptr())) != 0:
                        raise RuntimeError("flashsca_phase_log failed")
                    fb.sca_backward(v, l2i, inst.z, grid, img, wl.levels, wl.heads, off, lg, g,
                                    grad_value=gv, grad_offsets=go, grad_logits=gl)
                    torch.cuda.synchronize()
                    if lib.flashsca_phase_log(None) != 0:
                        raise RuntimeError("flashsca_phase_log failed")
                    logs.append(buf.cpu().numpy().reshape(waves, SLOTS).copy())
            spans = []
            for lg_ in logs:
                live = lg_[:, 0] > 0
                spans.append((lg_[live, 13].max() - lg_[live, 0].min()) * TICK_US)
            rec = {"sca_backward": f"BEVFormer-base P={P}",
                   "config": f"B={wl.B} N={wl.N} C={wl.C} {wl.dtype} heads={wl.heads} "
                             f"levels={len(wl.levels)} BEV {wl.X}x{wl.Y} Z={wl.Z}",
                   "launch": info, "calls_recorded": calls, "backward_ms_per_call": per_call,
                   "kernel_span_us_median": round(float(np.median(spans)), 3),
                   **sca_backward_table(np.concatenate(logs))}
            results.append(rec)
            print(json.dumps(rec), flush=True)
            del v, l2i, off, lg, g, gv, go, gl, buf
    finally:
        fb._LIB_PATH, fb._LIB = plain_path, plain_lib
    return results


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("workloads", nargs="*", default=["rep", "half_batch"])
    ap.add_argument("--calls", type=int, default=5)
    ap.add_argument("--sca-backward", type=int, nargs="+", default=None, metavar="P")
    args = ap.parse_args(argv)
    if not os.path.exists(LIB_PATH):
        raise FileNotFoundError(f"{LIB_PATH} is not built (python -m paper_2607_10071_amd.build)")
    if args.sca_backward:
        run_sca_backward(args.sca_backward, min(args.calls, 3))
    else:
        run(args.workloads, args.calls)
    return 0


if __name__ == "__main__":
    sys.exit(main())
