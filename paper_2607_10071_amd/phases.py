"""Phase breakdown of the fused Sampling-VT forward (measurement tool).

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


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("workloads", nargs="*", default=["rep", "half_batch"])
    ap.add_argument("--calls", type=int, default=5)
    args = ap.parse_args(argv)
    if not os.path.exists(LIB_PATH):
        raise FileNotFoundError(f"{LIB_PATH} is not built (python -m paper_2607_10071_amd.build)")
    run(args.workloads, args.calls)
    return 0


if __name__ == "__main__":
    sys.exit(main())
