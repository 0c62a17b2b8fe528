"""The forward through the C ABI alone, from a C++ program (GPU).

`tests/c_abi_forward` (built by build() from tests/c_abi_forward.cpp) uses
plain HIP memory and a HIP stream and no Python or torch.  The test writes a
seeded instance's inputs to a file, runs the program as a child process and
checks its output against the oracle under the bar of the forward parity
tests.
"""
import os
import subprocess

import numpy as np
import pytest

import oracle
import synth
import test_gpu_parity as tp

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi_forward")


def _write_inputs(path, inst, reduce):
    wl = inst.wl
    hdr = np.array([wl.B, wl.N, wl.H, wl.W, wl.C, wl.img_h, wl.img_w, wl.X, wl.Y, len(inst.z),
                    0 if reduce == "mean" else 1], np.int32)
    grid = np.array([wl.x_min, wl.dx, wl.y_min, wl.dy, wl.depth_eps], np.float32)
    with open(path, "wb") as f:
        for a in (hdr, grid, np.asarray(inst.features, np.float32),
                  np.asarray(inst.lidar2img, np.float32), np.asarray(inst.z, np.float32)):
            f.write(np.ascontiguousarray(a).tobytes())


@pytest.mark.parametrize("name,reduce", [("tiny", "mean"), ("tiny", "sum"), ("rep", "mean")])
def test_c_program_forward_matches_oracle(tmp_path, name, reduce):
    assert os.path.exists(EXE), "tests/c_abi_forward is not built: run __graft_entry__.build()"
    inst = synth.make_workload(synth.config(name))
    wl = inst.wl
    assert wl.dtype == "f32"
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    _write_inputs(inp, inst, reduce)
    print(f"[case] C program forward {name} {reduce}", flush=True)
    r = subprocess.run([EXE, str(inp), str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr + r.stdout
    gpu = np.fromfile(out, np.float32).reshape(wl.B, wl.C, wl.X, wl.Y)
    ref, scale, _ = oracle.run_instance(inst, reduce)
    tp.assert_parity(gpu, ref, scale, tp.RTOL["f32"], f"C program {name} {reduce}")
