"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle (plain C) is rebuilt with gcc's -fsanitize=address,undefined and
  every entry point runs on the tiny FlashBEV and FlashSCA instances.
* The library's host code (argument checks and launch plans of both C ABIs)
  is rebuilt with the sanitizers on the host side only (-Xarch_host before
  each -fsanitize=; the gfx950 code is built as usual) and the ABI test
  files run against it.  Every case there stops before any HIP call, so no
  GPU is needed.

Each run is a subprocess with the sanitizer runtime preloaded (ASan must be
the first library loaded), leak checking off (the Python interpreter itself
is not instrumented) and UBSan halting on the first report.  Where another
library is already preloaded the tests skip rather than change that list.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

ORACLE_DRIVER = r"""
import sys
import numpy as np
sys.path.insert(0, sys.argv[2])
import oracle, synth
path = sys.argv[1]
oracle._build.LIB = path
inst = synth.make_workload(synth.config("tiny"))
wl = inst.wl
for reduce in ("mean", "sum"):
    oracle.run_instance(inst, reduce, 2)
g = np.random.default_rng(0).standard_normal((wl.B, wl.C, wl.X, wl.Y)).astype(np.float32)
oracle.backward_instance(inst, g, "mean", 2)
oracle.project(inst.lidar2img, inst.z, (wl.H, wl.W), (wl.img_h, wl.img_w), wl.B, wl.N, wl.X,
               wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy)
cells = np.array([[0, i, j] for i in range(0, wl.X, 7) for j in range(0, wl.Y, 5)], np.int32)
oracle.cells_instance(inst, cells, "mean", 2)
s = synth.make_sca_workload(synth.sca_config("sca_tiny"))
sw = s.wl
for reduce in ("mean", "sum"):
    oracle.sca_instance(s, reduce, 2, libpath=path)
gs = np.random.default_rng(1).standard_normal((sw.B, sw.Q, sw.C)).astype(np.float32)
oracle.sca_backward_instance(s, gs, "mean", 2, libpath=path)
oracle.sca_reference_points(s.lidar2img, s.z, sw.B, sw.N, (sw.img_h, sw.img_w), sw.X, sw.Y,
                            sw.x_min, sw.dx, sw.y_min, sw.dy, libpath=path)
assert oracle.lib()._name == path
print("oracle entry points done", flush=True)
"""

ABI_DRIVER = r"""
import sys
sys.path.insert(0, sys.argv[2])
import pytest
import paper_2607_10071_amd as fb
fb._LIB_PATH = sys.argv[1]
rc = pytest.main(["-q", "-p", "no:cacheprovider", "-m", "not gpu",
                  sys.argv[2] + "/tests/test_abi.py", sys.argv[2] + "/tests/test_sca_abi.py"])
assert fb._lib()._name == sys.argv[1]
sys.exit(int(rc))
"""


def _env(runtime):
    env = dict(os.environ)
    env["LD_PRELOAD"] = runtime
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "2"
    return env


def _check(proc):
    out = proc.stdout + proc.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert "runtime error" not in out, out[-4000:]
    assert proc.returncode == 0, out[-4000:]


@pytest.fixture(autouse=True)
def _no_other_preload():
    if os.environ.get("LD_PRELOAD"):
        pytest.skip("another library is preloaded; ASan's runtime has to come first")


def test_oracle_under_asan_and_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not found")
    runtime = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    if not os.path.isabs(runtime) or not os.path.exists(runtime):
        pytest.skip("gcc's ASan runtime not found")
    lib = str(tmp_path / "liboracle_san.so")
    src = [os.path.join(ROOT, "oracle", f) for f in ("flashbev_oracle.c", "flashsca_oracle.c")]
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off",
                    "-fno-fast-math", "-fPIC", "-shared", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    *src, "-o", lib, "-lm"], check=True)
    proc = subprocess.run([sys.executable, "-c", ORACLE_DRIVER, lib, ROOT], capture_output=True,
                          text=True, env=_env(runtime), timeout=600)
    _check(proc)
    assert "oracle entry points done" in proc.stdout


def test_abi_host_code_under_asan_and_ubsan(tmp_path):
    hipcc = "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    clang = "/opt/rocm/llvm/bin/clang"
    rt = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                        capture_output=True, text=True).stdout.strip() if os.path.exists(clang) else ""
    if not os.path.isabs(rt) or not os.path.exists(rt):
        pytest.skip("clang's ASan runtime not found")
    csrc = os.path.join(ROOT, "paper_2607_10071_amd", "csrc")
    lib = str(tmp_path / "libflashbev_san.so")
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
                    "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang",
                    "-packed-fp32-ops", "-fPIC", "-shared",
                    "-Xarch_host", "-fsanitize=address",
                    "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-fno-sanitize-recover=undefined",
                    "-Xarch_host", "-shared-libsan",
                    "-I" + os.path.join(ROOT, "include"), "-I" + csrc,
                    os.path.join(csrc, "flashbev.hip"), os.path.join(csrc, "flashsca.hip"),
                    "-o", lib], check=True, capture_output=True)
    proc = subprocess.run([sys.executable, "-c", ABI_DRIVER, lib, ROOT], capture_output=True,
                          text=True, env=_env(rt), timeout=600)
    _check(proc)
    assert " passed" in proc.stdout and "failed" not in proc.stdout, proc.stdout[-2000:]
