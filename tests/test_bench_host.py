"""Host-side logic of bench.py, pinned against figures the paper prints.

tests/golden/paper_figures.json holds the cited values.  The bench reports
the tensorized baseline's analytic footprint (Alg. 1 materializes
Features3D = B N C X Y Z elements, plus a masked copy of it) and the
algorithmic bytes of one fused call (features and matrices read once, the
output written once).
"""
import json
import os

import pytest

import bench
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_figures.json")


def ref_workload():
    g = json.load(open(GOLDEN))["reference_setting"]
    return synth.Workload(name="paper_ref", cfg_id=6, B=g["B"], N=g["N"], img_h=448, img_w=800,
                          H=g["H"], W=g["W"], C=g["C"], dtype=g["dtype"], X=g["X"], Y=g["Y"],
                          x_min=-50.0, dx=0.5, y_min=-50.0, dy=0.5, z_lo=-5.0, z_hi=5.0, Z=g["Z"])


def test_features3d_footprint_matches_table4():
    # the tensorized forward holds Features3D and its masked copy at once:
    # 2 x 983.04 MB = 1966.08 MB against the printed 1971.94 MB
    gold = json.load(open(GOLDEN))["table4_tensorized_forward_peak_MB"]["value"]
    fp = bench.tensorized_footprint(ref_workload())
    assert fp["features3d_bytes"] == 1 * 6 * 128 * 200 * 200 * 8 * 4
    assert abs(2 * fp["features3d_bytes"] / 1e6 - gold) / gold < 0.01
    # the sum of all Alg. 1 intermediates bounds the peak from above
    assert fp["alg1_all_writes_bytes"] / 1e6 > gold


def test_fused_footprint_matches_table6_and_is_independent_of_z():
    gold = json.load(open(GOLDEN))["table6_flashbev_trt_peak_MB"]["value"]
    for z in (8, 16, 32):
        wl = ref_workload().with_(Z=z)
        inputs_and_output = bench.algorithmic_bytes(wl) - wl.B * wl.N * 64  # minus the matrices
        assert abs(inputs_and_output / 1e6 - gold) / gold < 0.01
        assert bench.algorithmic_bytes(wl) == bench.algorithmic_bytes(ref_workload())


def test_tensorized_footprint_grows_linearly_in_z_like_table6():
    vals = json.load(open(GOLDEN))["table6_tensorized_trt_peak_MB"]["value"]
    # printed increments: 2514-1294 = 1220 and 4994-2514 = 2480 (ratio ~2)
    f = [bench.tensorized_footprint(ref_workload().with_(Z=z))["features3d_bytes"] for z in (8, 16, 32)]
    assert (f[2] - f[1]) == 2 * (f[1] - f[0])
    assert abs((vals[2] - vals[1]) / (vals[1] - vals[0]) - 2.0) < 0.05


def test_samples_per_call_definition():
    wl = synth.config("rep")
    assert wl.samples == 1 * 200 * 200 * 8 * 6 == 1_920_000
    assert bench.algorithmic_bytes(wl) == 6 * 32 * 88 * 80 * 4 + 6 * 64 + 80 * 200 * 200 * 4


def test_traffic_is_dropped_when_the_kernel_changes(tmp_path, monkeypatch):
    data = {"rep": {"kernel_sha": "0" * 16, "bytes_per_launch": 123}}
    (tmp_path / "traffic.json").write_text(json.dumps(data))
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path))
    assert bench.load_traffic("rep") is None
    data["rep"]["kernel_sha"] = bench.kernel_hash()
    (tmp_path / "traffic.json").write_text(json.dumps(data))
    assert bench.load_traffic("rep") == 123
    assert bench.load_traffic("other") is None


def test_more_than_one_gpu_is_refused():
    assert bench.main(["--gpus", "2"]) == 2
