"""Property tests of the C ABI's argument checks and launch plans (CPU only).

Random dimensions, dtypes, grids, heights and point counts, extreme ones
included, go through the launch-geometry entry points of both operators,
which run every argument check and the whole launch plan without a HIP
call.  Every call must return a documented status; an accepted one must
give a launch the hardware can run (workgroups within the grid limit, at
most 1024 threads, LDS within 160 KiB) and one that covers the output.
"""
import math

import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

import paper_2607_10071_amd as fb  # noqa: E402

STATUS = set(fb.STATUS.values())
LDS_MAX = 160 * 1024

dims = st.one_of(st.integers(-3, 70), st.integers(70, 5000), st.sampled_from([2**31 - 1, 2**20]))
small = st.integers(-2, 40)


def _status(e):
    return e.status if isinstance(e, fb.FlashBevError) else None


@settings(max_examples=600, deadline=None)
@given(B=small, N=st.integers(-1, 70), H=dims, W=dims, C=st.integers(-1, 2100),
       dtype=st.sampled_from(["f32", "f16", "bf16"]), X=dims, Y=dims,
       Z=st.integers(-1, 300), img=st.integers(-1, 4000), backward=st.booleans())
def test_flashbev_plans(B, N, H, W, C, dtype, X, Y, Z, img, backward):
    grid = fb.BevGrid(-50.0, 0.5, X, -50.0, 0.5, Y)
    z = np.linspace(-4.0, 2.0, max(Z, 0)).astype(np.float32)
    shape = (B, N, H, W, C)
    info_fn = fb.backward_launch_info if backward else fb.launch_info
    try:
        # a negative Z cannot be expressed by a host array; it is tested in test_abi
        info = info_fn(shape, dtype, z, grid, (img, img))
    except fb.FlashBevError as e:
        assert _status(e) in STATUS and _status(e) != 0
        return
    assert 0 <= info["workgroups"] <= 2**31 - 1
    assert 0 < info["threads"] <= 1024 and info["threads"] % 64 == 0
    assert 0 <= info["lds_bytes"] <= LDS_MAX
    if not backward and info["workgroups"] > 0:
        # the forward's tiles cover every output cell of every batch element
        cells = X * Y
        waves = info["threads"] // 64
        assert info["workgroups"] * waves * info["cells_per_wave"] * 64 >= B * cells


@settings(max_examples=600, deadline=None)
@given(B=small, N=st.integers(-1, 40), C=st.integers(-1, 1200), heads=st.integers(-1, 20),
       L=st.integers(0, 10), hw=st.integers(-1, 400), P=st.integers(-1, 80),
       Z=st.integers(1, 40), X=dims, Y=dims, dtype=st.sampled_from(["f32", "f16", "bf16"]),
       backward=st.booleans())
def test_flashsca_plans(B, N, C, heads, L, hw, P, Z, X, Y, dtype, backward):
    levels = [(hw, hw + 1)] * L
    S = sum(max(h, 0) * max(w, 0) for h, w in levels)
    grid = fb.BevGrid(-50.0, 0.5, X, -50.0, 0.5, Y)
    z = np.linspace(-4.0, 2.0, Z).astype(np.float32)
    try:
        info = fb.sca_launch_info((B, N, S, C), dtype, heads, levels, z, grid, (900, 1600), P,
                                  backward=backward)
    except (fb.FlashBevError, ValueError, ZeroDivisionError) as e:
        if isinstance(e, fb.FlashBevError):
            assert _status(e) in STATUS and _status(e) != 0
        return
    assert 0 <= info["workgroups"] <= 2**31 - 1
    assert 0 < info["threads"] <= 1024 and info["threads"] % 64 == 0
    assert 0 <= info["lds_bytes"] <= LDS_MAX
    assert info["lanes_per_head"] >= 1 and info["lane_bytes"] in (2, 4, 8, 16)
    if info["workgroups"] > 0:
        D = C // heads
        es = 4 if dtype == "f32" else 2
        assert info["lanes_per_head"] * info["lane_bytes"] >= D * es
        assert math.gcd(info["lanes_per_head"], 64) == info["lanes_per_head"]
