"""GPU parity on seeded random shapes (forward, backward and FlashSCA).

Each case draws its dimensions from a fixed seed: camera count, feature-map
size, channels and dtype, grid shape and extent, height bins, and for
FlashSCA heads, levels, points and anchors.  Every element is compared with
the oracle under the same bars as the other parity tests.  The shapes stay
small so the oracle answers in well under a second per case.  A second
FlashSCA family draws grids of whole 16 x 16 query blocks, 8 or 16 heads and
many points per head, the shapes that take the heads-to-XCDs and azimuth
orders.
"""
import numpy as np
import pytest

import synth
import test_gpu_backward as tb
import test_gpu_parity as tp
import test_gpu_sca as ts
import test_gpu_sca_backward as tsb

pytestmark = pytest.mark.gpu

DTYPES = ("f32", "f16", "bf16")


def _fbev_workload(seed):
    r = np.random.default_rng([7001, seed])
    img_h, img_w = int(r.choice([128, 256, 384])), int(r.choice([352, 704, 800]))
    stride = int(r.choice([4, 8, 16]))
    half = float(r.uniform(10.0, 60.0))
    X, Y = int(r.integers(1, 70)), int(r.integers(1, 70))
    return synth.Workload(
        name=f"rand{seed}", cfg_id=9000 + seed, B=int(r.integers(1, 3)), N=int(r.integers(1, 9)),
        img_h=img_h, img_w=img_w, H=max(1, img_h // stride), W=max(1, img_w // stride),
        C=int(r.choice([1, 3, 8, 16, 33, 64, 80, 128, 200])), dtype=str(r.choice(DTYPES)),
        X=X, Y=Y, x_min=-half, dx=2 * half / X, y_min=-half, dy=2 * half / Y,
        z_lo=-5.0, z_hi=float(r.uniform(0.0, 6.0)), Z=int(r.integers(1, 13)))


@pytest.mark.parametrize("seed", range(40))
def test_forward_random_shapes(device, seed):
    import paper_2607_10071_amd as fb
    inst = synth.make_workload(_fbev_workload(seed))
    reduce = "sum" if seed % 5 == 4 else "mean"
    tp.check_instance(fb, inst, device, reduce, what=f"random forward {seed}")


@pytest.mark.parametrize("seed", range(40))
def test_backward_random_shapes(device, seed):
    import paper_2607_10071_amd as fb
    wl = _fbev_workload(100 + seed)
    inst = synth.make_workload(wl)
    reduce = "sum" if seed % 4 == 3 else "mean"
    tb.check(fb, inst, device, reduce, what=f"random backward {seed}")


def _sca_workload(seed):
    r = np.random.default_rng([7002, seed])
    L = int(r.integers(1, 5))
    levels = tuple((int(r.integers(1, 40)), int(r.integers(1, 60))) for _ in range(L))
    Z = int(r.choice([1, 2, 3, 4]))
    P = Z * int(r.integers(1, 5))
    heads = int(r.choice([1, 2, 3, 4, 8]))
    D = int(r.choice([1, 3, 4, 8, 16, 32]))
    half = float(r.uniform(10.0, 60.0))
    X, Y = int(r.integers(1, 30)), int(r.integers(1, 30))
    return synth.ScaWorkload(
        name=f"srand{seed}", cfg_id=9500 + seed, B=int(r.integers(1, 3)),
        N=int(r.integers(1, 9)), img_h=int(r.choice([256, 448, 900])),
        img_w=int(r.choice([704, 800, 1600])), levels=levels, C=heads * D, heads=heads, P=P, Z=Z,
        dtype=str(r.choice(DTYPES)), X=X, Y=Y, x_min=-half, dx=2 * half / X, y_min=-half,
        dy=2 * half / Y, offset_noise=float(r.uniform(0.0, 3.0)))


@pytest.mark.parametrize("seed", range(40))
def test_sca_forward_random_shapes(device, seed):
    import paper_2607_10071_amd as fb
    inst = synth.make_sca_workload(_sca_workload(seed))
    reduce = "sum" if seed % 5 == 4 else "mean"
    ts.check(fb, inst, device, reduce, what=f"random sca {seed}")


@pytest.mark.parametrize("seed", range(40))
def test_sca_backward_random_shapes(device, seed):
    import paper_2607_10071_amd as fb
    inst = synth.make_sca_workload(_sca_workload(100 + seed))
    reduce = "sum" if seed % 4 == 3 else "mean"
    tsb.check(fb, inst, device, reduce, what=f"random sca backward {seed}")


def _sca_ordered_workload(seed):
    # grids of whole 16 x 16 query blocks, heads a multiple of 8 and many
    # points per head: the shapes that take the heads-to-XCDs order and the
    # azimuth order of the blocks (forward from 128 points per head,
    # backward above 32)
    r = np.random.default_rng([7003, seed])
    L = int(r.integers(2, 5))
    levels = tuple((int(r.integers(2, 30)), int(r.integers(2, 50))) for _ in range(L))
    Z = int(r.choice([2, 4]))
    P = Z * int(r.integers(-(-33 // (Z * L)), -(-160 // (Z * L)) + 1))
    heads = int(r.choice([8, 16]))
    D = int(r.choice([2, 4, 8, 32]))
    half = float(r.uniform(15.0, 50.0))
    X, Y = 16 * int(r.integers(1, 3)), 16 * int(r.integers(1, 3))
    return synth.ScaWorkload(
        name=f"sord{seed}", cfg_id=9700 + seed, B=int(r.integers(1, 3)),
        N=int(r.integers(2, 7)), img_h=int(r.choice([256, 448])),
        img_w=int(r.choice([704, 800])), levels=levels, C=heads * D, heads=heads, P=P, Z=Z,
        dtype=str(r.choice(DTYPES)), X=X, Y=Y, x_min=-half, dx=2 * half / X, y_min=-half,
        dy=2 * half / Y, offset_noise=float(r.uniform(0.0, 3.0)))


@pytest.mark.parametrize("seed", range(12))
def test_sca_forward_random_ordered_shapes(device, seed):
    import paper_2607_10071_amd as fb
    inst = synth.make_sca_workload(_sca_ordered_workload(seed))
    ts.check(fb, inst, device, what=f"random ordered sca {seed}")


@pytest.mark.parametrize("seed", range(12))
def test_sca_backward_random_ordered_shapes(device, seed):
    import paper_2607_10071_amd as fb
    inst = synth.make_sca_workload(_sca_ordered_workload(100 + seed))
    tsb.check(fb, inst, device, what=f"random ordered sca backward {seed}")
