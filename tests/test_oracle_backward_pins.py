"""Pins of the CPU oracle's backward (gradient of Eq. 1 w.r.t. the feature maps).

Eq. 1 is linear in the features, so its gradient is the transpose of a
linear map.  The backward oracle is pinned by:
  * the Jacobian of the independent numpy brute force (Alg. 1, tensorized),
    built column by column from unit feature maps on tiny inputs, then
    transposed and applied to a random output gradient;
  * the adjoint identity <fwd(F), G> = <F, bwd(G)> against the forward
    oracle (itself pinned in test_oracle_pins.py), in both reduce modes;
  * invariants: the per-pixel term counts add up to the forward's in-range
    tap count, and pixels no tap reaches get exactly zero.
"""
import numpy as np
import pytest

import oracle
import synth
from brute_force import tensorized_sample_vt
from test_oracle_pins import small_workload


def _bwd(inst, g, reduce="mean"):
    return oracle.backward_instance(inst, g, reduce)


def _grad(inst, seed=11):
    wl = inst.wl
    rng = np.random.default_rng(seed)
    return rng.standard_normal((wl.B, wl.C, wl.X, wl.Y)).astype(np.float32)


def _jacobian_brute(inst, reduce):
    """d out[b, :, i, j] / d F[b', n, y, x, :] for one channel, by columns."""
    wl = inst.wl
    B, N, H, W, _ = inst.features.shape
    cols = []
    for q in range(B * N * H * W):
        e = np.zeros((B, N, H, W, 1), dtype=np.float32)
        e.reshape(-1)[q] = 1.0
        out = tensorized_sample_vt(e, inst.lidar2img, inst.z, (wl.img_h, wl.img_w), wl.X, wl.Y,
                                   wl.x_min, wl.dx, wl.y_min, wl.dy, wl.depth_eps, reduce)
        cols.append(out[:, 0].reshape(-1))             # [B*X*Y]
    return np.stack(cols, axis=1)                      # [B*X*Y, B*N*H*W]


@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_backward_is_transpose_of_brute_force_jacobian(reduce):
    inst = small_workload(B=2, N=6, H=4, W=6, C=3, X=9, Y=8, Z=3, seed=4)
    wl = inst.wl
    B, N, H, W, C = inst.features.shape
    mask, _, _ = oracle.project(inst.lidar2img, inst.z, (H, W), (wl.img_h, wl.img_w), B, N,
                                wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy)
    assert (mask.sum(axis=-1) >= 2).any(), "no cell seen by two cameras: mean == sum"
    J = _jacobian_brute(inst, reduce)
    assert np.count_nonzero(J) > 20
    g = _grad(inst)
    gf, scale, terms = _bwd(inst, g, reduce)
    # channels are independent: the same J applies to every channel
    gcells = g.astype(np.float64).transpose(0, 2, 3, 1).reshape(B * wl.X * wl.Y, C)
    ref = (J.T @ gcells).reshape(B, N, H, W, C)
    assert np.all(np.abs(gf - ref) <= 1e-12 * (scale + np.abs(ref)) + 1e-300)
    # scale bounds the result and is zero exactly where no term arrives
    assert np.all(np.abs(gf) <= scale * (1 + 1e-12))
    assert np.all((terms == 0) == np.all(scale == 0, axis=-1))


@pytest.mark.parametrize("reduce", ["mean", "sum"])
@pytest.mark.parametrize("which", ["tiny", "ragged"])
def test_adjoint_identity_with_forward_oracle(reduce, which):
    inst = (synth.make_workload(synth.config("tiny")) if which == "tiny"
            else small_workload(B=2, N=6, H=7, W=11, C=3, X=9, Y=8, Z=4, seed=9))
    g = _grad(inst, seed=5)
    out, oscale, _ = oracle.run_instance(inst, reduce)
    gf, bscale, _ = _bwd(inst, g, reduce)
    lhs = float(np.sum(out * g.astype(np.float64)))
    rhs = float(np.sum(inst.features.astype(np.float64) * gf))
    bound = float(np.sum(oscale * np.abs(g.astype(np.float64))))
    assert bound > 0
    assert abs(lhs - rhs) <= 1e-11 * bound, (lhs, rhs, bound)


def test_term_counts_add_up_to_forward_taps():
    inst = synth.make_workload(synth.config("tiny"))
    _, _, cnt = oracle.run_instance(inst)
    _, _, terms = _bwd(inst, _grad(inst))
    assert int(terms.sum()) == cnt["taps"] > 0


def test_pixels_no_tap_reaches_are_exactly_zero():
    inst = small_workload(B=1, N=3, H=9, W=13, C=2, X=4, Y=3, Z=2, seed=3)
    gf, scale, terms = _bwd(inst, _grad(inst))
    untouched = terms == 0
    assert untouched.any() and (~untouched).any()
    assert np.all(gf[untouched] == 0.0) and np.all(scale[untouched] == 0.0)


def test_zero_output_gradient_gives_zero():
    inst = small_workload(seed=2)
    wl = inst.wl
    gf, scale, terms = _bwd(inst, np.zeros((wl.B, wl.C, wl.X, wl.Y), np.float32))
    assert np.all(gf == 0.0) and np.all(scale == 0.0) and terms.sum() > 0
