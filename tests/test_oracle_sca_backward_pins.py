"""Pins of the FlashSCA backward oracle (gradients with respect to the value
maps, the sampling offsets and the attention logits).

  * torch autograd through BEVFormer's dense path (tests/sca_dense.py:
    grid_sample and softmax in float64), compared on queries whose hit
    decisions and points whose bilinear cell do not hinge on float32 versus
    float64 rounding (the offset gradient jumps where a location crosses a
    pixel);
  * central finite differences of the forward oracle (pinned in
    test_oracle_sca_pins.py) with respect to logits and offsets;
  * the adjoint identity <fwd(V), G> = <V, d value(G)> (the output is linear
    in the value);
  * invariants: the logits' gradient sums to zero over each head (softmax is
    shift invariant); queries no camera sees get zero offset and logit
    gradients.
"""
import numpy as np
import pytest

import oracle
import synth
from sca_dense import dense_sca_grads, robust_queries
from test_oracle_sca_pins import small_sca


def _g(inst, seed=3):
    wl = inst.wl
    return np.random.default_rng(seed).standard_normal((wl.B, wl.Q, wl.C)).astype(np.float32)


def _bwd(inst, g, reduce="mean"):
    return oracle.sca_backward_instance(inst, g, reduce)


def _dense(inst, g, reduce="mean"):
    wl = inst.wl
    return dense_sca_grads(inst.value, inst.lidar2img, inst.z, inst.offsets, inst.logits, g,
                           wl.levels, wl.heads, (wl.img_h, wl.img_w), wl.X, wl.Y, wl.x_min,
                           wl.dx, wl.y_min, wl.dy, wl.depth_eps, reduce)


# float32 (oracle) versus float64 (dense) sampling locations move each
# bilinear weight by a few 1e-5; see DENSE_TOL in test_oracle_sca_pins.py
TOL = 4e-3


@pytest.mark.parametrize("which,reduce", [("small", "mean"), ("small_p8", "sum"),
                                          ("tiny", "mean")])
def test_backward_equals_autograd_of_dense_path(which, reduce):
    inst = {"small": lambda: small_sca(21),
            "small_p8": lambda: small_sca(22, P=8, Z=4, levels=((24, 64), (12, 32))),
            "tiny": lambda: synth.make_sca_workload(synth.sca_config("sca_tiny"))}[which]()
    wl = inst.wl
    g = _g(inst)
    r = _bwd(inst, g, reduce)
    gv, goff, glg, pix, hit = _dense(inst, g, reduce)
    keep = robust_queries(inst.lidar2img, inst.z, wl.X, wl.Y, wl.x_min, wl.dx, wl.y_min, wl.dy,
                          (wl.img_h, wl.img_w))
    assert keep.all(), "choose inputs without boundary anchors"
    # value gradient: continuous in the locations.  A corner whose float64
    # location lies within rounding of a map border can carry a weight of
    # ~1e-5 on one side only; allow 1e-4 pixel of weight times the gradient.
    err = np.abs(r["value"] - gv)
    atol = 1e-4 * float(np.abs(g).max())
    assert np.all(err <= TOL * r["value_scale"] + atol), err.max()
    assert np.count_nonzero(r["value"]) > 100
    # logits gradient: continuous in the locations
    err = np.abs(r["logits"] - glg)
    assert np.all(err <= TOL * r["logits_scale"] + 1e-12), err.max()
    # offsets gradient: skip points whose location lies within 1e-3 pixel of
    # a pixel line in any hit camera (the derivative jumps there)
    frac = pix - np.floor(pix)
    near = (np.minimum(frac, 1.0 - frac) < 1e-3).any(axis=-1)       # [B, N, Q, h, L, P]
    near = (near & hit[:, :, :, None, None, None]).any(axis=1)      # [B, Q, h, L, P]
    ok = ~near
    assert ok.mean() > 0.95
    err = np.abs(r["offsets"] - goff)[ok]
    assert np.all(err <= TOL * r["offsets_scale"][ok] + 1e-12), err.max()
    assert np.count_nonzero(r["offsets"]) > 100


def _objective(inst, g):
    out, _, _, _ = oracle.sca_instance(inst)
    return float(np.sum(out * g.astype(np.float64)))


def test_logits_gradient_is_a_finite_difference():
    inst = small_sca(23, B=1, X=5, Y=4)
    g = _g(inst)
    r = _bwd(inst, g)
    rng = np.random.default_rng(1)
    idx = [tuple(int(rng.integers(0, n)) for n in inst.logits.shape) for _ in range(40)]
    h = 2.0 ** -8
    checked = 0
    for ix in idx:
        base = float(inst.logits[ix])
        inst.logits[ix] = base + h
        fp = _objective(inst, g)
        inst.logits[ix] = base - h
        fm = _objective(inst, g)
        inst.logits[ix] = base
        fd = (fp - fm) / (2 * h)
        # second-order error of the softmax: well below the gradient scale
        assert abs(fd - r["logits"][ix]) <= 1e-3 * r["logits_scale"][ix] + 1e-9, (ix, fd, r["logits"][ix])
        checked += r["logits"][ix] != 0
    assert checked > 10


def test_offsets_gradient_is_a_finite_difference():
    inst = small_sca(24, B=1, X=5, Y=4)
    wl = inst.wl
    g = _g(inst)
    r = _bwd(inst, g)
    _, _, _, pix, hit = _dense(inst, g)
    rng = np.random.default_rng(2)
    h = 2.0 ** -6
    checked = 0
    for _ in range(60):
        ix = tuple(int(rng.integers(0, n)) for n in inst.offsets.shape[:-1])
        comp = int(rng.integers(0, 2))
        b, q, m, l, k = ix
        # the bilinear sample is linear in the location inside one pixel cell:
        # keep the step inside it in every hit camera
        locs = pix[b, :, q, m, l, k, comp][hit[b, :, q]]
        fr = locs - np.floor(locs)
        if len(locs) and np.min(np.minimum(fr, 1.0 - fr)) < 4 * h:
            continue
        base = float(inst.offsets[ix + (comp,)])
        inst.offsets[ix + (comp,)] = base + h
        fp = _objective(inst, g)
        inst.offsets[ix + (comp,)] = base - h
        fm = _objective(inst, g)
        inst.offsets[ix + (comp,)] = base
        fd = (fp - fm) / (2 * h)
        sc = r["offsets_scale"][ix + (comp,)]
        assert abs(fd - r["offsets"][ix + (comp,)]) <= 2e-3 * sc + 1e-9, (ix, comp, fd, r["offsets"][ix + (comp,)])
        checked += r["offsets"][ix + (comp,)] != 0
    assert checked > 10


@pytest.mark.parametrize("reduce", ["mean", "sum"])
def test_value_gradient_adjoint_identity(reduce):
    inst = small_sca(25)
    g = _g(inst)
    out, oscale, _, _ = oracle.sca_instance(inst, reduce)
    r = _bwd(inst, g, reduce)
    lhs = float(np.sum(out * g.astype(np.float64)))
    rhs = float(np.sum(inst.value.astype(np.float64) * r["value"]))
    bound = float(np.sum(oscale * np.abs(g)))
    assert abs(lhs - rhs) <= 1e-11 * bound, (lhs, rhs)


def test_invariants():
    inst = small_sca(26)
    wl = inst.wl
    g = _g(inst)
    r = _bwd(inst, g)
    # softmax shift invariance: the logits' gradient sums to zero per head
    s = r["logits"].reshape(wl.B, wl.Q, wl.heads, -1).sum(axis=-1)
    sc = r["logits_scale"].reshape(wl.B, wl.Q, wl.heads, -1).sum(axis=-1)
    assert np.all(np.abs(s) <= 1e-12 * sc + 1e-300)
    # queries no camera sees: zero offset and logit gradients, no terms
    _, _, _, hit = oracle.sca_reference_points(inst.lidar2img, inst.z, wl.B, wl.N,
                                               (wl.img_h, wl.img_w), wl.X, wl.Y, wl.x_min,
                                               wl.dx, wl.y_min, wl.dy)
    none = ~hit.any(axis=-1)
    assert none.any()
    assert np.all(r["offsets"][none] == 0) and np.all(r["logits"][none] == 0)
    assert np.all(r["point_terms"][none] == 0)
    # value terms: every in-range corner of every hit camera lands somewhere
    assert int(r["value_terms"].sum()) == int(r["point_terms"].sum())
