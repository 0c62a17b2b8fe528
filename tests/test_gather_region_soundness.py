"""Soundness of the gather-form backward's candidate regions (CPU).

The gather form of the backward (flashbev_sample_vt_backward_ws) takes the
feature-map pixels a few at a time (a group: g consecutive columns of one
row py, or of rows py and py + 1 (py even) where g is at most 2) and, for
each height, enumerates only the BEV cells inside a region of that
height's plane: five half-planes in float64 (depth above depth_eps; u and v
inside the group's tap support and the image), each loosened by 2^-18 of
the magnitudes of its terms, cut into row intervals over a range of rows
bounded algebraically (each pair of column bounds is linear in the row
index, so it holds on a half-line of rows, widened by one row).  Every
candidate is then re-checked with the forward's float32 recipe, so the
region only has to contain every sample that reaches the group.

This file restates the region in numpy float64 (the kernel's operations in
the kernel's order, none fused) and checks it against the oracle's own
projection pass (Sec. 3.1's mask and the feature coordinates): every valid
sample (b, cell, z, n) whose bilinear taps (Sec. 3.3) touch a pixel of a
group must be a candidate of that group at that height.  The GPU parity
tests then check the compiled kernel end to end.
"""
import numpy as np
import pytest

import oracle
from test_cull_soundness import random_matrices, ring_matrices

F = np.float32
E = 2.0 ** -18


def region_has(m12, zk, i, j, py, nrows, px0, g, grid, img_hw, feat_hw, eps):
    """Whether cell (i, j) is a candidate of the group (rows py .. py+nrows-1,
    columns px0 .. px0+g-1) at height zk for a camera with rows m12 [..., 12]
    (float32); every argument broadcasts."""
    x_min, dx, X, y_min, dy, Y = grid
    img_h, img_w = img_hw
    H, W = feat_hw
    mr = np.asarray(m12, F).astype(np.float64)
    m = [mr[..., t] for t in range(12)]
    x_min_d, dx_d, y_min_d, dy_d = (float(F(v)) for v in (x_min, dx, y_min, dy))
    sx, sy = F(W) / F(img_w), F(H) / F(img_h)
    isx, isy = 1.0 / float(sx), 1.0 / float(sy)
    xmax = abs(x_min_d) + (X + 1.0) * abs(dx_d)
    ymax = abs(y_min_d) + (Y + 1.0) * abs(dy_d)
    shape = np.broadcast(i, j, np.asarray(zk), mr[..., 0], py, px0).shape
    with np.errstate(all="ignore"):
        U0 = np.maximum(0.0, (px0 - 0.5) * isx)
        U1 = np.minimum(float(img_w), ((px0 + g) + 0.5) * isx)
        V0 = np.maximum(0.0, (py - 0.5) * isy)
        V1 = np.minimum(float(img_h), ((py + nrows) + 0.5) * isy)
        support = (U0 < U1) & (V0 < V1)
        zd = np.asarray(zk, F).astype(np.float64)
        Mu0 = (np.abs(m[0]) * xmax + np.abs(m[1]) * ymax) + np.abs(m[3])
        Mv0 = (np.abs(m[4]) * xmax + np.abs(m[5]) * ymax) + np.abs(m[7])
        Md0 = (np.abs(m[8]) * xmax + np.abs(m[9]) * ymax) + np.abs(m[11])
        yc0 = y_min_d + 0.5 * dy_d
        xr0 = x_min_d + 0.5 * dx_d
        xspan = abs(xr0) + abs(dx_d) * X
        # height-free terms of the five planes
        ad, bd = m[8], m[9]
        pab = [(ad, bd)]
        for S, sg, ra, rb in ((U0, 1.0, m[0], m[1]), (U1, -1.0, m[0], m[1]),
                              (V0, 1.0, m[4], m[5]), (V1, -1.0, m[4], m[5])):
            pab.append((sg * (ra - S * ad), sg * (rb - S * bd)))
        tab = []
        for pa, pb in pab:
            beta = pb * dy_d
            kind = np.where(beta > 1e-200, 1, np.where(beta < -1e-200, -1, 0))
            rho = np.where(kind != 0, 1.0 / np.where(kind != 0, beta, 1.0), 0.0)
            Bs = pa * dx_d
            tab.append((pa, pb, rho, np.abs(beta) * Y, kind, np.where(kind != 0, -Bs * rho, Bs)))
        # the height's offsets
        Mu, Mv, Md = Mu0 + np.abs(m[2] * zd), Mv0 + np.abs(m[6] * zd), Md0 + np.abs(m[10] * zd)
        cu, cv, cd = m[2] * zd + m[3], m[6] * zd + m[7], m[10] * zd + m[11]

        def ok(M):
            return (M == 0.0) | (M > 1e-30)
        tame = (Mu < 1e36) & (Mv < 1e36) & (Md < 1e36) & ok(Mu) & ok(Mv) & ok(Md)
        E_ = E
        pc = [cd - float(F(eps)) + E_ * Md,
              (cu - U0 * cd) + E_ * (Mu + U0 * Md),
              -(cu - U1 * cd) + E_ * (Mu + U1 * Md),
              (cv - V0 * cd) + E_ * (Mv + V0 * Md),
              -(cv - V1 * cd) + E_ * (Mv + V1 * Md)]
        gam, T0, TM = [], [], []
        for q in range(5):
            pa, pb, rho, sj, kind, _ = tab[q]
            gq = pc[q] + pb * yc0
            A = pa * xr0 + gq
            Mq = np.abs(pa) * xspan + np.abs(gq)
            gam.append(gq)
            T0.append(np.where(kind != 0, -A * rho, A + sj))
            TM.append(np.where(kind != 0, Mq * np.abs(rho), Mq + sj))
        # the row range
        rlo = np.zeros(shape, np.int64)
        rhi = np.full(shape, X - 1, np.int64)
        none = np.zeros(shape, bool)

        def bound(act, al, be, rbe, mm):
            nonlocal rlo, rhi, none
            tiny = 2.0 ** -40 * mm
            slope = act & (np.abs(be) > tiny)
            b = np.fmin(np.fmax(-al * rbe, -4.0), X + 4.0)
            rlo = np.where(slope & (be > 0), np.maximum(rlo, np.floor(b).astype(np.int64) - 1), rlo)
            rhi = np.where(slope & (be < 0), np.minimum(rhi, np.ceil(b).astype(np.int64) + 1), rhi)
            none |= act & ~slope & (al + np.abs(be) * X < -tiny)
        for pp in range(6):
            for qq in range(6):
                if pp == 5 and qq == 5:
                    continue
                up = True if pp == 5 else tab[pp][4] < 0
                lw = True if qq == 5 else tab[qq][4] > 0
                be = (0.0 if pp == 5 else tab[pp][5]) - (0.0 if qq == 5 else tab[qq][5])
                rbe = np.where(be != 0.0, 1.0 / np.where(be != 0.0, be, 1.0), 0.0)
                t0p, mp = (float(Y), float(Y)) if pp == 5 else (T0[pp], TM[pp])
                t0q, mq = (-1.0, 1.0) if qq == 5 else (T0[qq], TM[qq])
                bound(up & lw, t0p - t0q, be, rbe, mp + mq)
        for q in range(5):
            be = tab[q][5]
            rbe = np.where(be != 0.0, 1.0 / np.where(be != 0.0, be, 1.0), 0.0)
            bound(tab[q][4] == 0, T0[q], be, rbe, TM[q])
        inrows = ~none & (i >= np.maximum(rlo, 0)) & (i <= np.minimum(rhi, X - 1))
        # the row's column interval
        x = x_min_d + (i + 0.5) * dx_d
        lo = np.full(shape, -1.0)
        hi = np.full(shape, float(Y))
        empty = np.zeros(shape, bool)
        for q in range(5):
            pa, _, rho, sj, kind, _ = tab[q]
            v = pa * x + gam[q]
            lo = np.where(kind > 0, np.fmax(lo, -v * rho), lo)
            hi = np.where(kind < 0, np.fmin(hi, -v * rho), hi)
            empty |= (kind == 0) & (v + sj < 0.0)
        lo = np.fmin(lo, float(Y))
        hi = np.fmax(hi, -1.0)
        jlo = np.maximum(0, np.ceil(lo))
        jhi = np.minimum(Y - 1, np.floor(hi))
        region = inrows & ~empty & (jlo <= j) & (j <= jhi)
    return support & np.isfinite(zd) & (region | ~tame)


def check(l2i, z, grid, img_hw, feat_hw, cpws=(1, 3, 8), eps=1e-5):
    """Every (valid sample, group it reaches) pair must be a candidate; returns
    the number of pairs checked."""
    x_min, dx, X, y_min, dy, Y = grid
    B, N = l2i.shape[:2]
    H, W = feat_hw
    mask, xf, yf = oracle.project(l2i, z, feat_hw, img_hw, B, N, X, Y, x_min, dx, y_min, dy, eps)
    b, i, j, k, n = np.nonzero(mask)
    x0 = np.floor(xf[b, i, j, k, n]).astype(np.int64)
    y0 = np.floor(yf[b, i, j, k, n]).astype(np.int64)
    m12 = l2i[b, n, :3, :].reshape(-1, 12)
    zk = np.asarray(z, F)[k]
    pairs = 0
    for cpw in cpws:
        for dyr in (0, 1):
            py = y0 + dyr
            for dxc in (0, 1):
                px = x0 + dxc
                sel = (py >= 0) & (py < H) & (px >= 0) & (px < W)
                if not sel.any():
                    continue
                px0 = (px[sel] // cpw) * cpw
                g = np.minimum(W - px0, cpw)
                R = 2 if cpw <= 2 else 1          # rows per group
                gy = (py[sel] // R) * R           # the group's first row
                nrows = np.minimum(H - gy, R)
                has = region_has(m12[sel], zk[sel], i[sel], j[sel], gy, nrows, px0, g, grid,
                                 img_hw, feat_hw, eps)
                assert has.all(), (cpw, np.argwhere(~has)[:5].ravel(), b[sel][~has][:5],
                                   i[sel][~has][:5], j[sel][~has][:5], k[sel][~has][:5],
                                   n[sel][~has][:5])
                pairs += int(sel.sum())
    return pairs


@pytest.mark.parametrize("seed", range(24))
def test_random_cameras_every_reaching_sample_is_a_candidate(seed):
    rng = np.random.default_rng([8300, seed])
    img_h, img_w = (256, 704) if seed % 2 else (900, 1600)
    stride = (4, 8, 16)[seed % 3]
    B, N, Z = 1, int(rng.integers(1, 7)), int(rng.integers(1, 20))
    half = float(rng.uniform(5.0, 80.0))
    X, Y = int(rng.integers(8, 90)), int(rng.integers(8, 90))
    z = rng.uniform(-30.0, 30.0, Z).astype(np.float32)
    l2i = random_matrices(rng, N, img_h, img_w)[None]
    grid = (-half, 2 * half / X, X, -half, 2 * half / Y, Y)
    check(l2i, z, grid, (img_h, img_w), (img_h // stride, img_w // stride))


def test_ring_rig_at_benchmark_scale():
    """The benchmark's rig over a 200 x 200 grid and Z = 8 from -5 to 3 m."""
    z = ((np.arange(8) + 0.5) - 5.0).astype(np.float32)
    pairs = check(ring_matrices(6, 256, 704)[None], z, (-50.0, 0.5, 200, -50.0, 0.5, 200),
                  (256, 704), (32, 88), cpws=(3,))
    assert pairs > 10000


def test_offset_and_mirrored_grids():
    """A grid far from the origin (large x_min against its pitch) and one
    with negative pitches: the slack bounds and the index form cover both."""
    rng = np.random.default_rng(8301)
    l2i = random_matrices(rng, 4, 256, 704)[None]
    z = np.linspace(-6, 6, 9).astype(np.float32)
    check(l2i, z, (900.0, 0.05, 120, -1000.0, 0.07, 90), (256, 704), (32, 88))
    check(l2i, z, (20.0, -0.4, 100, 15.0, -0.3, 100), (256, 704), (32, 88))


def test_degenerate_and_extreme_rows():
    """Zero rows, a camera looking straight down, one at the grid's height,
    one with entries near float32 overflow, one with a NaN entry, one whose
    u and v rows are scaled to 1e-36 and one whose u and v rows are scaled
    into float32's subnormal range (2e-44: the recipe's rounding there is
    absolute rather than relative).  The last four get no region: every
    cell is a candidate."""
    l2i = np.zeros((1, 7, 4, 4), np.float32)
    l2i[0, 0, 1] = [0, 500, 0, 128]
    l2i[0, 0, 2] = [1, 0, 0, 0]
    l2i[0, 1, 0] = [500, 0, 352, 0]
    l2i[0, 1, 1] = [0, 500, 128, 0]
    l2i[0, 1, 2] = [0, 0, -1, 10]
    l2i[0, 2, :3] = np.array([[352, -500, 0, 0], [128, 0, -500, 0], [1, 0, 0, 0]], np.float32)
    l2i[0, 3, :3] = np.array([[3e37, 1, 0, 0], [0, 2e37, 0, 0], [1, 0, 0, 5]], np.float32)
    l2i[0, 4, :3] = np.array([[352, -500, 0, 0], [128, 0, -500, np.nan], [1, 0, 0, 0]], np.float32)
    l2i[0, 5] = l2i[0, 2]
    l2i[0, 5, :2] *= np.float32(1e-36)
    l2i[0, 6] = l2i[0, 2]
    l2i[0, 6, :2] *= np.float32(2e-44)
    l2i[0, :, 3, 3] = 1
    z = np.array([-5.0, -1.0, 0.0, 2.0], np.float32)
    check(l2i, z, (-30.0, 1.0, 60, -30.0, 1.0, 60), (256, 704), (32, 88))
