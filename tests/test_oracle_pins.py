"""Pins of the oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with itself: each checks it against
an independent statement -- a hand derivation (tests/golden), brute-force
search, an analytic scene, a closed form, an invariant of the operator, or a
library routine applied to a special case.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth
from synth.configs import C1, C2, C3, C4, C5

from conftest import latent_maps, ulp_diff

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def decode(word):
    w = np.asarray(word).astype(np.int64) & 0xFFFFFFFF
    x0 = (w & 0xFFF) - 1
    y0 = ((w >> 12) & 0xFFF) - 1
    mask = (w >> 24) & 0xF
    return x0, y0, mask


def taps_of(word, W):
    """Raster indices of the taps set in one word, ascending k."""
    x0, y0, mask = decode(word)
    out = []
    for k in range(4):
        if int(mask) >> k & 1:
            out.append(int((y0 + (k >> 1)) * W + (x0 + (k & 1))))
    return out


def ortho_cams(R, t, f, cs):
    n = len(cs)
    return {"model": np.ones(n, np.int32), "R": np.array([R] * n, np.float32),
            "t": np.array([t] * n, np.float32), "fx": np.full(n, f, np.float32),
            "fy": np.full(n, f, np.float32), "cx": np.array([c[0] for c in cs], np.float32),
            "cy": np.array([c[1] for c in cs], np.float32)}


def batch(c, B=1):
    return {k: np.ascontiguousarray(np.broadcast_to(v, (B,) + v.shape)) for k, v in c.items()}


# ---------------------------------------------------------------------------
# O1 downsample
# ---------------------------------------------------------------------------

def test_downsample_constant_block_exact():
    hi = np.full((2, 16, 24, 3), 0.3, np.float32)
    hi[..., 1] = -1.7
    lo = oracle.downsample(hi, 8)
    assert lo.shape == (2, 2, 3, 3)
    assert np.all(lo[..., 0] == np.float32(0.3)) and np.all(lo[..., 1] == np.float32(-1.7))


def test_downsample_linear_ramp_is_block_centre():
    f = 4
    y, x = np.meshgrid(np.arange(32) + 0.5, np.arange(32) + 0.5, indexing="ij")
    hi = np.stack([0.01 * x, -0.02 * y + 0.5, 0.003 * x + 0.007 * y], -1).astype(np.float32)[None]
    lo = oracle.downsample(hi, f)
    cy, cx = np.meshgrid(np.arange(8) * f + f / 2, np.arange(8) * f + f / 2, indexing="ij")
    want = np.stack([0.01 * cx, -0.02 * cy + 0.5, 0.003 * cx + 0.007 * cy], -1)
    np.testing.assert_allclose(lo[0], want, rtol=0, atol=2e-7)


def test_downsample_majority_rule_and_foreground_mean():
    f = 4
    hi = np.full((1, 4, 12, 3), np.nan, np.float32)
    vals = np.arange(16, dtype=np.float32).reshape(4, 4) + 1
    # block 0: exactly half foreground -> kept, mean over foreground only
    b0 = np.full((4, 4), np.nan, np.float32)
    b0.flat[:8] = vals.flat[:8]
    # block 1: one short of half -> background
    b1 = np.full((4, 4), np.nan, np.float32)
    b1.flat[:7] = vals.flat[:7]
    # block 2: a single non-finite component makes a sample background
    b2 = vals.copy()
    for k, blk in enumerate((b0, b1, b2)):
        for c in range(3):
            hi[0, :, 4 * k:4 * k + 4, c] = blk
    hi[0, 0, 8, 2] = np.inf
    lo = oracle.downsample(hi, f)
    assert lo[0, 0, 0, 0] == np.float32(np.mean(vals.flat[:8]))
    assert np.isnan(lo[0, 0, 1]).all()
    fg = np.ones((4, 4), bool)
    fg[0, 0] = False
    assert lo[0, 0, 2, 0] == np.float32(vals[fg].astype(np.float64).mean())


def test_downsample_matches_numpy_masked_mean(maps):
    w = synth.shrink(C2)
    hi = synth.render_position_maps(w)[0, :2]
    f = w.factor
    lo = oracle.downsample(hi, f)
    M, Hr, Wr, _ = hi.shape
    blk = hi.reshape(M, Hr // f, f, Wr // f, f, 3).transpose(0, 1, 3, 2, 4, 5).reshape(M, Hr // f, Wr // f, f * f, 3)
    fg = np.isfinite(blk).all(-1)
    n = fg.sum(-1)
    s = np.where(fg[..., None], blk.astype(np.float64), 0.0).sum(-2)
    want = (s / np.maximum(n, 1)[..., None]).astype(np.float32)
    want[2 * n < f * f] = np.nan
    np.testing.assert_array_equal(np.isnan(lo), np.isnan(want))
    fin = np.isfinite(want)
    assert ulp_diff(lo[fin], want[fin]).max() <= 1


# ---------------------------------------------------------------------------
# O2 bbox / tolerance
# ---------------------------------------------------------------------------

def test_bbox_matches_numpy_and_hand_tolerance(maps):
    P = maps("torus_6v_96_b4")
    bb = oracle.bbox(P, 0.01)
    for b in range(P.shape[0]):
        q = P[b].reshape(-1, 3)
        q = q[np.isfinite(q).all(1)]
        np.testing.assert_array_equal(bb[b, :3], q.min(0))
        np.testing.assert_array_equal(bb[b, 3:6], q.max(0))
    # hand example: two points (0,0,0) and (3,4,12): diagonal 13, 1% -> 0.13, squared 0.0169
    P2 = np.full((2, 1, 2, 2, 3), np.nan, np.float32)
    P2[0, 0, 0, 0] = (0, 0, 0)
    P2[0, 0, 1, 1] = (3, 4, 12)
    bb2 = oracle.bbox(P2, 0.01)
    assert abs(float(bb2[0, 6]) - 0.0169) <= 2 * np.spacing(np.float32(0.0169))
    assert np.all(bb2[1] == 0)          # no foreground: empty box, zero tolerance


# ---------------------------------------------------------------------------
# O3 correspondence
# ---------------------------------------------------------------------------

def test_golden_toy_plane_shift():
    g = json.load(open(os.path.join(GOLDEN, "toy_plane_shift.json")))
    H, W, h = g["H"], g["W"], g["pitch"]
    cam = g["cameras"]
    cams = batch(ortho_cams(cam["R"], cam["t"], cam["f"], cam["c"]))
    pos = np.zeros((1, 2, H, W, 3), np.float32)
    for v, (cx, cy) in enumerate(cam["c"]):
        for j in range(H):
            for i in range(W):
                pos[0, v, j, i] = ((i + 0.5 - cx) * h, -(j + 0.5 - cy) * h, 0.0)
    bb = oracle.bbox(pos, g["tol_frac"])
    for e in g["expect"]:
        K = e["K"]
        corr, wts, nvis = oracle.build(pos, cams, [0], K, bb)
        i, j = e["pixel"]
        assert int(corr[0, 0, j, i, 0]) == e["word"], e
        np.testing.assert_array_equal(wts[0, 0, j, i, 0], np.array(e["weights"][:K]))
        assert nvis[0, 0, j, i] == 1


def _bruteforce_valid(P, Q, tol2):
    """Exhaustive in-tolerance search: every foreground source sample within
    tol of P (float32 squared distance)."""
    d = (Q - P).astype(np.float32)
    d2 = (d[..., 0] * d[..., 0] + d[..., 1] * d[..., 1]) + d[..., 2] * d[..., 2]
    ok = np.isfinite(Q).all(-1) & (d2 <= np.float32(tol2))
    return np.flatnonzero(ok), d2.ravel()


# the tiny workload's rig, and the same sphere seen from elevated cameras
# (non-symmetric rotations, so a transposed rotation cannot go unnoticed)
C1_ELEV = synth.shrink(C1, elevations_deg=(30.0, -20.0, 10.0, 45.0),
                       azimuths_deg=(0.0, 80.0, 200.0, 290.0))


def _rig_maps(w):
    if w is C1:
        from conftest import latent_maps
        return latent_maps(C1.name)
    return synth.raycast_radial(w.displacement, synth.sphere_params(w, 0), synth.cameras(w),
                                w.H, w.W)[None]


@pytest.mark.parametrize("rig", ["flat", "elevated"])
@pytest.mark.parametrize("anchors", [[0], [1], [2], [3], [0, 2], [1, 3, 0]])
@pytest.mark.parametrize("K", [1, 2, 4])
def test_bruteforce_exhaustive_search_tiny_views(rig, anchors, K):
    """Tiny sphere: orthographic maps ray-cast through pixel centres and a
    tolerance below one pixel pitch, so the footprint search must find exactly
    the in-tolerance samples an exhaustive search over the whole anchor view
    finds; K=1 must pick the exhaustive nearest one."""
    w = C1 if rig == "flat" else C1_ELEV
    P = _rig_maps(w)
    cams = synth.batch_cameras(w)
    bb = oracle.bbox(P, C1.tol_frac)
    tol2 = bb[0, 6]
    pitch = 2 * C1.ortho_half_extent / C1.W
    assert math.sqrt(tol2) < 0.6 * pitch     # the premise of this pin
    anchors = sorted(anchors)
    corr, wts, nvis = oracle.build(P, cams, anchors, K, bb)
    targets = [v for v in range(C1.N) if v not in anchors]
    checked = singles = 0
    for ti, v in enumerate(targets):
        for j in range(C1.H):
            for i in range(C1.W):
                Pp = P[0, v, j, i]
                nv_expect = 0
                for s, u in enumerate(anchors):
                    word = int(corr[0, ti, j, i, s])
                    if not np.isfinite(Pp).all():
                        assert word == 0
                        continue
                    valid, d2 = _bruteforce_valid(Pp, P[0, u].reshape(-1, 3), tol2)
                    got = taps_of(word, C1.W) if word else []
                    if len(valid) == 0:
                        assert word == 0
                        continue
                    nv_expect += 1
                    if K == 1:
                        best = valid[np.argmin(d2[valid])]
                        assert got == [int(best)]
                    else:
                        # every in-tolerance sample is selected unless more than K
                        assert len(valid) <= K
                        if len(valid) == 1:
                            assert got == [int(valid[0])]
                            singles += 1
                        else:
                            # zero-area taps are dropped from the mask; what stays is a subset
                            assert set(got) <= set(valid.tolist()) and len(got) >= 1
                    checked += 1
                assert nvis[0, ti, j, i] == nv_expect
    assert checked > 100
    assert K == 1 or singles > 100


def test_identity_duplicate_view(maps):
    """A target identical to the anchor (same camera, same map) maps every
    foreground token onto itself with weight 1, for K=1 and K=4."""
    P = maps(C1.name)[:, :1]
    P2 = np.concatenate([P, P], axis=1)
    c = synth.cameras(C1)
    cams = batch({k: np.concatenate([v[:1], v[:1]]) for k, v in c.items()})
    bb = oracle.bbox(P2, C1.tol_frac)
    fg = np.isfinite(P[0, 0]).all(-1)
    for K in (1, 4):
        corr, wts, nvis = oracle.build(P2, cams, [0], K, bb)
        for j in range(C1.H):
            for i in range(C1.W):
                word = int(corr[0, 0, j, i, 0])
                if not fg[j, i]:
                    assert word == 0
                    continue
                assert taps_of(word, C1.W) == [j * C1.W + i]
                assert wts[0, 0, j, i, 0, 0] == 1.0


def test_analytic_occlusion_two_planes():
    """Back plane z=0 ([-1,1]^2) behind a square z=0.5 ([-0.3,0.3]^2).
    Target: orthographic, looking down -z.  Anchor: orthographic, tilted
    30 deg about +y.  A back-plane point (x, y, 0) is hidden from the anchor
    exactly when x + 0.5*tan(30 deg) lies in [-0.3, 0.3] and |y| <= 0.3."""
    quads = [(-1.0, 1.0, 0.0), (-0.3, 0.3, 0.5)]
    V, T = [], []
    for lo, hi, z in quads:
        b = len(V)
        V += [(lo, lo, z), (hi, lo, z), (hi, hi, z), (lo, hi, z)]
        T += [(b, b + 1, b + 2), (b, b + 2, b + 3)]
    V = np.array(V, np.float64)
    T = np.array(T, np.int32)
    H = W = 40
    he = 1.15
    th = math.radians(30)
    cams = {"model": np.ones(2, np.int32), "R": np.zeros((2, 3, 3), np.float32),
            "t": np.zeros((2, 3), np.float32), "fx": np.full(2, W / (2 * he), np.float32),
            "fy": np.full(2, H / (2 * he), np.float32), "cx": np.full(2, W / 2, np.float32),
            "cy": np.full(2, H / 2, np.float32)}
    for v, ang in enumerate((0.0, th)):
        d = np.array([math.sin(ang), 0.0, math.cos(ang)])      # towards the camera
        fwd = -d
        right = np.cross(fwd, [0, 1, 0]); right /= np.linalg.norm(right)
        down = np.cross(fwd, right)
        R = np.stack([right, down, fwd])
        cams["R"][v] = R
        cams["t"][v] = -R @ (3.0 * d)
    out = np.empty((2, H, W, 3), np.float32)
    import ctypes
    L = synth.lib()
    cr = synth.cams_for_renderer(cams)
    rc = L.synth_render_mesh(V.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), V.shape[0],
                             T.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), T.shape[0],
                             cr.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), 2, H, W,
                             out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), 1)
    assert rc == 0
    pos = out[None]
    bb = oracle.bbox(pos, 0.05)
    corr, wts, nvis = oracle.build(pos, batch(cams), [1], 4, bb)
    pitch = 2 * he / W
    margin = 1.5 * pitch
    n_vis_checked = n_occ_checked = 0
    for j in range(H):
        for i in range(W):
            P = pos[0, 0, j, i]
            if not np.isfinite(P).all():
                assert corr[0, 0, j, i, 0] == 0
                continue
            x, y, z = (float(c) for c in P)
            if z > 0.25:      # the front square: nothing occludes it
                if abs(x) < 0.3 - margin and abs(y) < 0.3 - margin:
                    assert nvis[0, 0, j, i] == 1
                    n_vis_checked += 1
                continue
            xs = x + 0.5 * math.tan(th)
            occluded = abs(xs) <= 0.3 and abs(y) <= 0.3
            near_edge = (abs(abs(xs) - 0.3) < margin or abs(abs(y) - 0.3) < margin
                         or abs(x) > 1 - margin or abs(y) > 1 - margin)
            if near_edge:
                continue
            if occluded:
                assert nvis[0, 0, j, i] == 0, (i, j, x, y)
                n_occ_checked += 1
            else:
                assert nvis[0, 0, j, i] == 1, (i, j, x, y)
                n_vis_checked += 1
    assert n_occ_checked > 20 and n_vis_checked > 200


def _project64(P, cam, v):
    R = cam["R"][v].astype(np.float64)
    t = cam["t"][v].astype(np.float64)
    xc = R @ P.astype(np.float64) + t
    if cam["model"][v] == 0:
        return cam["fx"][v] * xc[0] / xc[2] + cam["cx"][v], cam["fy"][v] * xc[1] / xc[2] + cam["cy"][v]
    return cam["fx"][v] * xc[0] + cam["cx"][v], cam["fy"][v] * xc[1] + cam["cy"][v]


def _overlap(a0, a1, b0, b1):
    return max(0.0, min(a1, b1) - max(a0, b0))


@pytest.mark.parametrize("name", [C2.name, C4.name])
def test_weights_are_pixel_overlap_areas(maps, name):
    """Each kept tap's weight, before the division by n_vis, is the overlap of
    a unit square centred on the projection with the tap's pixel, renormalised
    over the kept taps (computed here by interval intersection in double)."""
    w = synth.CONFIGS[name]
    P = maps(name)
    cams = synth.cameras(w)
    bcams = synth.batch_cameras(w)
    A = oracle.anchors(w.N, w.a, 0)
    bb = oracle.bbox(P, w.tol_frac)
    corr, wts, nvis = oracle.build(P, bcams, A, 4, bb)
    targets = [v for v in range(w.N) if v not in A]
    rs = np.random.default_rng(0)
    idx = np.argwhere(nvis[0] > 0)
    checked = 0
    for ti, j, i in idx[rs.choice(len(idx), size=min(400, len(idx)), replace=False)]:
        v = targets[ti]
        for s, u in enumerate(A):
            word = int(corr[0, ti, j, i, s])
            if not word:
                continue
            px, py = _project64(P[0, v, j, i], cams, u)
            areas = []
            for q in taps_of(word, w.W):
                qy, qx = divmod(q, w.W)
                areas.append(_overlap(px - 0.5, px + 0.5, qx, qx + 1) * _overlap(py - 0.5, py + 0.5, qy, qy + 1))
            S = sum(areas)
            got = wts[0, ti, j, i, s, :len(areas)] * nvis[0, ti, j, i]
            # every kept tap's pixel centre lies within one pixel of the projection
            for q in taps_of(word, w.W):
                qy, qx = divmod(q, w.W)
                assert abs(qx + 0.5 - px) <= 1 + 1e-4 and abs(qy + 0.5 - py) <= 1 + 1e-4
            if len(areas) > 1 or S > 1e-9:
                assert S > 1e-9
                np.testing.assert_allclose(got, np.array(areas) / S, rtol=0, atol=2e-5)
            checked += 1
    assert checked > 50


@pytest.mark.parametrize("name", [C1.name, C2.name, C4.name, C3.name])
def test_operator_invariants(maps, name):
    w = synth.CONFIGS[name]
    P = maps(name)
    bcams = synth.batch_cameras(w)
    bb = oracle.bbox(P, w.tol_frac)
    for c in range(2):
        A = list(w.fixed_anchors) if w.fixed_anchors else oracle.anchors(w.N, w.a, c)
        for K in (1, w.K):
            corr, wts, nvis = oracle.build(P, bcams, A, K, bb)
            targets = [v for v in range(w.N) if v not in A]
            x0, y0, mask = decode(corr)
            nz = corr != 0
            assert np.all((nvis > 0) == nz.any(-1))
            assert np.all(nvis == nz.sum(-1))
            # row-stochastic on visible rows, zero rows elsewhere
            rs = wts.sum(axis=(-1, -2))
            np.testing.assert_allclose(rs[nvis > 0], 1.0, rtol=0, atol=1e-12)
            assert np.all(rs[nvis == 0] == 0)
            assert np.all(wts >= 0)
            # popcount(mask) taps carry positive weight, no more than K
            pc = np.vectorize(lambda m: bin(int(m)).count("1"))(mask)
            assert np.all(pc <= K)
            for k in range(K):
                assert np.all((wts[..., k] > 0) == (pc > k))
            assert np.all(corr[~nz] == 0)
            # taps on the grid
            for k in range(4):
                on = nz & ((mask >> k) & 1).astype(bool)
                xx = x0 + (k & 1)
                yy = y0 + (k >> 1)
                assert np.all((xx[on] >= 0) & (xx[on] < w.W) & (yy[on] >= 0) & (yy[on] < w.H))
            # background targets are empty
            bg = ~np.isfinite(P[:, targets]).all(-1)
            assert np.all(nvis[bg] == 0)


def test_all_views_anchors_gives_empty_operator(maps):
    P = maps(C1.name)
    corr, wts, nvis = oracle.build(P, synth.batch_cameras(C1), [0, 1, 2, 3], 4, oracle.bbox(P))
    assert corr.shape[1] == 0 and wts.size == 0


def test_two_identical_anchors_split_weight(maps):
    """Multi-anchor aggregation: two anchors that see a token identically
    contribute half each (the normalised sum of their transports)."""
    P = maps(C1.name)
    P3 = np.concatenate([P[:, :1], P[:, :1], P[:, 1:2]], axis=1)
    c = synth.cameras(C1)
    cams = batch({k: np.concatenate([v[:1], v[:1], v[1:2]]) for k, v in c.items()})
    bb = oracle.bbox(P3, C1.tol_frac)
    corr, wts, nvis = oracle.build(P3, cams, [0, 1], 1, bb)
    vis = nvis[0, 0] > 0
    assert vis.sum() > 50
    assert np.all(nvis[0, 0][vis] == 2)
    np.testing.assert_array_equal(corr[0, 0, ..., 0][vis], corr[0, 0, ..., 1][vis])
    assert np.all(wts[0, 0][vis][:, :, 0] == 0.5)


# ---------------------------------------------------------------------------
# O4 transport (Eq. 1)
# ---------------------------------------------------------------------------

def _transport_case(name, dtype=None, seed=0, c=0, K=None):
    w = synth.CONFIGS[name]
    from conftest import latent_maps
    P = latent_maps(name)
    B = P.shape[0]
    A = list(w.fixed_anchors) if w.fixed_anchors else oracle.anchors(w.N, w.a, c)
    K = w.K if K is None else K
    corr, wts, nvis = oracle.build(P, synth.batch_cameras(w), A, K, oracle.bbox(P, w.tol_frac))
    dtype = dtype or w.dtype
    rs = np.random.default_rng(seed)
    prev = rs.standard_normal((B, w.N, w.H, w.W, w.C)).astype(np.float32)
    new = prev[:, A] + 0.1 * rs.standard_normal((B, len(A), w.H, w.W, w.C)).astype(np.float32)
    return w, A, corr, wts, nvis, synth.storage(prev, dtype), synth.storage(new, dtype), dtype


@pytest.mark.parametrize("name,dtype", [(C1.name, "f32"), (C2.name, "f32"), (C4.name, "bf16")])
def test_transport_zero_delta_is_bit_copy(name, dtype):
    w, A, corr, wts, nvis, prev, new, dtype = _transport_case(name, dtype)
    same = prev[:, A].copy()
    exact, state = oracle.transport(prev, same, corr, wts, A, dtype)
    np.testing.assert_array_equal(state, prev)


@pytest.mark.parametrize("name", [C2.name, C4.name])
def test_transport_dense_matrix_form(name):
    """Eq. 1 as an explicit sparse matrix: x0(v) = x0_prev(v) + G_{A->v} @ Delta,
    with G assembled densely from the decoded taps and applied by matmul."""
    w, A, corr, wts, nvis, prev, new, dtype = _transport_case(name)
    exact, state = oracle.transport(prev, new, corr, wts, A, dtype)
    pv = synth.values(prev, dtype).astype(np.float64)
    nv = synth.values(new, dtype).astype(np.float64)
    HW = w.H * w.W
    targets = [v for v in range(w.N) if v not in A]
    for b in range(w.B):
        delta = (nv[b] - pv[b, A]).reshape(len(A) * HW, w.C)   # stacked anchor increments
        for ti, v in enumerate(targets):
            G = np.zeros((HW, len(A) * HW))
            cw = corr[b, ti].reshape(HW, len(A))
            ww = wts[b, ti].reshape(HW, len(A), -1)
            for p in range(HW):
                for s in range(len(A)):
                    for jj, q in enumerate(taps_of(int(cw[p, s]), w.W) if cw[p, s] else []):
                        G[p, s * HW + q] += ww[p, s, jj]
            want = pv[b, v].reshape(HW, w.C) + G @ delta
            np.testing.assert_allclose(exact[b, v].reshape(HW, w.C), want, rtol=0, atol=1e-12)
        for s, u in enumerate(A):
            np.testing.assert_array_equal(state[b, u], new[b, s])


def test_transport_constant_delta_and_convexity():
    name = C2.name
    w, A, corr, wts, nvis, prev, new, dtype = _transport_case(name)
    # values on a coarse grid so prev + 0.25 is exact in float32
    rs = np.random.default_rng(3)
    prev = (rs.integers(-64, 64, size=prev.shape) / 64.0).astype(np.float32)
    new = prev[:, A] + np.float32(0.25)
    exact, state = oracle.transport(prev, new, corr, wts, A, "f32")
    targets = [v for v in range(w.N) if v not in A]
    vis = nvis > 0
    for ti, v in enumerate(targets):
        np.testing.assert_array_equal(state[:, v][vis[:, ti]], prev[:, v][vis[:, ti]] + np.float32(0.25))
        np.testing.assert_array_equal(state[:, v][~vis[:, ti]], prev[:, v][~vis[:, ti]])
    # convex hull: a random increment lands inside [min, max] of its taps
    w, A, corr, wts, nvis, prev, new, dtype = _transport_case(name, seed=5)
    exact, state = oracle.transport(prev, new, corr, wts, A, "f32")
    delta = new.astype(np.float64) - prev[:, A]
    HW = w.H * w.W
    for ti, v in enumerate(targets):
        inc = (exact[0, v] - prev[0, v]).reshape(HW, w.C)
        cw = corr[0, ti].reshape(HW, len(A))
        for p in np.flatnonzero(nvis[0, ti].ravel() > 0)[:300]:
            vals = [delta[0, s].reshape(HW, w.C)[q] for s in range(len(A)) if cw[p, s]
                    for q in taps_of(int(cw[p, s]), w.W)]
            vals = np.array(vals)
            assert np.all(inc[p] >= vals.min(0) - 1e-12) and np.all(inc[p] <= vals.max(0) + 1e-12)


def test_transport_identity_copies_delta(maps):
    P = maps(C1.name)[:, :1]
    P2 = np.concatenate([P, P], axis=1)
    c = synth.cameras(C1)
    cams = batch({k: np.concatenate([v[:1], v[:1]]) for k, v in c.items()})
    corr, wts, nvis = oracle.build(P2, cams, [0], 4, oracle.bbox(P2, C1.tol_frac))
    rs = np.random.default_rng(1)
    x = rs.standard_normal((1, 1, 32, 32, 4)).astype(np.float32)
    prev = np.concatenate([x, x], axis=1)
    new = x + 0.1 * rs.standard_normal(x.shape).astype(np.float32)
    exact, state = oracle.transport(prev, new, corr, wts, [0], "f32")
    fg = np.isfinite(P[0, 0]).all(-1)
    np.testing.assert_array_equal(state[0, 1][fg], new[0, 0][fg])
    np.testing.assert_array_equal(state[0, 1][~fg], prev[0, 1][~fg])


def test_transport_all_anchors_is_copy():
    rs = np.random.default_rng(2)
    prev = synth.storage(rs.standard_normal((2, 3, 5, 7, 4)).astype(np.float32), "bf16")
    new = synth.storage(rs.standard_normal((2, 3, 5, 7, 4)).astype(np.float32), "bf16")
    corr = np.zeros((2, 0, 5, 7, 3), np.int32)
    wts = np.zeros((2, 0, 5, 7, 3, 4))
    _, state = oracle.transport(prev, new, corr, wts, [0, 1, 2], "bf16")
    np.testing.assert_array_equal(state, new)


def test_bf16_rounding_is_nearest_even():
    # values exactly between two bf16 neighbours go to the even one
    one = 1.0
    ulp = 2.0 ** -7
    x = np.array([one + ulp / 2, one + 1.5 * ulp, -(one + ulp / 2), one + ulp / 2 + 1e-12, 3.0e38, 0.0, -0.0])
    got = oracle.store(x, "bf16")
    want = np.array([0x3F80, 0x3F82, 0xBF80, 0x3F81, 0x7F62, 0x0000, 0x8000], np.uint16)
    np.testing.assert_array_equal(got, want)


# ---------------------------------------------------------------------------
# O5 reconstruction
# ---------------------------------------------------------------------------

def test_alpha_bar_matches_log_sum():
    betas = np.linspace(1e-4, 0.02, 1000)
    cum = np.exp(np.cumsum(np.log1p(-betas)))
    for t in (0, 1, 32, 500, 760, 800, 999):
        assert abs(oracle.alpha_bar(t) - cum[t]) <= 1e-12 * cum[t] + 1e-18
    assert oracle.alpha_bar(-1) == 1.0
    assert abs(oracle.alpha_bar(999) - 4.0358e-5) < 1e-8      # the DDPM linear schedule's end


def test_ddim_timesteps_trailing():
    assert oracle.ddim_timesteps(10) == [999, 899, 799, 699, 599, 499, 399, 299, 199, 99, -1]
    ts = oracle.ddim_timesteps(30)
    assert ts[0] == 999 and ts[1] == 966 and ts[-2] == 32 and ts[-1] == -1
    assert all(a > b for a, b in zip(ts, ts[1:]))


@pytest.mark.parametrize("t,tn", [(800, 760), (999, 966), (32, -1), (100, 50)])
def test_ddim_closed_forms_round_trip(t, tn):
    rs = np.random.default_rng(t)
    x0 = rs.standard_normal(4096).astype(np.float32)
    eps = rs.standard_normal(4096).astype(np.float32)
    ab, abn = oracle.alpha_bar(t), oracle.alpha_bar(tn)
    xt64 = math.sqrt(ab) * x0.astype(np.float64) + math.sqrt(1 - ab) * eps.astype(np.float64)
    xt = xt64.astype(np.float32)
    err_in = np.abs(xt.astype(np.float64) - xt64)           # storage rounding of x_t
    xn, e = oracle.reconstruct(xt, x0, "f32", "ddim", t, tn, pred="eps")
    bound = err_in / math.sqrt(1 - ab) + 1e-12
    assert np.all(np.abs(e - eps) <= bound)
    want = math.sqrt(abn) * x0.astype(np.float64) + math.sqrt(1 - abn) * eps.astype(np.float64)
    assert np.all(np.abs(xn - want) <= math.sqrt(1 - abn) * bound + 1e-12)
    _, v = oracle.reconstruct(xt, x0, "f32", "ddim", t, tn, pred="v")
    vwant = math.sqrt(ab) * eps.astype(np.float64) - math.sqrt(1 - ab) * x0.astype(np.float64)
    assert np.all(np.abs(v - vwant) <= math.sqrt(ab) * bound + 1e-12)
    if tn == -1:
        np.testing.assert_array_equal(xn, x0.astype(np.float64))


@pytest.mark.parametrize("s,sn", [(1.0, 29 / 30), (0.5, 0.48), (0.04, 0.0), (0.7, 0.2)])
def test_flow_euler_closed_forms(s, sn):
    rs = np.random.default_rng(int(s * 100))
    x0 = rs.standard_normal(4096).astype(np.float32)
    eps = rs.standard_normal(4096).astype(np.float32)
    xt64 = (1 - s) * x0.astype(np.float64) + s * eps.astype(np.float64)
    xt = xt64.astype(np.float32)
    bound = np.abs(xt - xt64) / s + 1e-12
    xn, vel = oracle.reconstruct(xt, x0, "f32", "flow", s, sn, pred="vel")
    assert np.all(np.abs(vel - (eps.astype(np.float64) - x0)) <= bound)
    # along a straight path the Euler step is exact
    want = (1 - sn) * x0.astype(np.float64) + sn * eps.astype(np.float64)
    assert np.all(np.abs(xn - want) <= np.abs(xt - xt64) + (s - sn) * bound + 1e-12)


def test_reconstruct_rejects_bad_arguments():
    x = np.zeros(4, np.float32)
    with pytest.raises(ValueError):
        oracle.reconstruct(x, x, "f32", "flow", 0.0, 0.0)
    with pytest.raises(ValueError):
        oracle.reconstruct(x, x, "f32", "ddim", 500, 600)
    with pytest.raises(ValueError):
        oracle.reconstruct(x, x, "f32", "ddim", 500, 400, pred="vel")


# ---------------------------------------------------------------------------
# O6 schedule, O7 trajectory
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("N,a", [(4, 1), (6, 2), (10, 3), (12, 4), (6, 6), (7, 3), (5, 2)])
def test_anchor_rotation_returns_every_view(N, a):
    """Every view is an anchor in every window of ceil(N/a) consecutive
    cached steps (Sec. 3.2, batch-sliced anchor forward)."""
    win = math.ceil(N / a)
    sets = [oracle.anchors(N, a, c) for c in range(3 * N)]
    for A in sets:
        assert len(set(A)) == a and A == sorted(A) and all(0 <= x < N for x in A)
    for c0 in range(len(sets) - win + 1):
        seen = set().union(*map(set, sets[c0:c0 + win]))
        assert seen == set(range(N)), (c0, sets[c0:c0 + win])


def test_full_step_sets():
    assert [k for k, f in enumerate(oracle.full_steps("periodic", 30, 5)) if f] == [0, 5, 10, 15, 20, 25]
    assert [k for k, f in enumerate(oracle.full_steps("periodic", 30, 4)) if f] == [0, 4, 8, 12, 16, 20, 24, 28]
    assert [k for k, f in enumerate(oracle.full_steps("head_mid_tail", 30)) if f] == [0, 1, 15, 29]
    assert [k for k, f in enumerate(oracle.full_steps("head_mid_tail", 50)) if f] == [0, 1, 25, 49]
    # the paper's Hunyuan operating point: 10 steps, four of them full
    assert sum(oracle.full_steps("head_mid_tail", 10)) == 4
    # "a=2, E=5, S=10": the two-step head and E = 5 refresh steps at the end
    assert [k for k, f in enumerate(oracle.full_steps("head_tail_e", 10, 5)) if f] == [0, 1, 5, 6, 7, 8, 9]
    assert [k for k, f in enumerate(oracle.full_steps("head_tail_e", 30, 1)) if f] == [0, 1, 29]
    assert [k for k, f in enumerate(oracle.full_steps("head_tail_e", 8, 0)) if f] == [0, 1]
    assert all(oracle.full_steps("head_tail_e", 6, 6))
    with pytest.raises(ValueError):
        oracle.full_steps("head_tail_e", 10, 11)


@pytest.mark.parametrize("kind,dtype", [("ddim", "f32"), ("flow", "bf16")])
def test_all_anchor_trajectory_equals_plain_sampler(maps, kind, dtype):
    """With every view an anchor at every cached step (a = N) the cached loop
    is bit-identical to the plain sampler (every step full)."""
    w = synth.shrink(C2, dtype=dtype)
    P = maps(C2.name)
    S = 6
    rs = np.random.default_rng(7)
    xt0 = synth.storage(rs.standard_normal((1, w.N, w.H, w.W, w.C)).astype(np.float32), dtype)
    preds = {k: synth.storage(rs.standard_normal((1, w.N, w.H, w.W, w.C)).astype(np.float32), dtype)
             for k in range(S)}

    def stub(k, views):
        return preds[k][:, views]

    cams = synth.batch_cameras(w)
    cached = oracle.trajectory(xt0, stub, P, cams, 4, 0.01, dtype, kind, S, [1] + [0] * (S - 1), w.N)
    plain = oracle.trajectory(xt0, stub, P, cams, 4, 0.01, dtype, kind, S, [1] * S, w.N)
    for r1, r2 in zip(cached, plain):
        np.testing.assert_array_equal(r1["x_t"], r2["x_t"])
        np.testing.assert_array_equal(r1["x0"], r2["x0"])


# ---------------------------------------------------------------------------
# O8 multistep (UniPC) update
# ---------------------------------------------------------------------------

def test_unipc_order1_predictor_is_ddim():
    """UniPC of order 1 without the corrector is the DDIM step (closed form)."""
    S = 10
    ts = oracle.ddim_timesteps(S)
    rs = np.random.default_rng(0)
    x = rs.standard_normal(1024).astype(np.float32)
    m = rs.standard_normal(1024).astype(np.float32)
    for k in range(S):
        co = oracle.unipc_coeffs(S, k, order=1, corrector=False)
        _, xn = oracle.unipc_apply(co, x, None, None, None, m, "f32")
        want, _ = oracle.reconstruct(x, m, "f32", "ddim", ts[k], ts[k + 1])
        np.testing.assert_allclose(xn, want, rtol=0, atol=1e-12)


def test_unipc_constant_history_is_ddim_chain():
    """With the same x0 prediction at every step the multistep terms vanish:
    the corrected sample equals the DDIM step from the previous corrected
    sample, and the prediction equals the DDIM step from the corrected one."""
    S = 12
    ts = oracle.ddim_timesteps(S)
    rs = np.random.default_rng(1)
    m = rs.standard_normal(512).astype(np.float32)
    xprev = rs.standard_normal(512).astype(np.float32)
    for k in range(1, S):
        co = oracle.unipc_coeffs(S, k, order=2, corrector=True)
        assert co[0] == 1
        xc, xn = oracle.unipc_apply(co, None, xprev, m, m, m, "f32")
        want_c, _ = oracle.reconstruct(xprev, m, "f32", "ddim", ts[k - 1], ts[k])
        np.testing.assert_allclose(xc, want_c, rtol=0, atol=1e-9)
        want_n, _ = oracle.reconstruct(xc.astype(np.float32), m, "f32", "ddim", ts[k], ts[k + 1])
        np.testing.assert_allclose(xn, want_n, rtol=0, atol=1e-6)


def _unipc_error(S, order, corrector, c0=0.3, c1=0.7, t_check=99):
    """Run UniPC on a 'model' whose x0 prediction is c0 + c1 * lambda_t (it
    ignores x); the data-prediction ODE then has the exact solution
    x_t = (sigma_t / sigma_s) x_s + sigma_t [e^lam (c0 + c1 (lam - 1))]_s^t.
    Returns |x - x_exact| at timestep t_check."""
    ts = oracle.ddim_timesteps(S)
    lam = lambda t: 0.5 * math.log(oracle.alpha_bar(t) / (1 - oracle.alpha_bar(t)))
    sig = lambda t: math.sqrt(1 - oracle.alpha_bar(t))
    F = lambda L: math.exp(L) * (c0 + c1 * (L - 1))
    x0_start = 0.2
    t0 = ts[0]
    exact = lambda t: sig(t) / sig(t0) * x0_start + sig(t) * (F(lam(t)) - F(lam(t0)))
    xt = np.array([x0_start], np.float64)
    xprev = m1 = m2 = None
    for k in range(S):
        mk = np.array([c0 + c1 * lam(ts[k])])
        co = oracle.unipc_coeffs(S, k, order=order, corrector=corrector)
        xc = co[7] * 0 + (co[3] * xprev[0] + co[4] * (m2[0] if m2 is not None else 0) + co[5] * m1[0] + co[6] * mk[0]
                          if co[0] else xt[0])
        if ts[k] == t_check:
            return abs(xc - exact(t_check))
        xn = co[7] * xc + co[8] * (m1[0] if m1 is not None else 0) + co[9] * mk[0]
        xprev, m2, m1, xt = np.array([xc]), m1, mk, np.array([xn])
    raise AssertionError("t_check not on the grid")


def test_unipc_convergence_order():
    """Against the exact solution: halving the step cuts the error ~4x with
    the second-order solver and ~2x with DDIM (first order)."""
    e2 = [_unipc_error(S, 2, True) for S in (10, 20, 40)]
    e1 = [_unipc_error(S, 1, False) for S in (10, 20, 40)]
    assert e2[0] / e2[1] > 3.0 and e2[1] / e2[2] > 3.0, e2
    assert 1.5 < e1[0] / e1[1] < 2.6 and 1.5 < e1[1] / e1[2] < 2.6, e1
    assert e2[2] < e1[2] / 10


def test_unipc_orders_warm_up_and_final_step():
    """Multistep orders: first order at step 0 (no history yet), first order on
    the last step, the corrector taking the previous step's predictor order."""
    S = 10
    pp = [int(oracle.unipc_coeffs(S, k, order=2)[2]) for k in range(S)]
    pc = [int(oracle.unipc_coeffs(S, k, order=2)[1]) for k in range(S)]
    assert pp == [1] + [2] * (S - 2) + [1]
    assert pc == [0, 1] + [2] * (S - 2)
    assert oracle.unipc_coeffs(S, 0, order=2)[0] == 0        # no corrector before any history
    # the last step lands on sigma = 0: the prediction is the clean estimate
    co = oracle.unipc_coeffs(S, S - 1, order=2)
    assert co[7] == 0 and co[8] == 0 and co[9] == 1


# ---------------------------------------------------------------------------
# O9 token staleness and the coverage-driven schedule
# ---------------------------------------------------------------------------

def _toy_coverage():
    """1 asset, 3 views of 1 x 4 tokens; token 2 of view 1 is background.
    Anchor 0 sees tokens 0, 1 of view 1; anchor 1 sees tokens 2, 3 of view 2
    and token 0 of view 0; anchor 2 sees nothing."""
    pos = np.zeros((1, 3, 1, 4, 3), np.float32)
    pos[0, 1, 0, 2] = np.nan
    seen = np.zeros((3, 1, 3, 1, 4), np.uint8)
    seen[0, 0, 1, 0, [0, 1]] = 1
    seen[1, 0, 2, 0, [2, 3]] = 1
    seen[1, 0, 0, 0, 0] = 1
    return pos, seen


def test_coverage_hand_sequence():
    pos, seen = _toy_coverage()
    st = oracle.coverage_init(pos)
    assert st.reshape(3, 4).tolist() == [[0, 0, 0, 0], [0, 0, 255, 0], [0, 0, 0, 0]]
    # step with A = {0}: view 0 fresh; view 1 tokens 0, 1 seen; the rest miss a step
    st, stats = oracle.coverage_update(st, seen, [0], R=2)
    assert st.reshape(3, 4).tolist() == [[0, 0, 0, 0], [0, 0, 255, 1], [1, 1, 1, 1]]
    assert stats[0].tolist() == [[4, 0, 0, 0], [3, 0, 1, 1], [4, 0, 4, 1]]
    # A = {1}: view 1 fresh, view 0 token 0 and view 2 tokens 2, 3 seen
    st, stats = oracle.coverage_update(st, seen, [1], R=2)
    assert st.reshape(3, 4).tolist() == [[0, 1, 1, 1], [0, 0, 255, 0], [2, 2, 0, 0]]
    assert stats[0].tolist() == [[4, 0, 3, 1], [3, 0, 0, 0], [4, 2, 4, 2]]
    # A = {2} twice: view 2 fresh; views 0 and 1 age
    st, _ = oracle.coverage_update(st, seen, [2], R=2)
    st, stats = oracle.coverage_update(st, seen, [2], R=2)
    assert st.reshape(3, 4).tolist() == [[2, 3, 3, 3], [2, 2, 255, 2], [0, 0, 0, 0]]
    assert stats[0].tolist() == [[4, 4, 11, 3], [3, 3, 6, 2], [4, 0, 0, 0]]
    # a full step (every view an anchor) resets every foreground token
    st, stats = oracle.coverage_update(st, seen, [0, 1, 2], R=1)
    assert st.reshape(3, 4).tolist() == [[0, 0, 0, 0], [0, 0, 255, 0], [0, 0, 0, 0]]
    assert stats[0, :, 1].tolist() == [0, 0, 0]


def test_coverage_gains_and_greedy_by_hand():
    pos, seen = _toy_coverage()
    st = np.array([[2, 3, 3, 3], [2, 2, 255, 2], [0, 0, 0, 0]], np.uint8).reshape(1, 3, 1, 4)
    # weights 1 + staleness: view 0: 3 4 4 4; view 1: 3 3 - 3; view 2: 1 1 1 1
    # u = 0: own view (15) + view 1 tokens 0, 1 (6) = 21; u = 1: own (9) + view 0
    # token 0 (3) + view 2 tokens 2, 3 (2) = 14; u = 2: own (4)
    assert oracle.coverage_gains(st, seen, []).tolist() == [21, 14, 4]
    # after choosing 0: u = 1 adds view 1 token 3 (3) and view 2 tokens 2, 3 (2)
    assert oracle.coverage_gains(st, seen, [0]).tolist() == [0, 5, 4]
    assert oracle.coverage_select(st, seen, 2) == [0, 1]
    assert oracle.coverage_select(st, seen, 2, forced=[2]) == [0, 2]
    assert oracle.coverage_select(st, seen, 3) == [0, 1, 2]
    with pytest.raises(ValueError):
        oracle.coverage_select(st, seen, 2, forced=[1, 1])


def _weighted_coverage(st, seen, S):
    B, N = st.shape[:2]
    w = np.where(st == 255, 0, 1 + st.astype(np.int64))
    cov = np.zeros(st.shape, bool)
    for u in S:
        cov[:, u] = True
        cov |= seen[u].astype(bool)
    return int((w * cov).sum())


def test_coverage_greedy_against_brute_force():
    """Greedy picks the best single view first, and its set reaches at least
    (1 - 1/e) of the best weighted coverage over all a-subsets (the classical
    bound for greedy maximum coverage) on random small instances."""
    import itertools
    rs = np.random.default_rng(4)
    for trial in range(12):
        N, a, H, W = 6, 2 + trial % 2, 5, 7
        st = rs.integers(0, 6, (2, N, H, W)).astype(np.uint8)
        st[rs.random(st.shape) < 0.1] = 255
        seen = (rs.random((N, 2, N, H, W)) < 0.3).astype(np.uint8)
        for u in range(N):
            seen[u, :, u] = 0
        g = oracle.coverage_gains(st, seen, [])
        single = [_weighted_coverage(st, seen, [u]) for u in range(N)]
        assert g.tolist() == single
        S = oracle.coverage_select(st, seen, a)
        assert int(np.argmax(single)) in S
        best = max(_weighted_coverage(st, seen, c) for c in itertools.combinations(range(N), a))
        assert _weighted_coverage(st, seen, S) >= (1 - 1 / np.e) * best


def test_coverage_saturates_and_keeps_background():
    pos, seen = _toy_coverage()
    st = oracle.coverage_init(pos)
    for _ in range(300):
        st, stats = oracle.coverage_update(st, seen, [2], R=1)
    assert st[0, 0].max() == 254 and st[0, 1, 0, 2] == 255
    assert stats[0, 0].tolist() == [4, 4, 4 * 254, 254]


def test_coverage_pairs_or_equals_set_visibility():
    """A set sees a token iff one of its anchors does on its own: the OR of
    the single-anchor pairs equals n_vis > 0 of the set's own build."""
    P = latent_maps("hunyuan_torus_6v_64")
    w = synth.CONFIGS["hunyuan_torus_6v_64"]
    cams = synth.batch_cameras(w)
    bb = oracle.bbox(P, w.tol_frac)
    seen = oracle.coverage_pairs(P, cams, w.K, bb)
    for u in range(w.N):
        assert not seen[u, :, u].any()
    for c in range(3):
        A = oracle.anchors(w.N, w.a, c)
        _, _, nvis = oracle.build(P, cams, A, w.K, bb)
        targets = [v for v in range(w.N) if v not in A]
        for ti, v in enumerate(targets):
            np.testing.assert_array_equal(np.any(seen[A][:, :, v], axis=0), nvis[:, ti] > 0)


def test_refresh_due():
    stats = np.zeros((2, 3, 4), np.uint32)
    stats[..., 0] = 100
    stats[0, 1, 1] = 30                        # 30 of 600 foreground tokens stale >= R
    assert oracle.refresh_due(stats, 0.04)
    assert not oracle.refresh_due(stats, 0.05)
    assert not oracle.refresh_due(np.zeros((1, 1, 4), np.uint32), 0.0)


def test_coverage_score_hand_and_brute_force():
    pos, seen = _toy_coverage()
    st = np.array([[2, 3, 3, 3], [2, 2, 255, 2], [0, 0, 0, 0]], np.uint8).reshape(1, 3, 1, 4)
    # {0}: 21 (as the gain above); {1, 2}: own views 9 + 4, view 0 token 0 (3) = 16
    assert oracle.coverage_score(st, seen, [[0, 0], [1, 2]]).tolist() == [21, 16]
    rs = np.random.default_rng(8)
    for trial in range(6):
        N, a = 7, 3
        st = rs.integers(0, 9, (2, N, 4, 6)).astype(np.uint8)
        st[rs.random(st.shape) < 0.1] = 255
        seen = (rs.random((N, 2, N, 4, 6)) < 0.25).astype(np.uint8)
        for u in range(N):
            seen[u, :, u] = 0
        sets = [list(rs.choice(N, a, replace=False)) for _ in range(5)]
        assert oracle.coverage_score(st, seen, sets).tolist() == [_weighted_coverage(st, seen, S) for S in sets]


def test_rotation_sets():
    assert oracle.rotation_sets(12, 4) == [[0, 3, 6, 9], [1, 4, 7, 10], [2, 5, 8, 11]]
    assert oracle.rotation_sets(6, 2) == [[0, 3], [1, 4], [2, 5]]
    assert len(oracle.rotation_sets(10, 3)) == 10


# ---------------------------------------------------------------------------
# O7/O8/O9 loop level: the oracle's own trajectory and schedule functions
# ---------------------------------------------------------------------------
# Each pin takes the oracle module (or a planted-mutation copy of its
# loop-level functions) so that test_planted_loop_mutations_fail_pins can
# show every planted mistake failing one of them.

def _lam(t):
    ab = oracle.alpha_bar(t)
    return 0.5 * math.log(ab / (1 - ab))


def _pin_unipc_trajectory_exact_ode(orc):
    """oracle.trajectory_unipc, every step full, on a model whose x0 is
    c0 + c1 * lambda_t: the data-prediction ODE has the exact solution
    x_t = (sigma_t / sigma_s) x_s + sigma_t [e^lam (c0 + c1 (lam - 1))]_s^t,
    and halving the step must cut the error of the corrected sample by the
    solver's order: third order for order 2 with the corrector (the corrector
    raises the order by one), second order for order 1 with it, first order
    (DDIM) without."""
    c0, c1, x_start, t_check = 0.3, 0.7, 0.2, 99
    sig = lambda t: math.sqrt(1 - oracle.alpha_bar(t))
    F = lambda L: math.exp(L) * (c0 + c1 * (L - 1))

    def err(S, order, corr):
        ts = oracle.ddim_timesteps(S)
        exact = sig(t_check) / sig(ts[0]) * x_start + sig(t_check) * (F(_lam(t_check)) - F(_lam(ts[0])))
        k = ts.index(t_check)
        pos = np.zeros((1, 2, 1, 4, 3), np.float32)
        xt0 = np.full((1, 2, 1, 4, 4), x_start, np.float32)
        stub = lambda kk, views: np.full((1, len(views), 1, 4, 4), c0 + c1 * _lam(ts[kk]), np.float32)
        recs = orc.trajectory_unipc(xt0, stub, pos, None, 4, 0.01, "f32", S, [1] * S, 1, order, corr, steps=k + 1)
        got = recs[k]["x_c_exact"] if corr else recs[k - 1]["x_t_exact"]
        return float(np.abs(got - exact).max())

    e2c = [err(S, 2, True) for S in (10, 20, 40)]
    e1c = [err(S, 1, True) for S in (10, 20, 40)]
    e1 = [err(S, 1, False) for S in (10, 20, 40)]
    assert e2c[0] / e2c[1] > 6 and e2c[1] / e2c[2] > 6, e2c
    assert e1c[0] / e1c[1] > 3 and e1c[1] / e1c[2] > 3, e1c
    assert all(1.5 < e1[i] / e1[i + 1] < 2.6 for i in range(2)), e1
    assert e2c[2] < 1e-5


def _pin_unipc_history_by_hand(orc):
    """A mixed full / cached trajectory whose x0 history is known by hand:
    three views that see nothing of each other (all background), so at a
    cached step the anchor takes its new prediction and every other view
    keeps its stored x0 (Sec. 3.2, invalid matches).  Each view's prediction
    at step k is the constant 1 + k/8 + u/64; the anchor of cached step c is
    view c mod 3.  The expected corrected samples and predictions follow
    from the UniPC recurrence on those scalars (coefficients from
    oracle.unipc_coeffs, pinned above), with x_c and x_t stored as float32
    between steps."""
    S, N = 6, 3
    full = [1, 0, 0, 1, 0, 0]
    p = lambda k, u: 1.0 + k / 8 + u / 64
    # x0 store after each step, by hand: m0 = p0; m1 = (p1[0], m0[1], m0[2]);
    # m2 = (m1[0], p2[1], m1[2]); m3 = p3; m4 = (m3[0], m3[1], p4[2]);
    # m5 = (p5[0], m4[1], m4[2])
    m = [[p(0, 0), p(0, 1), p(0, 2)],
         [p(1, 0), p(0, 1), p(0, 2)],
         [p(1, 0), p(2, 1), p(0, 2)],
         [p(3, 0), p(3, 1), p(3, 2)],
         [p(3, 0), p(3, 1), p(4, 2)],
         [p(5, 0), p(3, 1), p(4, 2)]]
    anchors = [[0, 1, 2], [0], [1], [0, 1, 2], [2], [0]]
    pos = np.full((1, N, 1, 4, 3), np.nan, np.float32)
    cams = batch(ortho_cams(np.eye(3), [0, 0, 0], 1.0, [(2, 0.5)] * N))
    x_start = np.array([0.25, -0.5, 0.75], np.float32)
    xt0 = np.ascontiguousarray(np.broadcast_to(x_start[None, :, None, None, None], (1, N, 1, 4, 4)))

    def stub(k, views):
        return np.ascontiguousarray(np.broadcast_to(
            np.array([p(k, u) for u in views], np.float32)[None, :, None, None, None], (1, len(views), 1, 4, 4)))

    recs = orc.trajectory_unipc(xt0, stub, pos, cams, 4, 0.01, "f32", S, full, 1, 2, True)
    assert [r["anchors"] for r in recs] == anchors
    x = [float(v) for v in x_start]
    xprev = [None] * N
    for k, r in enumerate(recs):
        co = oracle.unipc_coeffs(S, k, 2, True)
        for u in range(N):
            m2 = m[k - 2][u] if k >= 2 else 0.0
            m1 = m[k - 1][u] if k >= 1 else 0.0
            mk = m[k][u]
            xc = co[3] * xprev[u] + co[4] * m2 + co[5] * m1 + co[6] * mk if co[0] else x[u]
            xn = co[7] * xc + co[8] * m1 + co[9] * mk
            assert np.all(r["x0"][0, u] == np.float32(mk)), (k, u)
            np.testing.assert_allclose(r["x_c_exact"][0, u], xc, rtol=0, atol=1e-12, err_msg=f"x_c k={k} u={u}")
            np.testing.assert_allclose(r["x_t_exact"][0, u], xn, rtol=0, atol=1e-12, err_msg=f"x_t k={k} u={u}")
            xprev[u] = float(np.float32(xc))
            x[u] = float(np.float32(xn))


def _pin_forced_views_by_hand(orc):
    """The coverage schedule's forced views and anchor gaps on the toy scene
    (three views of 1 x 4 tokens; _toy_coverage), derived by hand.

    a = 1, max_gap = 1, step 0 full: step 1 forces nothing (all gaps 0) and
    the greedy takes view 0 (gains 6, 6, 4: the tie goes to the lower view);
    from then on the views whose gap reached 1 are forced, the longest gap
    first and equal gaps to the lower view: 1 (gaps 0 1 1), 2 (1 0 2),
    0 (2 1 0), 1, 2.

    a = 1, max_gap = 2, steps 0 and 3 full: step 1 greedy 0 (tie), step 2
    greedy 1 (gains 6, 9, 8 with weights 1 + staleness), step 3 full resets
    every gap, so steps 4 and 5 repeat steps 1 and 2, and step 6 forces
    view 2 (gap 2).

    a = 2, max_gap = 1: step 1 greedy {0, then 2} (after 0, view 1 adds 3 and
    view 2 adds 4); step 2 forces view 1 and the greedy adds 0 (3 against 2);
    step 3 forces view 2 and the greedy adds 0 (6 against 4)."""
    pos, seen = _toy_coverage()
    st0 = orc.coverage_init(pos)
    cases = [
        (1, 1, [1, 0, 0, 0, 0, 0, 0],
         [[0, 1, 2], [0], [1], [2], [0], [1], [2]],
         [[0, 0, 0], [0, 1, 1], [1, 0, 2], [2, 1, 0], [0, 2, 1], [1, 0, 2], [2, 1, 0]]),
        (1, 2, [1, 0, 0, 1, 0, 0, 0],
         [[0, 1, 2], [0], [1], [0, 1, 2], [0], [1], [2]],
         [[0, 0, 0], [0, 1, 1], [1, 0, 2], [0, 0, 0], [0, 1, 1], [1, 0, 2], [2, 1, 0]]),
        (2, 1, [1, 0, 0, 0],
         [[0, 1, 2], [0, 2], [0, 1], [0, 2]],
         [[0, 0, 0], [0, 1, 0], [0, 0, 1], [0, 1, 0]]),
    ]
    for a, max_gap, full, want_a, want_gap in cases:
        recs = orc.schedule_adaptive(seen, st0, full, a, "coverage", max_gap=max_gap, R=2)
        assert [r["anchors"] for r in recs] == want_a, (a, max_gap)
        assert [r["gap"] for r in recs] == want_gap, (a, max_gap)
        assert [r["full"] for r in recs] == [bool(f) for f in full]
    assert orc.forced_views([0, 1, 1], 1, 1) == [1]
    assert orc.forced_views([1, 0, 2], 3, 1) == [2, 0]
    assert orc.forced_views([3, 3, 3], 2, 2) == [0, 1]
    assert orc.forced_views([5, 5, 5], 3, 0) == []
    assert orc.advance_gaps([1, 0, 2], [2], False) == [2, 1, 0]
    assert orc.advance_gaps([1, 0, 2], [], True) == [0, 0, 0]


def test_unipc_trajectory_exact_ode():
    _pin_unipc_trajectory_exact_ode(oracle)


def test_unipc_trajectory_history_by_hand():
    _pin_unipc_history_by_hand(oracle)


def test_forced_views_and_gaps_by_hand():
    _pin_forced_views_by_hand(oracle)


def _mutant(fn_name, old, new):
    """A copy of the oracle's loop-level Python functions with one planted
    mistake (a source replacement in fn_name); the copies call each other."""
    import inspect
    import types
    ns = dict(vars(oracle))
    for fn in ("forced_views", "advance_gaps", "schedule_adaptive", "trajectory_unipc"):
        src = inspect.getsource(getattr(oracle, fn))
        if fn == fn_name:
            assert old in src, f"the planted mistake no longer matches {fn}"
            src = src.replace(old, new)
        exec(compile(src, f"<mutant {fn}>", "exec"), ns)
    return types.SimpleNamespace(**ns)


@pytest.mark.parametrize("fn,old,new", [
    # the multistep history shifted wrongly: m_{k-1} and m_{k-2} swapped
    ("trajectory_unipc", "x_prev, m2, m1 = xc_s, m1, mk", "x_prev, m2, m1 = xc_s, mk, m1"),
    # a cached step transporting onto the x0 of step k-2 instead of k-1
    ("trajectory_unipc", "transport(m1, stub(k, A)", "transport(m2 if m2 is not None else m1, stub(k, A)"),
    # the corrected sample not carried to the next step
    ("trajectory_unipc", "x_prev, m2, m1 = xc_s, m1, mk", "x_prev, m2, m1 = x_t, m1, mk"),
    # a full step not resetting the anchor gaps
    ("schedule_adaptive", "gap = advance_gaps(gap, A, is_full)",
     "gap = advance_gaps(gap, A, is_full) if not is_full else gap"),
    # equal gaps going to the higher view
    ("forced_views", "due.sort(key=lambda v: (-gap[v], v))", "due.sort(key=lambda v: (-gap[v], -v))"),
    # the forced list not capped at a
    ("forced_views", "return due[:a]", "return due[:a + 1]"),
])
def test_planted_loop_mutations_fail_pins(fn, old, new):
    """Every planted mistake in the loop-level functions fails at least one
    of the pins above (and the unmutated copy passes them all)."""
    pins = (_pin_unipc_trajectory_exact_ode, _pin_unipc_history_by_hand, _pin_forced_views_by_hand)
    clean = _mutant(fn, old, old)
    for pin in pins:
        pin(clean)
    bad = _mutant(fn, old, new)
    failed = []
    for pin in pins:
        try:
            pin(bad)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake in {fn}"
