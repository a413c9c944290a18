"""The documented limits, element by element against the oracle:
  * grids at GC_MAX_GRID along one axis (4094 x 40 and 40 x 4094: footprint
    coordinates above 2048 use the top bit of the packed word's 12-bit fields);
  * GC_MAX_VIEWS views with GC_MAX_ANCHORS anchors (64 views, 8 anchors): the
    stored operator, its index, both launches, the on-the-fly operator and
    the coverage bits (64-bit view masks full);
  * GC_MAX_CHANNELS channels through the stored-operator path.
Bars as in the parity tests: words bit-exact, weights 1e-6, latents float32
1e-5 / bfloat16 2e-2 against the oracle's unrounded values."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth.configs import C2

from conftest import latent_maps, visible_weights
from test_gpu_properties import random_rig

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = {"f32": 1e-5, "bf16": 2e-2}


@pytest.fixture(scope="module")
def gc():
    import paper_2608_13255_amd as gc
    return gc


def to_dev(arr, dtype):
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr)).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(DEV).view(torch.bfloat16)


def vals(t, dtype):
    h = t.cpu().numpy() if dtype == "f32" else t.view(torch.int16).cpu().numpy().view(np.uint16)
    return synth.values(h, dtype).astype(np.float64)


def bits(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def sphere_problem(seed, N, H, W, pinhole=False):
    rs = np.random.default_rng(seed)
    cams = random_rig(rs, N, H, W, pinhole)
    prm = synth.sphere_params(synth.CONFIGS["tiny_sphere_4v_32"], seed % 7)
    P = synth.raycast_radial(0.05, prm, cams, H, W)[None]
    return rs, P, {k: v[None] for k, v in cams.items()}


def full_check(gc, P, bcams, anchors, K, C, dtype, rs, tol_frac=0.03, geom=True, pairs=True):
    N = P.shape[1]
    H, W = P.shape[2], P.shape[3]
    a = len(anchors)
    bb = oracle.bbox(P, tol_frac)
    corr_o, wts_o, nvis_o = oracle.build(P, bcams, anchors, K, bb)
    prev = synth.storage(0.5 * rs.standard_normal((1, N, H, W, C)).astype(np.float32), dtype)
    new = synth.storage(synth.values(prev, dtype)[:, anchors] + 0.1 * rs.standard_normal((1, a, H, W, C)).astype(np.float32), dtype)
    xt = synth.storage(0.5 * rs.standard_normal((1, N, H, W, C)).astype(np.float32), dtype)
    x0_exact, x0_state = oracle.transport(prev, new, corr_o, wts_o, anchors, dtype)
    xn_o, _ = oracle.reconstruct(xt, x0_state, dtype, "flow", 0.6, 0.55)
    Pd = torch.from_numpy(P).to(DEV)
    cams_d = gc.camera_tensor(bcams, DEV)
    bbd = gc.gc_posmap_bbox(Pd, tol_frac)
    corr, wts = gc.gc_build_correspondence(Pd, cams_d, anchors, K, bbd)
    np.testing.assert_array_equal(corr.cpu().numpy(), corr_o)
    assert np.abs(visible_weights(corr, wts) - wts_o).max(initial=0.0) <= 1e-6
    idx = gc.gc_index_correspondence(corr)
    assert idx.n_vis == int((nvis_o > 0).sum())
    smp = gc.Sampler(kind=gc.GC_FLOW_EULER)
    outs = []
    for index in (None, idx):
        x0_out, x_next, _ = gc.gc_transport_reconstruct(to_dev(prev, dtype), to_dev(new, dtype), corr, wts,
                                                        to_dev(xt, dtype), anchors, smp, 0.6, 0.55, index=index)
        assert np.abs(vals(x0_out, dtype) - x0_exact).max() <= TOL[dtype]
        same = np.ones(x0_state.shape, bool) if dtype == "f32" else (
            x0_out.view(torch.int16).cpu().numpy().view(np.uint16) == x0_state)
        assert np.abs(vals(x_next, dtype) - xn_o)[same].max(initial=0.0) <= TOL[dtype]
        outs.append((x0_out, x_next))
    assert torch.equal(bits(outs[0][0]), bits(outs[1][0])) and torch.equal(bits(outs[0][1]), bits(outs[1][1]))
    if geom:
        g0, g1, _ = gc.gc_transport_reconstruct_geom(to_dev(prev, dtype), to_dev(new, dtype), Pd, cams_d, bbd,
                                                     to_dev(xt, dtype), anchors, K, smp, 0.6, 0.55)
        assert torch.equal(bits(g0), bits(outs[0][0])) and torch.equal(bits(g1), bits(outs[0][1]))
    if pairs:
        pb = gc.gc_coverage_pairs(Pd, cams_d, bbd).cpu().numpy().view(np.uint32)
        un = np.unpackbits(np.ascontiguousarray(pb).view(np.uint8), axis=-1, bitorder="little")
        un = un.reshape(N, 1, N, -1)[..., :H * W].reshape(N, 1, N, H, W)
        np.testing.assert_array_equal(un, oracle.coverage_pairs(P, bcams, K, bb))
    return corr_o


@pytest.mark.parametrize("H,W", [(4094, 40), (40, 4094)])
def test_max_grid_extent(gc, H, W):
    rs, P, bcams = sphere_problem(3, 3, H, W)
    corr_o = full_check(gc, P, bcams, [1], 4, 4, "f32", rs, tol_frac=0.01, pairs=False)
    seen = corr_o[corr_o != 0]
    x1 = (seen & 0xfff).astype(np.int64)
    y1 = ((seen >> 12) & 0xfff).astype(np.int64)
    # footprints reach far along the long axis (coordinates above 2048 use the top bit of the 12-bit fields)
    assert max(x1.max(), y1.max()) > 3500


def test_max_views_and_anchors(gc):
    rs, P, bcams = sphere_problem(11, 64, 24, 20, pinhole=True)
    anchors = sorted(rs.choice(64, 8, replace=False).tolist())
    full_check(gc, P, bcams, anchors, 4, 8, "bf16", rs)
    # coverage over a full 64-view mask: staleness and a greedy selection of 8
    Pd = torch.from_numpy(P).to(DEV)
    cams_d = gc.camera_tensor(bcams, DEV)
    bbd = gc.gc_posmap_bbox(Pd, 0.03)
    pb = gc.gc_coverage_pairs(Pd, cams_d, bbd)
    seen = oracle.coverage_pairs(P, bcams, 4, oracle.bbox(P, 0.03))
    stale = gc.gc_coverage_init(Pd)
    st_o = oracle.coverage_init(P)
    for A in (anchors, list(range(64)), [63], anchors):
        stats = gc.gc_coverage_update(pb, stale, A, 2)
        st_o, stats_o = oracle.coverage_update(st_o, seen, A, 2)
        np.testing.assert_array_equal(stale.cpu().numpy(), st_o)
        np.testing.assert_array_equal(stats.cpu().numpy().view(np.uint32), stats_o)
    sel = gc.gc_coverage_select(pb, stale, 8, forced=[63]).cpu().tolist()
    assert sel == oracle.coverage_select(st_o, seen, 8, forced=[63])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_max_channels_stored_operator(gc, dtype):
    w = C2
    P = latent_maps(w.name)
    rs = np.random.default_rng(23)
    A = oracle.anchors(w.N, w.a, 1)
    full_check(gc, P, synth.batch_cameras(w), A, 4, 256, dtype, rs, tol_frac=w.tol_frac, pairs=False)
