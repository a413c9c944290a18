"""Property-based parity (hypothesis): random small problems -- grid sizes
that are not multiples of anything, 2-7 views, 1-4 anchors, K = 1..4, C = 4..16,
float32 / bfloat16, orthographic or pinhole rigs with random poses (points
behind a pinhole camera included), random background holes and tolerances --
through the whole per-step path against the oracle (the on-the-fly operator
bit for bit against the stored one, the coverage visibility bits against the
oracle's), plus HIP-graph replays.
"""
import math

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
import synth

from conftest import stored_x0_slack, visible_weights, x0_coef

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = {"f32": 1e-5, "bf16": 2e-2}


def to_dev(arr, dtype):
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr)).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(DEV).view(torch.bfloat16)


def to_host(t, dtype):
    return t.cpu().numpy() if dtype == "f32" else t.view(torch.int16).cpu().numpy().view(np.uint16)


def random_rig(rs, N, H, W, pinhole):
    cams = {"model": np.full(N, 0 if pinhole else 1, np.int32), "R": np.zeros((N, 3, 3), np.float32),
            "t": np.zeros((N, 3), np.float32), "fx": np.zeros(N, np.float32), "fy": np.zeros(N, np.float32),
            "cx": np.full(N, W / 2, np.float32), "cy": np.full(N, H / 2, np.float32)}
    for v in range(N):
        az, el = rs.uniform(0, 360), rs.uniform(-40, 40)
        dist = rs.uniform(1.2, 4.0) if pinhole else 3.0      # pinhole rigs may sit inside the bound
        R, t = synth.look_at_origin(az, el, dist)
        if pinhole and rs.random() < 0.25:
            F = np.diag([-1.0, 1.0, -1.0])        # turned away: the object is behind this camera
            R, t = F @ R, F @ t
        cams["R"][v], cams["t"][v] = R, t
        if pinhole:
            f = (W / 2) / math.tan(math.radians(rs.uniform(30, 60) / 2))
            cams["fx"][v], cams["fy"][v] = f, f * H / W * rs.uniform(0.8, 1.2)
        else:
            cams["fx"][v], cams["fy"][v] = W / 2.4, H / 2.4
    return cams


@settings(max_examples=30, deadline=None, derandomize=True, suppress_health_check=list(HealthCheck))
@given(seed=st.integers(0, 2 ** 31 - 1), H=st.integers(1, 40), W=st.integers(1, 40), N=st.integers(2, 7),
       a_frac=st.floats(0.0, 1.0), K=st.integers(1, 4), C=st.sampled_from([4, 8, 12, 16]),
       dtype=st.sampled_from(["f32", "bf16"]), pinhole=st.booleans(), tol=st.sampled_from([0.01, 0.03, 0.1]),
       holes=st.floats(0.0, 0.3), sampler=st.sampled_from(["ddim", "flow"]))
def test_random_problems_match_oracle(seed, H, W, N, a_frac, K, C, dtype, pinhole, tol, holes, sampler):
    import paper_2608_13255_amd as gc
    rs = np.random.default_rng(seed)
    a = 1 + int(a_frac * (min(N, 4) - 1) + 0.5)
    anchors = sorted(rs.choice(N, size=a, replace=False).tolist())
    cams = random_rig(rs, N, H, W, pinhole)
    prm = synth.sphere_params(synth.CONFIGS["tiny_sphere_4v_32"], int(seed % 7))
    P = synth.raycast_radial(0.05, prm, cams, H, W)[None]
    P[0][rs.random((N, H, W)) < holes] = np.nan
    bcams = {k: v[None] for k, v in cams.items()}
    bb = oracle.bbox(P, tol)
    corr_o, wts_o, nvis_o = oracle.build(P, bcams, anchors, K, bb)
    prev = synth.storage(rs.standard_normal((1, N, H, W, C)).astype(np.float32), dtype)
    new = synth.storage(synth.values(prev, dtype)[:, anchors] + 0.1 * rs.standard_normal((1, a, H, W, C)).astype(np.float32), dtype)
    xt = synth.storage(rs.standard_normal((1, N, H, W, C)).astype(np.float32), dtype)
    if sampler == "ddim":
        t, tn = int(rs.integers(1, 999)), None
        tn = int(rs.integers(-1, t))
        smp, pred = gc.Sampler(kind=gc.GC_DDIM, pred_out=gc.GC_PRED_EPS), "eps"
        cond = max(1.0, 1 / math.sqrt(1 - oracle.alpha_bar(t)))
    else:
        t = float(rs.uniform(0.05, 1.0))
        tn = float(rs.uniform(0.0, t))
        smp, pred = gc.Sampler(kind=gc.GC_FLOW_EULER, pred_out=gc.GC_PRED_VEL), "vel"
        cond = max(1.0, 1 / t)
    x0_exact, x0_state = oracle.transport(prev, new, corr_o, wts_o, anchors, dtype)
    xn_o, mo_o = oracle.reconstruct(xt, x0_state, dtype, sampler, t, tn, pred=pred)

    Pd = torch.from_numpy(P).to(DEV)
    bbd = gc.gc_posmap_bbox(Pd, tol)
    np.testing.assert_array_equal(bbd.cpu().numpy()[:, 6].view(np.uint32), bb[:, 6].view(np.uint32))
    corr, wts = gc.gc_build_correspondence(Pd, gc.camera_tensor(bcams, DEV), anchors, K, bbd)
    np.testing.assert_array_equal(corr.cpu().numpy(), corr_o)
    assert np.abs(visible_weights(corr, wts) - wts_o).max(initial=0.0) <= 1e-6
    idx = gc.gc_index_correspondence(corr)
    assert idx.n_vis == int((nvis_o > 0).sum())
    outs = []
    for index in (None, idx):
        x0_out, x_next, mo = gc.gc_transport_reconstruct(to_dev(prev, dtype), to_dev(new, dtype), corr, wts,
                                                         to_dev(xt, dtype), anchors, smp, t, tn, index=index)
        outs.append((x0_out, x_next, mo))
        x0h = to_host(x0_out, dtype)
        assert np.abs(synth.values(x0h, dtype).astype(np.float64) - x0_exact).max() <= TOL[dtype]
        assert np.abs(synth.values(to_host(x_next, dtype), dtype).astype(np.float64) - xn_o).max() <= TOL[dtype]
        slack = stored_x0_slack(x0h, x0_state, dtype)
        err = np.abs(synth.values(to_host(mo, dtype), dtype).astype(np.float64) - mo_o)
        assert (err <= TOL[dtype] * cond + x0_coef(sampler, pred, t) * slack).all()
    # the on-the-fly operator equals the stored one bit for bit
    cams_d = gc.camera_tensor(bcams, DEV)
    geo = gc.gc_transport_reconstruct_geom(to_dev(prev, dtype), to_dev(new, dtype), Pd, cams_d, bbd,
                                           to_dev(xt, dtype), anchors, K, smp, t, tn)
    iv = torch.int32 if dtype == "f32" else torch.int16
    for g_, r_ in zip(geo, outs[0]):
        assert torch.equal(g_.view(iv), r_.view(iv))
    # single-anchor visibility bits equal the oracle's
    bits = gc.gc_coverage_pairs(Pd, cams_d, bbd).cpu().numpy().view(np.uint32)
    unpacked = np.unpackbits(np.ascontiguousarray(bits).view(np.uint8), axis=-1, bitorder="little")
    unpacked = unpacked.reshape(N, 1, N, -1)[..., :H * W].reshape(N, 1, N, H, W)
    np.testing.assert_array_equal(unpacked, oracle.coverage_pairs(P, bcams, K, bb))


def test_graph_replays_match_eager():
    """Fused steps captured in a HIP graph and replayed several times, with
    eager work and synchronisations between replays: every replay equals the
    eager result bit for bit."""
    import paper_2608_13255_amd as gc
    from conftest import latent_maps
    from synth.configs import C2
    w = C2
    P = torch.from_numpy(latent_maps(w.name)).to(DEV)
    cams = gc.camera_tensor(synth.batch_cameras(w), DEV)
    bb = gc.gc_posmap_bbox(P)
    rs = np.random.default_rng(0)
    sets = [gc.gc_schedule_anchors(w.N, w.a, c) for c in range(3)]
    ops = {tuple(A): gc.gc_build_correspondence(P, cams, A, w.K, bb) for A in sets}
    idx = {A: gc.gc_index_correspondence(ops[A][0]) for A in ops}
    x0 = torch.from_numpy(rs.standard_normal((1, w.N, w.H, w.W, w.C)).astype(np.float32)).to(DEV)
    news = [torch.from_numpy(rs.standard_normal((1, w.a, w.H, w.W, w.C)).astype(np.float32)).to(DEV) for _ in sets]
    xt = torch.from_numpy(rs.standard_normal((1, w.N, w.H, w.W, w.C)).astype(np.float32)).to(DEV)
    smp = gc.Sampler(kind=gc.GC_DDIM)
    outs = [(torch.empty_like(x0), torch.empty_like(x0)) for _ in sets]
    s = torch.cuda.Stream()
    calls = [gc.bind_transport_reconstruct(x0, news[i], *ops[tuple(A)], xt, A, smp, outs[i][0], outs[i][1],
                                           index=idx[tuple(A)], stream=s) for i, A in enumerate(sets)]
    times = [(966, 932), (932, 899), (899, 866)]
    with torch.cuda.stream(s):
        for c, (t, tn) in zip(calls, times):
            c(t, tn)
    torch.cuda.synchronize()
    eager = [(o.clone(), n.clone()) for o, n in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for c, (t, tn) in zip(calls, times):
            c(t, tn)
    for rep in range(4):
        for o, n in outs:
            o.fill_(float("nan"))
            n.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for (o, n), (eo, en) in zip(outs, eager):
            assert torch.equal(o.view(torch.int32), eo.view(torch.int32)), rep
            assert torch.equal(n.view(torch.int32), en.view(torch.int32)), rep
        _ = (x0 * 2).sum().item()          # eager work between replays


def test_graph_replays_other_paths():
    """The on-the-fly step (blocked and foreground launches), the fused UniPC
    step, the coverage update + greedy selection and the fused update +
    selection / scoring captured in one HIP graph: every replay (with eager
    work, state resets and synchronisations between replays) equals the
    eager result bit for bit."""
    import paper_2608_13255_amd as gc
    from conftest import latent_maps
    from synth.configs import C4
    w = C4
    P = torch.from_numpy(latent_maps(w.name)).to(DEV)
    cams = gc.camera_tensor(synth.batch_cameras(w), DEV)
    bb = gc.gc_posmap_bbox(P, w.tol_frac)
    rs = np.random.default_rng(5)
    shape = (1, w.N, w.H, w.W, w.C)
    bf = lambda sh: torch.from_numpy(rs.standard_normal(sh).astype(np.float32)).to(DEV).to(torch.bfloat16)
    A0, A1 = gc.gc_schedule_anchors(w.N, w.a, 0), gc.gc_schedule_anchors(w.N, w.a, 1)
    corr1, wts1 = gc.gc_build_correspondence(P, cams, A1, w.K, bb)
    idx1 = gc.gc_index_correspondence(corr1)
    x0, xt, xprev, m2 = bf(shape), bf(shape), bf(shape), bf(shape)
    new0, new1 = bf((1, w.a, w.H, w.W, w.C)), bf((1, w.a, w.H, w.W, w.C))
    smp = gc.Sampler(kind=gc.GC_DDIM, pred_out=gc.GC_PRED_EPS)
    st = gc.gc_unipc_coeffs(gc.Sampler(kind=gc.GC_DDIM), 30, 6, 2, True)
    outs = {k: torch.empty_like(x0) for k in ("g0", "g1", "g2", "h0", "h1", "h2", "u0", "u1", "u2")}
    fgi = gc.gc_index_foreground(P)
    pairs = gc.gc_coverage_pairs(P, cams, bb)
    stale0 = gc.gc_coverage_init(P)
    for A in (A0, A1, A0):
        gc.gc_coverage_update(pairs, stale0, A, 2)
    stale = stale0.clone()
    stats = torch.empty((1, w.N, 4), dtype=torch.int32, device=DEV)
    sel = torch.empty(w.a, dtype=torch.int32, device=DEV)
    ws = torch.empty(gc.gc_coverage_workspace_bytes(), dtype=torch.uint8, device=DEV)
    # the fused update + selection / scoring (their last block reads what every block added)
    stale2 = stale0.clone()
    stats2, stats3 = torch.empty_like(stats), torch.empty_like(stats)
    sel2 = torch.empty(w.a, dtype=torch.int32, device=DEV)
    rot = [gc.gc_schedule_anchors(w.N, w.a, c) for c in range(3)]
    sc3 = torch.empty(len(rot), dtype=torch.int64, device=DEV)
    ws2 = torch.empty(gc.gc_coverage_workspace_bytes(), dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()

    def step():
        gc.gc_transport_reconstruct_geom(x0, new0, P, cams, bb, xt, A0, w.K, smp, 700, 666, x0_out=outs["g0"],
                                         x_next=outs["g1"], model_out=outs["g2"], stream=s)
        gc.gc_transport_reconstruct_geom(x0, new1, P, cams, bb, xt, A1, w.K, smp, 700, 666, x0_out=outs["h0"],
                                         x_next=outs["h1"], model_out=outs["h2"], fg_index=fgi, stream=s)
        gc.gc_transport_unipc(x0, new1, corr1, wts1, A1, st, x_prev=xprev, m_km2=m2, x0_out=outs["u0"],
                              x_c=outs["u1"], x_next=outs["u2"], index=idx1, stream=s)
        gc.gc_coverage_update(pairs, stale, A1, 2, stats=stats, stream=s)
        gc.gc_coverage_select(pairs, stale, w.a, forced=[w.N - 1], out=sel, workspace=ws, stream=s)
        gc.gc_coverage_update_select(pairs, stale2, A0, 2, w.a, forced=[1], stats=stats2, out=sel2, workspace=ws2,
                                     stream=s)
        gc.gc_coverage_update_score(pairs, stale2, A1, 2, rot, stats=stats3, out=sc3, workspace=ws2, stream=s)

    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in outs.items()}
    eager_stale, eager_stats, eager_sel = stale.clone(), stats.clone(), sel.clone()
    fused = (stale2, stats2, sel2, stats3, sc3)
    eager_fused = [t.clone() for t in fused]
    g = torch.cuda.CUDAGraph()
    stale.copy_(stale0)
    stale2.copy_(stale0)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        step()
    for rep in range(4):
        stale.copy_(stale0)
        stale2.copy_(stale0)
        for v in outs.values():
            v.fill_(float("nan"))
        for t in (stats, sel, stats2, sel2, stats3, sc3):
            t.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v.view(torch.int16), eager[k].view(torch.int16)), (rep, k)
        assert torch.equal(stale, eager_stale) and torch.equal(stats, eager_stats) and torch.equal(sel, eager_sel), rep
        for t, e in zip(fused, eager_fused):
            assert torch.equal(t, e), rep
        _ = (x0.float() * 2).sum().item()  # eager work between replays
