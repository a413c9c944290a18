"""Cached step with the correspondence computed on the fly.

gc_transport_step_geom / gc_transport_reconstruct_geom evaluate G_{A->v}
inside the step with the builder's own device code, so their outputs must
equal gc_build_correspondence followed by gc_transport_step /
gc_transport_reconstruct bit for bit (x0_out, x_next, model_out), and the
transported x0 must meet the oracle's bar (float32 1e-5, bfloat16 2e-2
against its unrounded values; unseen tokens and anchor rows bit-exact).
Covered: every workload at full size, every lane-group size G in {1, 2, 4,
8} with a <= 4 and a > 4, K in {1, 2, 4}, ragged grids (a partial last
block per view), channel counts whose vectors do not fill a lane group or
need two rounds, background positions, a = N.

Every case also runs the foreground launch (with gc_index_foreground's index
of the position maps), which must give the same bits, and checks that index
against its definition: a bit per token set iff its three position
components are finite, and the foreground tokens' {token, x, y, z} records
in the lists' tile order.  Separately: all-background maps (an empty list), more
(asset, anchor) cameras than the launch stages (B * a > 64: the blocked
launch runs), and token counts that end inside a 32-bit word and a chunk.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth.configs import C1, C2, C3, C4, C5

from conftest import latent_maps, listed_in_tile_order

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


def to_host(t, dtype):
    return t.cpu().numpy() if dtype == "f32" else t.view(torch.int16).cpu().numpy().view(np.uint16)


def bits(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def sampler_of(gc, w):
    if w.sampler == "ddim":
        return gc.Sampler(kind=gc.GC_DDIM, pred_out=gc.GC_PRED_EPS)
    return gc.Sampler(kind=gc.GC_FLOW_EULER, pred_out=gc.GC_PRED_VEL)


def step_of(w, k):
    return w.ddim_single if w.ddim_single else oracle.step_times(w.sampler, w.S, k)


def inputs(w, P, A, k, C=None, dtype=None, seed=None):
    dtype = dtype or w.dtype
    if seed is None and C is None:
        prev = synth.storage(synth.x0_state(w, P, k - 1), dtype)
        new = synth.storage(synth.x0_state(w, P, k, views=A), dtype)
        xt = synth.storage(synth.mix(synth.values(prev, dtype), synth.eps_noise(w, k), 0.6, 0.8), dtype)
        return prev, new, xt
    rs = np.random.default_rng(seed)
    B, N, H, W = P.shape[:4]
    C = C or w.C
    prev = synth.storage(0.5 * rs.standard_normal((B, N, H, W, C)).astype(np.float32), dtype)
    new = synth.storage(0.5 * rs.standard_normal((B, len(A), H, W, C)).astype(np.float32), dtype)
    xt = synth.storage(0.5 * rs.standard_normal((B, N, H, W, C)).astype(np.float32), dtype)
    return prev, new, xt


def expected_foreground(P):
    """The foreground index by its definition: (bit words as uint32, records
    int32 [n_fg, 4])."""
    flat = np.ascontiguousarray(P, np.float32).reshape(-1, 3)
    fg = np.isfinite(flat).all(-1)
    n = fg.size
    words = np.packbits(np.concatenate([fg, np.zeros((-n) % 32, bool)]).astype(np.uint8), bitorder="little")
    words = words.view(np.uint32) if words.size else np.zeros(0, np.uint32)
    tok = listed_in_tile_order(fg, P.shape[-3], P.shape[-2]) if n else np.zeros(0, np.int32)
    recs = np.concatenate([tok[:, None], flat[tok].view(np.int32)], 1) if tok.size else np.zeros((0, 4), np.int32)
    return words, recs


def check_foreground_index(gc, Pd, P):
    fgi = gc.gc_index_foreground(Pd)
    words, recs = expected_foreground(P)
    assert fgi.n_fg == recs.shape[0]
    np.testing.assert_array_equal(fgi.fg_bits.cpu().numpy().view(np.uint32)[:words.size], words)
    np.testing.assert_array_equal(fgi.fg_recs[:fgi.n_fg].cpu().numpy(), recs)
    return fgi


def compare(gc, w, P, cams_np, A, K, prev, new, xt, dtype, smp, t, tn, oracle_check=True):
    Pd = torch.from_numpy(np.ascontiguousarray(P)).to(DEV)
    cams = gc.camera_tensor(cams_np, DEV)
    bb = gc.gc_posmap_bbox(Pd, w.tol_frac)
    prev_d, new_d, xt_d = to_dev(prev, dtype), to_dev(new, dtype), to_dev(xt, dtype)
    corr, wts = gc.gc_build_correspondence(Pd, cams, A, K, bb)
    # transport only
    ref = gc.gc_transport_step(prev_d, new_d, corr, wts, A)
    got = gc.gc_transport_step_geom(prev_d, new_d, Pd, cams, bb, A, K)
    assert torch.equal(bits(got), bits(ref))
    # fused with the sampler step
    r0, r1, r2 = gc.gc_transport_reconstruct(prev_d, new_d, corr, wts, xt_d, A, smp, t, tn)
    g0, g1, g2 = gc.gc_transport_reconstruct_geom(prev_d, new_d, Pd, cams, bb, xt_d, A, K, smp, t, tn)
    assert torch.equal(bits(g0), bits(r0)) and torch.equal(bits(g1), bits(r1)) and torch.equal(bits(g2), bits(r2))
    # the foreground launch: the same bits
    fgi = check_foreground_index(gc, Pd, P)
    got_fg = gc.gc_transport_step_geom(prev_d, new_d, Pd, cams, bb, A, K, fg_index=fgi)
    assert torch.equal(bits(got_fg), bits(ref))
    f0, f1, f2 = gc.gc_transport_reconstruct_geom(prev_d, new_d, Pd, cams, bb, xt_d, A, K, smp, t, tn, fg_index=fgi)
    assert torch.equal(bits(f0), bits(r0)) and torch.equal(bits(f1), bits(r1)) and torch.equal(bits(f2), bits(r2))
    if oracle_check:
        corr_o, wts_o, nvis_o = oracle.build(P, cams_np, A, K, oracle.bbox(P, w.tol_frac))
        ex, state = oracle.transport(prev, new, corr_o, wts_o, A, dtype)
        out = to_host(got, dtype)
        vals = synth.values(out, dtype).astype(np.float64)
        assert np.abs(vals - ex).max() <= TOL[dtype]
        for s, u in enumerate(A):
            np.testing.assert_array_equal(out[:, u], new[:, s])
        targets = [v for v in range(P.shape[1]) if v not in A]
        for ti, v in enumerate(targets):
            unseen = nvis_o[:, ti] == 0
            np.testing.assert_array_equal(out[:, v][unseen], prev[:, v][unseen])
    return got


@pytest.mark.parametrize("w", [C1, C2, C3, C4, C5], ids=lambda w: w.name)
def test_geom_equals_stored_operator(gc, w):
    P = latent_maps(w.name)
    smp = sampler_of(gc, w)
    for c in (0, 1):
        A = list(w.fixed_anchors) if w.fixed_anchors else oracle.anchors(w.N, w.a, c)
        k = 3 + c
        t, tn = step_of(w, k)
        prev, new, xt = inputs(w, P, A, k)
        compare(gc, w, P, synth.batch_cameras(w), A, w.K, prev, new, xt, w.dtype, smp, t, tn)


@pytest.mark.parametrize("a,C,dtype", [(5, 16, "bf16"), (8, 16, "bf16"), (6, 16, "f32"), (5, 64, "bf16"),
                                       (7, 4, "f32"), (3, 8, "f32")])
def test_geom_many_anchors_every_group_size(gc, a, C, dtype):
    """Lanes per target token G = channel vectors (rounded up to a power of
    two, at most 8); each lane evaluates anchor slots j, j + G, ...:
    (5 | 8, 16 bf16): G = 2, up to four slots per lane; (6, 16 f32): G = 4,
    two slots; (5, 64 bf16): G = 8, one slot; (7, 4 f32): G = 1, every slot
    in one lane; (3, 8 f32): G = 2 with a slot past a in the second lane."""
    w = synth.shrink(C5, B=2, a=a)
    P = latent_maps(C5.name, B=2)
    A = oracle.anchors(w.N, a, 1)
    prev, new, xt = inputs(w, P, A, 0, C=C, dtype=dtype, seed=a * 100 + C)
    compare(gc, w, P, synth.batch_cameras(w), A, 4, prev, new, xt, dtype, sampler_of(gc, w), 0.6, 0.58)


@pytest.mark.parametrize("K", [1, 2])
def test_geom_fewer_taps(gc, K):
    w = C2
    P = latent_maps(w.name)
    A = oracle.anchors(w.N, w.a, 0)
    prev, new, xt = inputs(w, P, A, 4)
    t, tn = step_of(w, 4)
    compare(gc, w, P, synth.batch_cameras(w), A, K, prev, new, xt, w.dtype, sampler_of(gc, w), t, tn)


@pytest.mark.parametrize("C,dtype", [(4, "bf16"), (12, "f32"), (64, "bf16"), (40, "bf16"), (256, "f32")])
def test_geom_channel_layouts(gc, C, dtype):
    """C = 4 bf16: 8-byte vectors; C = 12 f32: 3 vectors per 4-lane group;
    C = 64 bf16: 8 vectors, two rounds; C = 40 bf16: 5 vectors, a partial
    second round; C = 256 f32: 64 vectors (the channel limit)."""
    w = C2
    P = latent_maps(w.name)
    A = oracle.anchors(w.N, w.a, 2)
    prev, new, xt = inputs(w, P, A, 0, C=C, dtype=dtype, seed=C)
    compare(gc, w, P, synth.batch_cameras(w), A, w.K, prev, new, xt, dtype, sampler_of(gc, w), 500, 460)


def test_geom_ragged_grid_and_background(gc):
    """A 37 x 53 grid (not a multiple of the 64 tokens a block covers), with
    holes punched into the position maps (background tokens and taps)."""
    w = C2
    rs = np.random.default_rng(5)
    P = latent_maps(w.name)[:, :, 5:42, 3:56].copy()
    P[rs.random(P.shape[:4]) < 0.15] = np.nan
    cams = synth.batch_cameras(w)
    for key in ("cx", "cy"):
        cams[key] = (cams[key] - (3.0 if key == "cx" else 5.0)).astype(np.float32)
    A = oracle.anchors(w.N, w.a, 1)
    prev, new, xt = inputs(w, P, A, 0, C=4, dtype="f32", seed=17)
    compare(gc, w, P, cams, A, w.K, prev, new, xt, "f32", sampler_of(gc, w), 700, 660)


def test_geom_all_views_anchors(gc):
    """a = N: every row is an anchor row (pure copy of the new prediction)."""
    w = synth.shrink(C1, a=4)
    P = latent_maps(C1.name)
    A = [0, 1, 2, 3]
    prev, new, xt = inputs(w, P, A, 0, C=4, dtype="f32", seed=3)
    got = compare(gc, w, P, synth.batch_cameras(w), A, 4, prev, new, xt, "f32", sampler_of(gc, w), 800, 760)
    np.testing.assert_array_equal(got.cpu().numpy(), new)


def test_geom_foreground_all_background(gc):
    """Position maps with no finite sample: the foreground list is empty and
    every target token keeps its state; both launches agree."""
    w = synth.shrink(C2, B=2)
    P = np.full((2, w.N, 24, 40, 3), np.nan, np.float32)
    A = oracle.anchors(w.N, w.a, 0)
    prev, new, xt = inputs(w, P, A, 0, C=8, dtype="bf16", seed=11)
    got = compare(gc, w, P, synth.batch_cameras(w), A, w.K, prev, new, xt, "bf16", sampler_of(gc, w), 600, 560)
    targets = [v for v in range(w.N) if v not in A]
    np.testing.assert_array_equal(to_host(got, "bf16")[:, targets], prev[:, targets])


def test_geom_foreground_many_cameras_falls_back(gc):
    """B * a = 22 * 3 = 66 (asset, anchor) cameras exceed what the foreground
    launch stages: the blocked launch runs and the bits are the same."""
    w = synth.shrink(C1, B=22, a=3)
    P = latent_maps(C1.name, B=22)
    A = [0, 1, 3]
    prev, new, xt = inputs(w, P, A, 0, C=4, dtype="f32", seed=22)
    compare(gc, w, P, synth.batch_cameras(w), A, 4, prev, new, xt, "f32", sampler_of(gc, w), 800, 760,
            oracle_check=False)


@pytest.mark.parametrize("shape", [(1, 3, 7, 9), (2, 5, 33, 31), (1, 1, 1, 1), (3, 4, 32, 33), (1, 2, 1, 1100)])
def test_foreground_index_ragged(gc, shape):
    """Token counts that end inside a 32-bit word and inside a 1024-token
    chunk, single tokens, random holes."""
    rs = np.random.default_rng(sum(shape))
    P = rs.standard_normal(shape + (3,)).astype(np.float32)
    P[rs.random(shape) < 0.4] = np.nan
    P[..., 1][rs.random(shape) < 0.1] = np.inf     # one non-finite component is enough
    check_foreground_index(gc, torch.from_numpy(P).to(DEV), P)
