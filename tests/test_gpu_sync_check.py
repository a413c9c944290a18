"""GC_SYNC_CHECK=1: every entry point synchronises its stream and checks the
execution status before returning.  The setting is read once per process, so
one child process runs a whole cached step through the entry points with it
set and compares against the same calls in this process."""
import os
import subprocess
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import numpy as np, torch, sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import paper_2608_13255_amd as gc, oracle, synth
from conftest import latent_maps
w = synth.CONFIGS["hunyuan_torus_6v_64"]
P = torch.from_numpy(latent_maps(w.name)).cuda()
cams = gc.camera_tensor(synth.batch_cameras(w), "cuda")
bb = gc.gc_posmap_bbox(P, w.tol_frac)
A = [0, 3]
corr, wts = gc.gc_build_correspondence(P, cams, A, 4, bb)
idx = gc.gc_index_correspondence(corr)
g = torch.Generator().manual_seed(1)
prev = torch.randn((1, 6, 64, 64, 4), generator=g).cuda()
new = torch.randn((1, 2, 64, 64, 4), generator=g).cuda()
xt = torch.randn((1, 6, 64, 64, 4), generator=g).cuda()
smp = gc.Sampler(kind=gc.GC_DDIM, pred_out=gc.GC_PRED_EPS)
outs = list(gc.gc_transport_reconstruct(prev, new, corr, wts, xt, A, smp, 700, 660, index=idx))
outs += list(gc.gc_transport_unipc(prev, new, corr, wts, A, gc.gc_unipc_coeffs(gc.Sampler(kind=gc.GC_DDIM), 10, 4, 2, True),
                                   x_prev=xt, m_km2=prev, index=idx))
outs += list(gc.gc_transport_reconstruct_geom(prev, new, P, cams, bb, xt, A, 4, smp, 700, 660))
fgi = gc.gc_index_foreground(P)
outs += list(gc.gc_transport_reconstruct_geom(prev, new, P, cams, bb, xt, A, 4, smp, 700, 660, fg_index=fgi))
ust = gc.gc_unipc_coeffs(gc.Sampler(kind=gc.GC_DDIM), 10, 4, 2, True)
outs += list(gc.gc_transport_unipc_geom(prev, new, P, cams, bb, A, 4, ust, x_prev=xt, m_km2=prev, fg_index=fgi))
outs += [fgi.fg_bits, fgi.fg_recs[:fgi.n_fg]]
pairs = gc.gc_coverage_pairs(P, cams, bb)
stale = gc.gc_coverage_init(P)
stats = gc.gc_coverage_update(pairs, stale, A, 2)
sel = gc.gc_coverage_select(pairs, stale, 2)
st = gc.gc_unipc_coeffs(gc.Sampler(kind=gc.GC_DDIM), 10, 3, 2, True)
xc, xn = gc.gc_unipc_update(st, outs[0], x_prev=xt, m_km2=prev, m_km1=prev)
stats2, sel2 = gc.gc_coverage_update_select(pairs, stale, sel.tolist(), 2, 2, forced=[1])
stats3, sc3 = gc.gc_coverage_update_score(pairs, stale, sel2.tolist(), 2, [[0, 3], [1, 4], [2, 5]])
outs += [xc, xn, stats, sel, stats2, sel2, stats3, sc3, stale]
torch.save([o.cpu() for o in outs], sys.argv[1])
print("OK")
"""


def test_sync_check_mode_matches(tmp_path):
    script = tmp_path / "child.py"
    script.write_text(CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests")))
    res = {}
    for flag in ("0", "1"):
        out = tmp_path / f"out{flag}.pt"
        env = dict(os.environ, GC_SYNC_CHECK=flag)
        r = subprocess.run([sys.executable, str(script), str(out)], env=env, capture_output=True, text=True,
                           timeout=240)
        assert r.returncode == 0 and "OK" in r.stdout, r.stderr[-2000:]
        import torch
        res[flag] = torch.load(out, weights_only=True)
    for a, b in zip(res["0"], res["1"]):
        assert np.array_equal(a.numpy(), b.numpy())
