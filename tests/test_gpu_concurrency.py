"""The library keeps no state between calls (error messages are per thread):
two host threads, each with its own HIP stream, buffers and coverage
workspace, issue cached steps concurrently -- the stored operator with its
index, the on-the-fly step (blocked and foreground launches), the fused
UniPC step and a coverage update +
greedy selection -- and every result equals the same call run alone, bit
for bit.  ctypes releases the interpreter lock around each foreign call, so
the two threads' calls overlap on the host as well as on the device."""
import threading

import numpy as np
import pytest
import torch

import synth
from synth.configs import C4

from conftest import latent_maps

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def gc():
    import paper_2608_13255_amd as gc
    return gc


def bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


def test_two_threads_two_streams(gc):
    w = C4
    P = torch.from_numpy(latent_maps(w.name)).to(DEV)
    cams = gc.camera_tensor(synth.batch_cameras(w), DEV)
    bb = gc.gc_posmap_bbox(P, w.tol_frac)
    smp = gc.Sampler(kind=gc.GC_DDIM, pred_out=gc.GC_PRED_EPS)
    st = gc.gc_unipc_coeffs(gc.Sampler(kind=gc.GC_DDIM), w.S, 6, 2, True)
    pairs = gc.gc_coverage_pairs(P, cams, bb)
    fgi = gc.gc_index_foreground(P)
    shape = (1, w.N, w.H, w.W, w.C)

    def make(seed, c):
        rs = np.random.default_rng(seed)
        bf = lambda sh: torch.from_numpy(rs.standard_normal(sh).astype(np.float32)).to(DEV).to(torch.bfloat16)
        A = gc.gc_schedule_anchors(w.N, w.a, c)
        corr, wts = gc.gc_build_correspondence(P, cams, A, w.K, bb)
        job = dict(A=A, corr=corr, wts=wts, idx=gc.gc_index_correspondence(corr), x0=bf(shape), xt=bf(shape),
                   xprev=bf(shape), m2=bf(shape), new=bf((1, w.a, w.H, w.W, w.C)),
                   ws=torch.empty(gc.gc_coverage_workspace_bytes(), dtype=torch.uint8, device=DEV),
                   stale0=gc.gc_coverage_init(P), stream=torch.cuda.Stream())
        job["out"] = {k: torch.empty_like(job["x0"])
                      for k in ("f0", "f1", "f2", "g0", "g1", "g2", "h0", "h1", "h2", "u0", "u1", "u2")}
        job["stale"] = job["stale0"].clone()
        job["stats"] = torch.empty((1, w.N, 4), dtype=torch.int32, device=DEV)
        job["sel"] = torch.empty(w.a, dtype=torch.int32, device=DEV)
        return job

    def run(j, reps):
        s, o = j["stream"], j["out"]
        for _ in range(reps):
            gc.gc_transport_reconstruct(j["x0"], j["new"], j["corr"], j["wts"], j["xt"], j["A"], smp, 700, 666,
                                        x0_out=o["f0"], x_next=o["f1"], model_out=o["f2"], index=j["idx"], stream=s)
            gc.gc_transport_reconstruct_geom(j["x0"], j["new"], P, cams, bb, j["xt"], j["A"], w.K, smp, 700, 666,
                                             x0_out=o["g0"], x_next=o["g1"], model_out=o["g2"], stream=s)
            gc.gc_transport_reconstruct_geom(j["x0"], j["new"], P, cams, bb, j["xt"], j["A"], w.K, smp, 700, 666,
                                             x0_out=o["h0"], x_next=o["h1"], model_out=o["h2"], fg_index=fgi,
                                             stream=s)
            gc.gc_transport_unipc(j["x0"], j["new"], j["corr"], j["wts"], j["A"], st, x_prev=j["xprev"],
                                  m_km2=j["m2"], x0_out=o["u0"], x_c=o["u1"], x_next=o["u2"], index=j["idx"],
                                  stream=s)
        gc.gc_coverage_update(pairs, j["stale"], j["A"], 2, stats=j["stats"], stream=s)
        gc.gc_coverage_select(pairs, j["stale"], w.a, forced=[w.N - 1], out=j["sel"], workspace=j["ws"], stream=s)
        s.synchronize()

    jobs = [make(1, 0), make(2, 1)]
    ref = []
    for j in jobs:   # each alone
        run(j, 1)
        ref.append([t.clone() for t in (*j["out"].values(), j["stale"], j["stats"], j["sel"])])
    for j in jobs:
        j["stale"].copy_(j["stale0"])
        for t in j["out"].values():
            t.fill_(float("nan"))
    torch.cuda.synchronize()
    errors = []

    def worker(j):
        try:
            run(j, 20)
        except Exception as e:   # surfaced in the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(j,)) for j in jobs]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for j, r in zip(jobs, ref):
        got = [*j["out"].values(), j["stale"], j["stats"], j["sel"]]
        for x, y in zip(got, r):
            assert torch.equal(bits(x), bits(y))
