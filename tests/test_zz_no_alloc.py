"""The allocation-free visible-token index (gc_index_correspondence_noalloc)
through the C ABI against gc_index_correspondence with a caller workspace:
bits, list and count identical, on two calls in a row, the second with a
smaller input (the library's scratch keeps the first call's contents)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from synth.configs import C2, C5

from conftest import latent_maps, listed_in_tile_order

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _operator(gc, w, c):
    P = torch.from_numpy(latent_maps(w.name)).to(DEV)
    A = oracle.anchors(w.N, w.a, c)
    corr, _ = gc.gc_build_correspondence(P, gc.camera_tensor(synth.batch_cameras(w), DEV), A, w.K,
                                         gc.gc_posmap_bbox(P, w.tol_frac))
    return corr


def _index(gc, corr, noalloc):
    L = gc.lib()
    a = corr.shape[-1]
    n = corr.numel() // a
    n_views, H, W = corr.shape[0] * corr.shape[1], corr.shape[2], corr.shape[3]
    bits = torch.full(((n + 31) // 32,), -1, dtype=torch.int32, device=DEV)
    lst = torch.full((n,), -7, dtype=torch.int32, device=DEV)
    nv = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    s = torch.cuda.current_stream().cuda_stream
    if noalloc:
        rc = L.gc_index_correspondence_noalloc(corr.data_ptr(), n_views, H, W, a, bits.data_ptr(), lst.data_ptr(),
                                               nv.data_ptr(), s)
    else:
        ws = torch.empty(int(L.gc_index_workspace_bytes(n)), dtype=torch.uint8, device=DEV)
        rc = L.gc_index_correspondence(corr.data_ptr(), n_views, H, W, a, bits.data_ptr(), lst.data_ptr(),
                                       nv.data_ptr(), ws.data_ptr(), ws.numel(), s)
    assert rc == 0, L.gc_last_error().decode()
    torch.cuda.synchronize()
    k = int(nv.item())
    return bits.cpu().numpy(), lst[:k].cpu().numpy(), k


def test_noalloc_index_equals_workspace_index_twice():
    import paper_2608_13255_amd as gc
    for w, c in ((C5, 1), (C2, 2)):       # the second input is smaller than the first
        print(f"noalloc index: {w.name}, anchor set {c}", flush=True)
        corr = _operator(gc, w, c)
        b0, l0, n0 = _index(gc, corr, noalloc=False)
        b1, l1, n1 = _index(gc, corr, noalloc=True)
        assert n1 == n0 > 0
        np.testing.assert_array_equal(b1, b0)
        np.testing.assert_array_equal(l1, l0)
        # the list is the non-zero rows of the operator, in the lists' tile order
        rows = listed_in_tile_order(corr.view(-1, corr.shape[-1]).cpu().numpy().any(axis=1), corr.shape[2],
                                    corr.shape[3])
        np.testing.assert_array_equal(l1, rows)
