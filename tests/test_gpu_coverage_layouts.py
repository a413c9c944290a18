"""Staleness update, greedy selection and set scores on random visibility
bits, bit-exact against the oracle, over the layouts the token kernels
distinguish:
  * rows of a multiple of 32 tokens, 16-byte aligned (two 16-byte accesses
    per lane);
  * rows of 16 mod 32 tokens (the last word of a row half full);
  * ragged rows (1961 tokens: bytewise accesses, a partial last word);
  * a staleness tensor that starts one byte past an aligned address
    (bytewise accesses although the rows are whole words);
  * more 2048-token items than reduction blocks (blocks stride over items);
  * 12 views (the coverage-histogram path at its largest) and 14 views (the
    per-round passes that serve more views), aligned and ragged.
Visibility bits are drawn at random rather than from geometry, with random
garbage in each row's padding bits, which every call ignores, and in the
rows (u, b, u), which the view itself covers anyway.  Staleness values cover
0, the saturation value 254 and background 255."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def gc():
    import paper_2608_13255_amd as gc
    return gc


def random_case(seed, B, N, H, W, density):
    rs = np.random.default_rng(seed)
    HW = H * W
    seen = (rs.random((N, B, N, HW)) < density).astype(np.uint8)
    wpr = (HW + 31) // 32
    packed = np.packbits(seen, axis=-1, bitorder="little")
    words = np.zeros((N, B, N, wpr * 4), np.uint8)
    words[..., :packed.shape[-1]] = packed
    words = words.view(np.uint32).copy()
    if HW % 32:   # garbage in the padding bits of each row's last word
        words[..., -1] |= rs.integers(0, 2**32, (N, B, N), dtype=np.uint64).astype(np.uint32) & ~np.uint32((1 << (HW % 32)) - 1)
    stale = rs.choice(np.array([0, 1, 2, 3, 7, 100, 252, 253, 254, 255], np.uint8), (B, N, H, W),
                      p=[.2, .15, .1, .1, .1, .05, .05, .05, .1, .1])
    return rs, seen.reshape(N, B, N, H, W), words, stale


def device_stale(stale, offset):
    """The staleness tensor at byte `offset` of a zeroed buffer (returned too)."""
    n = stale.size
    buf = torch.zeros(n + 64, dtype=torch.uint8, device=DEV)
    t = buf[offset:offset + n].view(stale.shape)
    t.copy_(torch.from_numpy(stale))
    return t, buf


CASES = {
    "aligned_words": (1, 3, 10, 32, 48, 0),
    "half_word_rows": (2, 2, 7, 12, 20, 0),
    "ragged_rows": (3, 2, 6, 37, 53, 0),
    "unaligned_pointer": (4, 2, 5, 32, 32, 1),
    "more_items_than_blocks": (5, 1, 5, 1024, 1024, 0),
    "twelve_views": (6, 2, 12, 24, 40, 0),        # the largest view count of the histogram path
    "fourteen_views": (7, 2, 14, 16, 24, 0),      # beyond it: one pass over the tokens per round
    "fourteen_views_ragged": (8, 1, 14, 13, 29, 3),
}


@pytest.mark.parametrize("key", list(CASES))
def test_update_select_score(gc, key):
    seed, B, N, H, W, offset = CASES[key]
    rs, seen, words, stale = random_case(seed, B, N, H, W, density=0.3)
    bits = torch.from_numpy(words.view(np.int32)).to(DEV)
    st_d, buf = device_stale(stale, offset)
    assert (st_d.data_ptr() % 16 != 0) == (offset != 0)
    ws = torch.empty(gc.gc_coverage_workspace_bytes(), dtype=torch.uint8, device=DEV)
    a = min(3, N)
    for forced in ([], [N - 1], list(range(a))):
        got = gc.gc_coverage_select(bits, st_d, a, forced=forced, workspace=ws).cpu().tolist()
        assert got == oracle.coverage_select(stale, seen, a, forced=forced), forced
    sets = oracle.rotation_sets(N, a) + [sorted(rs.choice(N, a, replace=False).tolist())]
    got = gc.gc_coverage_score(bits, st_d, sets, workspace=ws).cpu().numpy().view(np.uint64)
    np.testing.assert_array_equal(got, oracle.coverage_score(stale, seen, sets))
    st_o = stale
    for i, A in enumerate([[0], sorted(rs.choice(N, a, replace=False).tolist()), list(range(N)), [N - 1], [1]]):
        R = (1, 2, 254, 255, 3)[i]
        stats = gc.gc_coverage_update(bits, st_d, A, R)
        st_o, stats_o = oracle.coverage_update(st_o, seen, A, R)
        np.testing.assert_array_equal(st_d.cpu().numpy(), st_o, err_msg=f"step {i}")
        np.testing.assert_array_equal(stats.cpu().numpy().view(np.uint32), stats_o, err_msg=f"step {i}")
    # the bytes around the tensor are untouched
    around = torch.cat([buf[:offset], buf[offset + stale.size:]]).cpu().numpy()
    assert not around.any()


def test_saturation_runs(gc):
    """Staleness climbs to 254 and stays there; background stays 255."""
    B, N, H, W = 1, 3, 16, 16
    rs, seen, words, stale = random_case(9, B, N, H, W, density=0.0)
    stale[...] = 250
    stale[0, 1, :2] = 255
    bits = torch.from_numpy(words.view(np.int32)).to(DEV)
    st_d, _ = device_stale(stale, 0)
    st_o = stale
    for _ in range(6):
        stats = gc.gc_coverage_update(bits, st_d, [0], 254)
        st_o, stats_o = oracle.coverage_update(st_o, seen, [0], 254)
        np.testing.assert_array_equal(st_d.cpu().numpy(), st_o)
        np.testing.assert_array_equal(stats.cpu().numpy().view(np.uint32), stats_o)
    got = st_d.cpu().numpy()
    assert (got[0, 0] == 0).all() and (got[0, 2] == 254).all() and (got[0, 1, :2] == 255).all()


@pytest.mark.parametrize("key", list(CASES))
def test_fused_update_select_score(gc, key):
    """gc_coverage_update_select / _score (the staleness step and the next
    step's choice in one pass) equal the oracle's update followed by its
    selection / scores on the updated staleness: staleness bytes, statistics
    and results bit for bit, over a few steps, whatever the workspace held."""
    seed, B, N, H, W, offset = CASES[key]
    rs, seen, words, stale = random_case(100 + seed, B, N, H, W, density=0.3)
    bits = torch.from_numpy(words.view(np.int32)).to(DEV)
    st_d, buf = device_stale(stale, offset)
    ws = torch.empty(gc.gc_coverage_workspace_bytes(), dtype=torch.uint8, device=DEV)
    a = min(3, N)
    sets = oracle.rotation_sets(N, a) + [sorted(rs.choice(N, a, replace=False).tolist())]
    st_o = stale
    steps = [([0], 1, []), (sorted(rs.choice(N, a, replace=False).tolist()), 2, [N - 1]), (list(range(N)), 254, []),
             ([N - 1], 3, list(range(a))), ([1], 2, [0])]
    for i, (A, R, forced) in enumerate(steps):
        ws.copy_(torch.randint(0, 256, ws.shape, dtype=torch.uint8, generator=torch.Generator().manual_seed(i)))
        if i % 2 == 0:
            stats, sel = gc.gc_coverage_update_select(bits, st_d, A, R, a, forced=forced, workspace=ws)
            st_o, stats_o = oracle.coverage_update(st_o, seen, A, R)
            assert sel.cpu().tolist() == oracle.coverage_select(st_o, seen, a, forced=forced), f"step {i}"
        else:
            stats, sc = gc.gc_coverage_update_score(bits, st_d, A, R, sets, workspace=ws)
            st_o, stats_o = oracle.coverage_update(st_o, seen, A, R)
            np.testing.assert_array_equal(sc.cpu().numpy().view(np.uint64), oracle.coverage_score(st_o, seen, sets),
                                          err_msg=f"step {i}")
        np.testing.assert_array_equal(st_d.cpu().numpy(), st_o, err_msg=f"step {i}")
        np.testing.assert_array_equal(stats.cpu().numpy().view(np.uint32), stats_o, err_msg=f"step {i}")
    around = torch.cat([buf[:offset], buf[offset + stale.size:]]).cpu().numpy()
    assert not around.any()
