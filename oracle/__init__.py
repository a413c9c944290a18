"""Oracle for GeoCache's per-step cross-view transport -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library (paper_2608_13255_amd) never
imports it and shares no code with it.

Thin numpy/ctypes marshalling over oracle.c (plain single-threaded C, double
precision for continuous outputs, float where a float decides an integer).
Every arithmetic step lives in oracle.c and cites the paper there; this file
adds only the trajectory loops, which string the C steps together in the
order of Sec. 3.2 ("Loop order") and Sec. 3.2 ("Drift-bounding schedule"),
and the integer rule of the coverage schedule's anchor gaps (forced_views,
advance_gaps; Sec. 5, adaptive anchor selection).

Latent arrays are float32 for dtype "f32" and uint16 bfloat16 bit patterns
for dtype "bf16".
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

DTYPES = {"f32": 0, "bf16": 1}
PRED = {"none": 0, "eps": 1, "v": 2, "vel": 3}
KIND = {"ddim": 0, "flow": 1}
FULL_RULE = {"periodic": 0, "head_mid_tail": 1, "head_tail_e": 2}

_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_vp = ctypes.c_void_p


def lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "liboracle.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `make -C oracle`")
        L = ctypes.CDLL(path)
        L.orc_downsample.argtypes = [_f32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int, _f32p]
        L.orc_bbox.argtypes = [_f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                               ctypes.c_float, _f32p]
        L.orc_build.argtypes = [_f32p, _i32p, _f32p, _f32p, _f32p, ctypes.c_int, ctypes.c_int,
                                ctypes.c_int, ctypes.c_int, _i32p, ctypes.c_int, ctypes.c_int, _f32p,
                                _i32p, _f64p, _i32p]
        L.orc_transport.argtypes = [_vp, _vp, _i32p, _f64p, _i32p, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, _f64p, _vp]
        L.orc_reconstruct.argtypes = [_vp, _vp, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_double,
                                      ctypes.c_double, ctypes.c_double, _f64p, _f64p]
        L.orc_alpha_bar.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_int]
        L.orc_alpha_bar.restype = ctypes.c_double
        L.orc_anchors.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int64, _i32p]
        L.orc_full_steps.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _u8p]
        L.orc_ddim_timesteps.argtypes = [ctypes.c_int, ctypes.c_int, _i32p]
        L.orc_store.argtypes = [_f64p, ctypes.c_int64, ctypes.c_int, _vp]
        L.orc_unipc_coeffs.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double, _i32p, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, ctypes.c_int, _f64p]
        L.orc_unipc_coeffs.restype = ctypes.c_int
        L.orc_unipc_apply.argtypes = [_vp, _vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_int, _f64p, _f64p, _f64p]
        L.orc_unipc_apply.restype = ctypes.c_int
        _u32p = ctypes.POINTER(ctypes.c_uint32)
        _u64p = ctypes.POINTER(ctypes.c_uint64)
        L.orc_cov_init.argtypes = [_f32p, ctypes.c_int64, _u8p]
        L.orc_cov_update.argtypes = [_u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int64, _i32p, ctypes.c_int,
                                     ctypes.c_int, _u8p, _u32p]
        L.orc_cov_gains.argtypes = [_u8p, _u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int64, _u8p, _u64p]
        L.orc_cov_select.argtypes = [_u8p, _u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int, _i32p,
                                     ctypes.c_int, _i32p]
        L.orc_refresh_due.argtypes = [_u32p, ctypes.c_int, ctypes.c_int, ctypes.c_double]
        L.orc_cov_score.argtypes = [_u8p, _u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int64, _i32p, ctypes.c_int,
                                    ctypes.c_int, _u64p]
        for f in ("orc_cov_init", "orc_cov_update", "orc_cov_gains", "orc_cov_select", "orc_refresh_due",
                  "orc_cov_score"):
            getattr(L, f).restype = ctypes.c_int
        for f in ("orc_downsample", "orc_bbox", "orc_build", "orc_transport", "orc_reconstruct",
                  "orc_anchors", "orc_full_steps", "orc_ddim_timesteps", "orc_store"):
            getattr(L, f).restype = ctypes.c_int
        _LIB = L
    return _LIB


def _p(a, t):
    return a.ctypes.data_as(t)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (code {rc})")


def _storage_dtype(dtype):
    return np.float32 if dtype == "f32" else np.uint16


# --------------------------------------------------------------------------
# steps
# --------------------------------------------------------------------------

def downsample(hi: np.ndarray, f: int) -> np.ndarray:
    """Area-downsample position maps [..., Hr, Wr, 3] by f (see oracle.c O1)."""
    hi = np.ascontiguousarray(hi, np.float32)
    lead = hi.shape[:-3]
    Hr, Wr = hi.shape[-3], hi.shape[-2]
    M = int(np.prod(lead)) if lead else 1
    out = np.empty(lead + (Hr // f, Wr // f, 3), np.float32)
    _check(lib().orc_downsample(_p(hi, _f32p), M, Hr, Wr, f, _p(out, _f32p)), "downsample")
    return out


def bbox(pos: np.ndarray, tol_frac: float = 0.01) -> np.ndarray:
    """Per-asset bbox + squared tolerance, [B][8] (see oracle.c O2)."""
    pos = np.ascontiguousarray(pos, np.float32)
    B, N, H, W, _ = pos.shape
    out = np.empty((B, 8), np.float32)
    _check(lib().orc_bbox(_p(pos, _f32p), B, N, H, W, tol_frac, _p(out, _f32p)), "bbox")
    return out


def _cam_arrays(cams: Dict[str, np.ndarray], B: int, N: int):
    model = np.ascontiguousarray(np.broadcast_to(cams["model"], (B, N)), np.int32)
    R = np.ascontiguousarray(np.broadcast_to(cams["R"], (B, N, 3, 3)), np.float32)
    t = np.ascontiguousarray(np.broadcast_to(cams["t"], (B, N, 3)), np.float32)
    k = np.ascontiguousarray(np.stack([np.broadcast_to(cams[n], (B, N)) for n in ("fx", "fy", "cx", "cy")],
                                      -1), np.float32)
    return model, R, t, k


def build(pos: np.ndarray, cams: Dict[str, np.ndarray], anchors: Sequence[int], K: int,
          bbox_arr: np.ndarray):
    """Correspondence G_{A->v} for every non-anchor view (see oracle.c O3).

    Returns (corr int32 [B][N-a][H][W][a], weights float64 [B][N-a][H][W][a][K],
    nvis int32 [B][N-a][H][W])."""
    pos = np.ascontiguousarray(pos, np.float32)
    B, N, H, W, _ = pos.shape
    A = np.ascontiguousarray(anchors, np.int32)
    a = A.shape[0]
    model, R, t, k = _cam_arrays(cams, B, N)
    bb = np.ascontiguousarray(bbox_arr, np.float32)
    NT = N - a
    corr = np.zeros((B, NT, H, W, a), np.int32)
    wts = np.zeros((B, NT, H, W, a, K), np.float64)
    nvis = np.zeros((B, NT, H, W), np.int32)
    _check(lib().orc_build(_p(pos, _f32p), _p(model, _i32p), _p(R, _f32p), _p(t, _f32p), _p(k, _f32p),
                           B, N, H, W, _p(A, _i32p), a, K, _p(bb, _f32p), _p(corr, _i32p),
                           _p(wts, _f64p), _p(nvis, _i32p)), "build")
    return corr, wts, nvis


def transport(x0_prev: np.ndarray, x0_anchor_new: np.ndarray, corr: np.ndarray, weights: np.ndarray,
              anchors: Sequence[int], dtype: str) -> Tuple[np.ndarray, np.ndarray]:
    """Delta transport, Eq. 1 (see oracle.c O4).

    Returns (x0 float64 unrounded [B][N][H][W][C], x0 state in storage dtype)."""
    sd = _storage_dtype(dtype)
    x0_prev = np.ascontiguousarray(x0_prev, sd)
    x0_anchor_new = np.ascontiguousarray(x0_anchor_new, sd)
    B, N, H, W, C = x0_prev.shape
    A = np.ascontiguousarray(anchors, np.int32)
    a = A.shape[0]
    K = weights.shape[-1]
    corr = np.ascontiguousarray(corr, np.int32)
    weights = np.ascontiguousarray(weights, np.float64)
    assert x0_anchor_new.shape == (B, a, H, W, C)
    assert corr.shape == (B, N - a, H, W, a) and weights.shape == (B, N - a, H, W, a, K)
    exact = np.empty(x0_prev.shape, np.float64)
    state = np.empty(x0_prev.shape, sd)
    _check(lib().orc_transport(x0_prev.ctypes.data, x0_anchor_new.ctypes.data, _p(corr, _i32p),
                               _p(weights, _f64p), _p(A, _i32p), a, B, N, H, W, C, K, DTYPES[dtype],
                               _p(exact, _f64p), state.ctypes.data), "transport")
    return exact, state


def reconstruct(x_t: np.ndarray, x0: np.ndarray, dtype: str, kind: str, t: float, t_next: float,
                pred: str = "none", T: int = 1000, beta_start: float = 1e-4,
                beta_end: float = 0.02) -> Tuple[np.ndarray, np.ndarray]:
    """Sampler-consistent reconstruction (see oracle.c O5).

    Returns (x_next float64, model_out float64 or None)."""
    sd = _storage_dtype(dtype)
    x_t = np.ascontiguousarray(x_t, sd)
    x0 = np.ascontiguousarray(x0, sd)
    assert x_t.shape == x0.shape
    xn = np.empty(x_t.shape, np.float64)
    mo = np.empty(x_t.shape, np.float64) if pred != "none" else None
    _check(lib().orc_reconstruct(x_t.ctypes.data, x0.ctypes.data, x_t.size, DTYPES[dtype], KIND[kind],
                                 PRED[pred], T, beta_start, beta_end, float(t), float(t_next),
                                 _p(xn, _f64p), _p(mo, _f64p) if mo is not None else None),
           "reconstruct")
    return xn, mo


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values into the storage dtype."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, _storage_dtype(dtype))
    _check(lib().orc_store(_p(x, _f64p), x.size, DTYPES[dtype], out.ctypes.data), "store")
    return out


def alpha_bar(t: int, T: int = 1000, beta_start: float = 1e-4, beta_end: float = 0.02) -> float:
    return lib().orc_alpha_bar(T, beta_start, beta_end, int(t))


def unipc_coeffs(S: int, k: int, order: int = 2, corrector: bool = True, T: int = 1000,
                 beta_start: float = 1e-4, beta_end: float = 0.02) -> np.ndarray:
    """Coefficients of UniPC step k of an S-step trailing-timestep trajectory
    (see oracle.c O8): [use_corrector, pc, pp, c_xprev, c_mk2, c_mk1, c_mk,
    p_xc, p_mk1, p_mk]."""
    ts = np.ascontiguousarray(ddim_timesteps(S, T), np.int32)
    c = np.zeros(10, np.float64)
    _check(lib().orc_unipc_coeffs(T, beta_start, beta_end, _p(ts, _i32p), S, k, order, int(corrector),
                                  _p(c, _f64p)), "unipc_coeffs")
    return c


def unipc_apply(coeffs: np.ndarray, x_cur, x_prev, m_km2, m_km1, m_k, dtype: str):
    """One UniPC update in double; returns (x_c, x_next) float64."""
    sd = _storage_dtype(dtype)
    arrs = [None if a is None else np.ascontiguousarray(a, sd) for a in (x_cur, x_prev, m_km2, m_km1, m_k)]
    n = arrs[4].size
    xc = np.empty(arrs[4].shape, np.float64)
    xn = np.empty(arrs[4].shape, np.float64)
    c = np.ascontiguousarray(coeffs, np.float64)
    _check(lib().orc_unipc_apply(*[None if a is None else a.ctypes.data for a in arrs], n, DTYPES[dtype],
                                 _p(c, _f64p), _p(xc, _f64p), _p(xn, _f64p)), "unipc_apply")
    return xc, xn


# --------------------------------------------------------------------------
# schedule
# --------------------------------------------------------------------------

def anchors(N: int, a: int, c: int) -> List[int]:
    out = np.empty(a, np.int32)
    _check(lib().orc_anchors(N, a, c, _p(out, _i32p)), "anchors")
    return out.tolist()


def full_steps(rule: str, S: int, E: int = 0) -> List[int]:
    out = np.zeros(S, np.uint8)
    _check(lib().orc_full_steps(FULL_RULE[rule], S, E, _p(out, _u8p)), "full_steps")
    return out.tolist()


def ddim_timesteps(S: int, T: int = 1000) -> List[int]:
    out = np.empty(S + 1, np.int32)
    _check(lib().orc_ddim_timesteps(T, S, _p(out, _i32p)), "ddim_timesteps")
    return out.tolist()


def step_times(kind: str, S: int, k: int, T: int = 1000) -> Tuple[float, float]:
    """(t, t_next) of sampler step k: DDIM integer timesteps, flow sigmas 1 - k/S."""
    if kind == "ddim":
        ts = ddim_timesteps(S, T)
        return float(ts[k]), float(ts[k + 1])
    return 1.0 - k / S, 1.0 - (k + 1) / S


# --------------------------------------------------------------------------
# trajectory (Sec. 3.2: loop order and drift-bounding schedule)
# --------------------------------------------------------------------------

def trajectory(x_t0: np.ndarray, stub, pos: np.ndarray, cams, K: int, tol_frac: float, dtype: str,
               kind: str, S: int, full: Sequence[int], a: int, steps: int = None,
               times=None):
    """Run `steps` sampler steps (default S) of the cached loop.

    stub(k, views) -> x0 storage array [B][len(views)][H][W][C]: the denoiser's
    prediction at step k for the given views (a synthetic stand-in).
    At a full step every view is predicted and only the reconstruction runs;
    at a cached step c the anchors A_c are predicted, their increment against
    the stored x0 is transported to the other views, and every view is then
    reconstructed.  x0(t) of all N views becomes the next reference.

    Returns the list of per-step records: anchors, the cached-step counter c
    after the step, the stored x_t and x0 (storage dtype) and their unrounded
    double values x_t_exact and x0_exact."""
    steps = S if steps is None else steps
    B, N = pos.shape[0], pos.shape[1]
    bb = bbox(pos, tol_frac)
    cache = {}
    x_t = x_t0
    x0_store = None
    c = 0
    out = []
    for k in range(steps):
        t, tn = times(k) if times is not None else step_times(kind, S, k)
        if full[k] or x0_store is None:
            x0_new = stub(k, list(range(N)))
            x0_state = x0_new
            x0_exact = (x0_new if dtype == "f32" else _bf16_values(x0_new)).astype(np.float64)
            A = list(range(N))
        else:
            A = anchors(N, a, c)
            c += 1
            key = tuple(A)
            if key not in cache:
                corr, w, _ = build(pos, cams, A, K, bb)
                cache[key] = (corr, w)
            corr, w = cache[key]
            x0_exact, x0_state = transport(x0_store, stub(k, A), corr, w, A, dtype)
        xn, _ = reconstruct(x_t, x0_state, dtype, kind, t, tn)
        x_t = store(xn, dtype)
        x0_store = x0_state
        out.append({"k": k, "anchors": A, "c": c, "x_t": x_t, "x0": x0_state, "x_t_exact": xn,
                    "x0_exact": x0_exact})
    return out


def trajectory_unipc(x_t0: np.ndarray, stub, pos: np.ndarray, cams, K: int, tol_frac: float, dtype: str, S: int,
                     full: Sequence[int], a: int, order: int = 2, corrector: bool = True, steps: int = None):
    """The cached loop with a UniPC data-prediction solver (see oracle.c O8):
    the x0 store is the solver's history.  Per step: x0 of every view (from
    the stub at a full step, by Eq. 1 at a cached step), then the UniPC
    corrector + predictor.  Returns per-step records like trajectory()
    plus the corrected sample x_c (exact and stored)."""
    steps = S if steps is None else steps
    B, N = pos.shape[0], pos.shape[1]
    bb = bbox(pos, tol_frac)
    cache = {}
    x_t, x_prev, m1, m2 = x_t0, None, None, None
    c = 0
    out = []
    for k in range(steps):
        if full[k] or m1 is None:
            mk = stub(k, list(range(N)))
            mk_exact = (mk if dtype == "f32" else _bf16_values(mk)).astype(np.float64)
            A = list(range(N))
        else:
            A = anchors(N, a, c)
            c += 1
            key = tuple(A)
            if key not in cache:
                corr, w, _ = build(pos, cams, A, K, bb)
                cache[key] = (corr, w)
            corr, w = cache[key]
            mk_exact, mk = transport(m1, stub(k, A), corr, w, A, dtype)
        co = unipc_coeffs(S, k, order, corrector)
        xc, xn = unipc_apply(co, x_t, x_prev, m2, m1, mk, dtype)
        xc_s = store(xc, dtype)
        x_t = store(xn, dtype)
        x_prev, m2, m1 = xc_s, m1, mk
        out.append({"k": k, "anchors": A, "c": c, "x_t": x_t, "x0": mk, "x_c": xc_s, "x_t_exact": xn,
                    "x0_exact": mk_exact, "x_c_exact": xc})
    return out


# --------------------------------------------------------------------------
# token staleness and the coverage-driven schedule (see oracle.c O9)
# --------------------------------------------------------------------------

def coverage_pairs(pos: np.ndarray, cams, K: int, bbox_arr: np.ndarray) -> np.ndarray:
    """seen[u][b][v][h][w] (uint8 0/1): anchor u alone sees token (v, h, w)
    -- a non-zero O3 word of the build for the anchor set {u}."""
    B, N, H, W, _ = pos.shape
    seen = np.zeros((N, B, N, H, W), np.uint8)
    for u in range(N):
        corr, _, _ = build(pos, cams, [u], K, bbox_arr)
        targets = [v for v in range(N) if v != u]
        for ti, v in enumerate(targets):
            seen[u, :, v] = corr[:, ti, :, :, 0] != 0
    return seen


def coverage_init(pos: np.ndarray) -> np.ndarray:
    """Staleness state [B][N][H][W] uint8: 0 for foreground, 255 for background."""
    pos = np.ascontiguousarray(pos, np.float32)
    out = np.empty(pos.shape[:-1], np.uint8)
    _check(lib().orc_cov_init(_p(pos, _f32p), out.size, _p(out, _u8p)), "cov_init")
    return out


def coverage_update(stale: np.ndarray, seen: np.ndarray, anchors: Sequence[int], R: int):
    """One step with anchor set `anchors` (all views for a full step):
    returns (new staleness, stats uint32 [B][N][4] = foreground tokens,
    tokens with staleness >= R, sum, max)."""
    B, N = stale.shape[:2]
    HW = int(np.prod(stale.shape[2:]))
    st = np.ascontiguousarray(stale, np.uint8).copy()
    sn = np.ascontiguousarray(seen, np.uint8)
    A = np.ascontiguousarray(anchors, np.int32)
    stats = np.zeros((B, N, 4), np.uint32)
    _check(lib().orc_cov_update(_p(sn, _u8p), B, N, HW, _p(A, _i32p), A.size, R, _p(st, _u8p),
                                stats.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))), "cov_update")
    return st, stats


def coverage_gains(stale: np.ndarray, seen: np.ndarray, chosen: Sequence[int]) -> np.ndarray:
    """Weighted coverage gain of every view given the chosen views (uint64 [N])."""
    B, N = stale.shape[:2]
    HW = int(np.prod(stale.shape[2:]))
    ch = np.zeros(N, np.uint8)
    ch[list(chosen)] = 1
    g = np.zeros(N, np.uint64)
    _check(lib().orc_cov_gains(_p(np.ascontiguousarray(seen, np.uint8), _u8p),
                               _p(np.ascontiguousarray(stale, np.uint8), _u8p), B, N, HW, _p(ch, _u8p),
                               g.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))), "cov_gains")
    return g


def coverage_select(stale: np.ndarray, seen: np.ndarray, a: int, forced: Sequence[int] = ()) -> List[int]:
    """Greedy weighted maximum coverage: forced views first, then a views in all; sorted."""
    B, N = stale.shape[:2]
    HW = int(np.prod(stale.shape[2:]))
    f = np.ascontiguousarray(list(forced) or [0], np.int32)
    out = np.empty(a, np.int32)
    _check(lib().orc_cov_select(_p(np.ascontiguousarray(seen, np.uint8), _u8p),
                                _p(np.ascontiguousarray(stale, np.uint8), _u8p), B, N, HW, a, _p(f, _i32p),
                                len(forced), _p(out, _i32p)), "cov_select")
    return out.tolist()


def coverage_score(stale: np.ndarray, seen: np.ndarray, sets: Sequence[Sequence[int]]) -> np.ndarray:
    """Weighted coverage (1 + staleness over covered foreground tokens) of each candidate set (uint64 [M])."""
    B, N = stale.shape[:2]
    HW = int(np.prod(stale.shape[2:]))
    S = np.ascontiguousarray(sets, np.int32)
    M, a = S.shape
    out = np.zeros(M, np.uint64)
    _check(lib().orc_cov_score(_p(np.ascontiguousarray(seen, np.uint8), _u8p),
                               _p(np.ascontiguousarray(stale, np.uint8), _u8p), B, N, HW, _p(S, _i32p), M, a,
                               out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))), "cov_score")
    return out


def rotation_sets(N: int, a: int) -> List[List[int]]:
    """The rotation's distinct anchor sets, in order of first appearance."""
    out = []
    for c in range(N):
        A = anchors(N, a, c)
        if A not in out:
            out.append(A)
    return out


def refresh_due(stats: np.ndarray, tau: float) -> bool:
    st = np.ascontiguousarray(stats, np.uint32)
    B, N = st.shape[:2]
    rc = lib().orc_refresh_due(st.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), B, N, tau)
    if rc < 0:
        raise ValueError("oracle refresh_due rejected its arguments")
    return bool(rc)


def forced_views(gap: Sequence[int], a: int, max_gap: int) -> List[int]:
    """Views that must be anchors of the next cached step (the limitations
    section's adaptive anchor selection, as read in oracle.c O9): every view
    whose gap -- cached steps since it was last an anchor -- has reached
    max_gap (max_gap 0: no view is forced), the longest gap first, equal gaps
    in ascending view order, at most a of them."""
    if max_gap <= 0:
        return []
    due = [v for v in range(len(gap)) if gap[v] >= max_gap]
    due.sort(key=lambda v: (-gap[v], v))
    return due[:a]


def advance_gaps(gap: Sequence[int], views: Sequence[int], full: bool) -> List[int]:
    """Every view's gap after a step: 0 for the step's anchors (every view at
    a full step, which predicts all of them), one more for the others."""
    return [0 if (full or v in views) else g + 1 for v, g in enumerate(gap)]


def schedule_adaptive(seen: np.ndarray, stale0: np.ndarray, full: Sequence[int], a: int, policy: str = "coverage",
                      max_gap: int = 0, tau: float = None, R: int = 2, steps: int = None):
    """The coverage-driven schedule alone (see oracle.c O9); it depends on
    the visibility pairs and the staleness only, never on latent values.
    Step k is full when full[k] says so, on the first step, or when
    refresh_due(stats of the previous step, tau).  A cached step's anchors
    come from the rotation over the cached-step counter (policy "rotate"),
    from the rotation's distinct sets, the one with the largest
    coverage_score (policy "rotation_coverage", ties to the earlier set), or
    from coverage_select with forced_views first (policy "coverage").  After
    every step the staleness is updated with the step's views (all views
    when full) and the gaps advance.  seen: [N][B][N][H][W] pairs (as from
    coverage_pairs); stale0: the initial staleness (coverage_init).
    Returns per-step records: k, anchors, full, c (cached steps so far),
    stale, stats and gap after the step."""
    N = stale0.shape[1]
    steps = len(full) if steps is None else steps
    stale, stats, gap, c = stale0, None, [0] * N, 0
    out = []
    for k in range(steps):
        is_full = bool(full[k]) or k == 0 or (tau is not None and stats is not None and refresh_due(stats, tau))
        if is_full:
            A = list(range(N))
        else:
            if policy == "rotate":
                A = anchors(N, a, c)
            elif policy == "rotation_coverage":
                cands = rotation_sets(N, a)
                sc = coverage_score(stale, seen, cands)
                A = cands[int(np.argmax(sc))]           # first maximum: ties go to the earlier set
            else:
                A = coverage_select(stale, seen, a, forced=forced_views(gap, a, max_gap))
            c += 1
        stale, stats = coverage_update(stale, seen, A, R)
        gap = advance_gaps(gap, A, is_full)
        out.append({"k": k, "anchors": list(A), "full": is_full, "c": c, "stale": stale.copy(),
                    "stats": stats.copy(), "gap": list(gap)})
    return out


def trajectory_adaptive(x_t0: np.ndarray, stub, pos: np.ndarray, cams, K: int, tol_frac: float, dtype: str,
                        kind: str, S: int, full: Sequence[int], a: int, policy: str = "coverage", max_gap: int = 0,
                        tau: float = None, R: int = 2, steps: int = None):
    """The cached loop of trajectory() with the coverage-driven schedule of
    schedule_adaptive() (the visibility pairs from this geometry's own
    builds).  Records as trajectory() plus full, stale, stats and gap after
    the step."""
    steps = S if steps is None else steps
    bb = bbox(pos, tol_frac)
    seen = coverage_pairs(pos, cams, K, bb)
    sched = schedule_adaptive(seen, coverage_init(pos), full, a, policy, max_gap, tau, R, steps)
    cache = {}
    x_t, x0_store = x_t0, None
    out = []
    for d in sched:
        k, A, is_full = d["k"], d["anchors"], d["full"]
        t, tn = step_times(kind, S, k)
        if is_full:
            x0_state = stub(k, A)
            x0_exact = (x0_state if dtype == "f32" else _bf16_values(x0_state)).astype(np.float64)
        else:
            key = tuple(A)
            if key not in cache:
                corr, w, _ = build(pos, cams, A, K, bb)
                cache[key] = (corr, w)
            corr, w = cache[key]
            x0_exact, x0_state = transport(x0_store, stub(k, A), corr, w, A, dtype)
        xn, _ = reconstruct(x_t, x0_state, dtype, kind, t, tn)
        x_t = store(xn, dtype)
        x0_store = x0_state
        out.append({"k": k, "anchors": A, "full": is_full, "c": d["c"], "x_t": x_t, "x0": x0_state,
                    "x_t_exact": xn, "x0_exact": x0_exact, "stale": d["stale"], "stats": d["stats"],
                    "gap": d["gap"]})
    return out


def _bf16_values(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)
