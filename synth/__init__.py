"""Seeded synthetic inputs for the cross-view transport path.

Input generation only: geometry (meshes / an analytic star-shaped surface),
cameras, rendered position maps and synthetic latent fields.  Nothing here
performs the transport, the correspondence search or the sampler update; both
the oracle and the HIP path consume the arrays produced here.

Recipe (stand-ins for the paper's eval200 assets, which are not available):
  * geometry: seeded displaced sphere / torus / (2,3) torus knot / union of
    three ellipsoids, displacement = normalised sum of six low-frequency
    sinusoids of the 3D position;
  * cameras: looking at the origin from azimuth/elevation rings;
  * position maps: per-pixel exact ray hits (double, stored as float),
    NaN background;
  * latents: x0 = smooth function of the 3D surface point + per-view noise,
    eps ~ N(0, 1).
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Dict, Tuple

import numpy as np

from .configs import BY_ID, CONFIGS, Workload, shrink  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

PURPOSE_GEOM = 1
PURPOSE_FIELD = 2
PURPOSE_VIEWNOISE = 3
PURPOSE_STEPNOISE = 4
PURPOSE_EPS = 5


def lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "libsynth.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `make -C synth`")
        L = ctypes.CDLL(path)
        dp = ctypes.POINTER(ctypes.c_double)
        L.synth_render_mesh.argtypes = [dp, ctypes.c_int64, ctypes.POINTER(ctypes.c_int32),
                                        ctypes.c_int64, dp, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, ctypes.POINTER(ctypes.c_float), ctypes.c_int]
        L.synth_render_mesh.restype = ctypes.c_int
        L.synth_raycast_radial.argtypes = [ctypes.c_double, dp, ctypes.c_int, dp, ctypes.c_int,
                                           ctypes.c_int, ctypes.c_int,
                                           ctypes.POINTER(ctypes.c_float), ctypes.c_int]
        L.synth_raycast_radial.restype = ctypes.c_int
        _LIB = L
    return _LIB


def rng(*key) -> np.random.Generator:
    return np.random.default_rng([int(k) for k in key])


# ----------------------------------------------------------------------------
# cameras
# ----------------------------------------------------------------------------

def look_at_origin(az_deg: float, el_deg: float, dist: float) -> Tuple[np.ndarray, np.ndarray]:
    """World->camera (R, t) for a camera on a sphere of radius `dist` looking
    at the origin; world Y is up, azimuth about +Y from +Z toward +X."""
    az, el = math.radians(az_deg), math.radians(el_deg)
    c = dist * np.array([math.cos(el) * math.sin(az), math.sin(el), math.cos(el) * math.cos(az)])
    fwd = -c / np.linalg.norm(c)
    up = np.array([0.0, 1.0, 0.0])
    right = np.cross(fwd, up)
    right /= np.linalg.norm(right)
    down = np.cross(fwd, right)
    R = np.stack([right, down, fwd])
    t = -R @ c
    return R, t


def bound_radius(w: Workload) -> float:
    d = abs(w.displacement)
    if w.geometry == "sphere":
        return 1.0 + d
    if w.geometry == "torus":
        return 1.4 + d
    if w.geometry == "torusknot":
        return 0.4 * 3.0 + 0.18 + d
    if w.geometry == "ellipsoids":
        return 1.3 + d
    raise ValueError(w.geometry)


def cameras(w: Workload, res: int = None) -> Dict[str, np.ndarray]:
    """Cameras of one asset as float32 arrays in pixel units of a `res`-square
    image (default: latent resolution).  Keys: model [N] int32, R [N,3,3],
    t [N,3], fx, fy, cx, cy [N]."""
    res = w.H if res is None else res
    assert w.H == w.W
    N = w.N
    R = np.zeros((N, 3, 3), np.float32)
    t = np.zeros((N, 3), np.float32)
    fx = np.zeros(N, np.float32)
    model = np.zeros(N, np.int32)
    rb = bound_radius(w)
    for v in range(N):
        if w.camera_model == "pinhole":
            half = math.radians(w.fov_deg / 2)
            dist = 1.1 * rb / math.sin(half)
            f = (res / 2.0) / math.tan(half)
            model[v] = 0
        else:
            dist = 3.0
            f = (res / 2.0) / w.ortho_half_extent
            model[v] = 1
        Rv, tv = look_at_origin(w.azimuths_deg[v], w.elevations_deg[v], dist)
        R[v] = Rv
        t[v] = tv
        fx[v] = f
    c = np.full(N, res / 2.0, np.float32)
    return {"model": model, "R": R, "t": t, "fx": fx.copy(), "fy": fx.copy(), "cx": c, "cy": c.copy()}


def cams_for_renderer(cams: Dict[str, np.ndarray]) -> np.ndarray:
    N = cams["model"].shape[0]
    out = np.zeros((N, 17), np.float64)
    out[:, 0] = cams["model"]
    out[:, 1:10] = cams["R"].reshape(N, 9)
    out[:, 10:13] = cams["t"]
    out[:, 13] = cams["fx"]
    out[:, 14] = cams["fy"]
    out[:, 15] = cams["cx"]
    out[:, 16] = cams["cy"]
    return out


def batch_cameras(w: Workload, res: int = None) -> Dict[str, np.ndarray]:
    """Cameras for all B assets: arrays with a leading [B] axis (every asset of
    a workload shares the camera rig)."""
    c = cameras(w, res)
    return {k: np.ascontiguousarray(np.broadcast_to(v, (w.B,) + v.shape)) for k, v in c.items()}


# ----------------------------------------------------------------------------
# geometry
# ----------------------------------------------------------------------------

def _disp_params(g: np.random.Generator, n: int = 6) -> np.ndarray:
    d = g.normal(size=(n, 3))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    f = g.uniform(1.0, 3.0, size=n)
    phi = g.uniform(0.0, 2 * math.pi, size=n)
    return np.concatenate([d, f[:, None], phi[:, None]], axis=1)


def _disp_field(P: np.ndarray, params: np.ndarray) -> np.ndarray:
    s = np.zeros(P.shape[:-1])
    for q in params:
        s += np.sin(q[3] * (P @ q[:3]) + q[4])
    return s / len(params)


def _grid_tris(nu: int, nv: int, offset: int = 0) -> np.ndarray:
    """Triangles of a (nu x nv) periodic-in-both grid."""
    i, j = np.meshgrid(np.arange(nu), np.arange(nv), indexing="ij")
    a = i * nv + j
    b = ((i + 1) % nu) * nv + j
    c = ((i + 1) % nu) * nv + (j + 1) % nv
    d = i * nv + (j + 1) % nv
    t1 = np.stack([a, b, c], -1).reshape(-1, 3)
    t2 = np.stack([a, c, d], -1).reshape(-1, 3)
    return (np.concatenate([t1, t2]) + offset).astype(np.int32)


def _vertex_normals(V: np.ndarray, T: np.ndarray) -> np.ndarray:
    n = np.zeros_like(V)
    fn = np.cross(V[T[:, 1]] - V[T[:, 0]], V[T[:, 2]] - V[T[:, 0]])
    for k in range(3):
        np.add.at(n, T[:, k], fn)
    n /= np.maximum(np.linalg.norm(n, axis=1, keepdims=True), 1e-30)
    return n


def _random_rotation(g: np.random.Generator) -> np.ndarray:
    q = g.normal(size=4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
                     [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
                     [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)]])


def mesh(w: Workload, asset: int, detail: int = 1) -> Tuple[np.ndarray, np.ndarray]:
    """Seeded triangle mesh (vertices [nv,3] float64, triangles [nt,3] int32)."""
    g = rng(w.cfg_id, asset, PURPOSE_GEOM)
    params = _disp_params(g)
    amp = w.displacement
    if w.geometry == "torus":
        nu, nv = 384 * detail, 128 * detail
        u = np.linspace(0, 2 * math.pi, nu, endpoint=False)
        v = np.linspace(0, 2 * math.pi, nv, endpoint=False)
        U, Vv = np.meshgrid(u, v, indexing="ij")
        Rr, r = 1.0, 0.4
        P = np.stack([(Rr + r * np.cos(Vv)) * np.cos(U), r * np.sin(Vv),
                      (Rr + r * np.cos(Vv)) * np.sin(U)], -1).reshape(-1, 3)
        Nrm = np.stack([np.cos(Vv) * np.cos(U), np.sin(Vv), np.cos(Vv) * np.sin(U)], -1).reshape(-1, 3)
        # a mild seeded tilt keeps assets distinct without hiding the hole
        ang = g.uniform(-0.35, 0.35)
        ca, sa = math.cos(ang), math.sin(ang)
        Rx = np.array([[1, 0, 0], [0, ca, -sa], [0, sa, ca]])
        P = P @ Rx.T
        Nrm = Nrm @ Rx.T
        V = P + amp * _disp_field(P, params)[:, None] * Nrm
        T = _grid_tris(nu, nv)
        return V, T
    if w.geometry == "torusknot":
        nu, nv = 1536 * detail, 48 * detail
        p_, q_ = 2, 3
        s = 0.4
        u = np.linspace(0, 2 * math.pi, nu, endpoint=False)

        def curve(uu):
            rr = 2.0 + np.cos(q_ * uu)
            return s * np.stack([rr * np.cos(p_ * uu), -np.sin(q_ * uu), rr * np.sin(p_ * uu)], -1)

        h = 1e-4
        c0 = curve(u)
        d1 = (curve(u + h) - curve(u - h)) / (2 * h)
        d2 = (curve(u + h) - 2 * c0 + curve(u - h)) / (h * h)
        T1 = d1 / np.linalg.norm(d1, axis=1, keepdims=True)
        N1 = d2 - (d2 * T1).sum(1, keepdims=True) * T1
        N1 /= np.linalg.norm(N1, axis=1, keepdims=True)
        B1 = np.cross(T1, N1)
        v = np.linspace(0, 2 * math.pi, nv, endpoint=False)
        tube = 0.18
        Nrm = (np.cos(v)[None, :, None] * N1[:, None, :] + np.sin(v)[None, :, None] * B1[:, None, :])
        P = c0[:, None, :] + tube * Nrm
        P = P.reshape(-1, 3)
        Nrm = Nrm.reshape(-1, 3)
        ang = g.uniform(0, 2 * math.pi)
        ca, sa = math.cos(ang), math.sin(ang)
        Ry = np.array([[ca, 0, sa], [0, 1, 0], [-sa, 0, ca]])
        P = P @ Ry.T
        Nrm = Nrm @ Ry.T
        V = P + amp * _disp_field(P, params)[:, None] * Nrm
        return V, _grid_tris(nu, nv)
    if w.geometry == "ellipsoids":
        Vs, Ts = [], []
        off = 0
        nu, nv = 256 * detail, 128 * detail
        for e in range(3):
            axes = g.uniform(0.4, 0.8, size=3)
            centre = g.normal(size=3)
            centre *= g.uniform(0.15, 0.5) / np.linalg.norm(centre)
            Rot = _random_rotation(g)
            # longitude periodic (nu), latitude open (nv interior rings) + 2 poles
            lon = np.linspace(0, 2 * math.pi, nu, endpoint=False)
            lat = (np.arange(nv) + 0.5) / nv * math.pi - math.pi / 2
            Lo, La = np.meshgrid(lon, lat, indexing="ij")
            S = np.stack([np.cos(La) * np.cos(Lo), np.sin(La), np.cos(La) * np.sin(Lo)], -1).reshape(-1, 3)
            S = np.concatenate([S, [[0, -1, 0], [0, 1, 0]]])
            Pl = S * axes
            Nl = S / axes
            Nl /= np.linalg.norm(Nl, axis=1, keepdims=True)
            P = Pl @ Rot.T + centre
            Nrm = Nl @ Rot.T
            V = P + amp * _disp_field(P, params)[:, None] * Nrm
            i, j = np.meshgrid(np.arange(nu), np.arange(nv - 1), indexing="ij")
            a = i * nv + j
            b = ((i + 1) % nu) * nv + j
            c = ((i + 1) % nu) * nv + j + 1
            d = i * nv + j + 1
            T = np.concatenate([np.stack([a, b, c], -1).reshape(-1, 3),
                                np.stack([a, c, d], -1).reshape(-1, 3)])
            south, north = nu * nv, nu * nv + 1
            ii = np.arange(nu)
            T = np.concatenate([T,
                                np.stack([np.full(nu, south), ((ii + 1) % nu) * nv, ii * nv], -1),
                                np.stack([np.full(nu, north), ii * nv + nv - 1,
                                          ((ii + 1) % nu) * nv + nv - 1], -1)])
            Vs.append(V)
            Ts.append(T + off)
            off += V.shape[0]
        return np.concatenate(Vs), np.concatenate(Ts).astype(np.int32)
    raise ValueError(f"no mesh for geometry {w.geometry}")


def sphere_params(w: Workload, asset: int) -> np.ndarray:
    return _disp_params(rng(w.cfg_id, asset, PURPOSE_GEOM))


# ----------------------------------------------------------------------------
# position maps
# ----------------------------------------------------------------------------

def _fptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _dptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def render_position_maps(w: Workload, assets=None, nthreads: int = 0) -> np.ndarray:
    """Position maps at render resolution: float32 [B][N][Hr][Wr][3], NaN background.

    The sphere workload is ray-cast directly at latent resolution."""
    L = lib()
    assets = range(w.B) if assets is None else assets
    Hr, Wr = w.render_hw
    outs = []
    cam = cams_for_renderer(cameras(w, Hr))
    for b in assets:
        out = np.empty((w.N, Hr, Wr, 3), np.float32)
        if w.geometry == "sphere":
            prm = np.ascontiguousarray(sphere_params(w, b))
            rc = L.synth_raycast_radial(w.displacement, _dptr(prm), prm.shape[0], _dptr(cam), w.N,
                                        Hr, Wr, _fptr(out), nthreads)
        else:
            V, T = mesh(w, b)
            V = np.ascontiguousarray(V, np.float64)
            T = np.ascontiguousarray(T, np.int32)
            rc = L.synth_render_mesh(_dptr(V), V.shape[0],
                                     T.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), T.shape[0],
                                     _dptr(cam), w.N, Hr, Wr, _fptr(out), nthreads)
        if rc != 0:
            raise RuntimeError(f"synth renderer failed with {rc}")
        outs.append(out)
    return np.stack(outs)


def raycast_radial(amp: float, params: np.ndarray, cams: Dict[str, np.ndarray], H: int, W: int,
                   nthreads: int = 0) -> np.ndarray:
    """Ray-cast r(w) = 1 + amp * D(w) for arbitrary cameras (pixel units of H x W)."""
    L = lib()
    cam = cams_for_renderer(cams)
    prm = np.ascontiguousarray(params, np.float64)
    out = np.empty((cam.shape[0], H, W, 3), np.float32)
    rc = L.synth_raycast_radial(float(amp), _dptr(prm), prm.shape[0], _dptr(cam), cam.shape[0],
                                H, W, _fptr(out), nthreads)
    if rc != 0:
        raise RuntimeError(f"synth ray-caster failed with {rc}")
    return out


# ----------------------------------------------------------------------------
# latents
# ----------------------------------------------------------------------------

def field_params(w: Workload, asset: int) -> Dict[str, np.ndarray]:
    g = rng(w.cfg_id, asset, PURPOSE_FIELD)
    C = w.C
    amp = g.uniform(0.2, 0.5, size=(C, 3))
    om = g.normal(size=(C, 3, 3))
    om /= np.linalg.norm(om, axis=2, keepdims=True)
    om *= g.uniform(1.0, 3.0, size=(C, 3, 1))
    phi = g.uniform(0, 2 * math.pi, size=(C, 3))
    psi = g.uniform(0.2, 0.5, size=(C, 3))
    return {"amp": amp, "omega": om, "phi": phi, "psi": psi}


def clean_field(P: np.ndarray, prm: Dict[str, np.ndarray], tau: float) -> np.ndarray:
    """g_c(P, tau) = sum_j amp_cj * sin(omega_cj . P + phi_cj + 2 pi psi_cj tau).
    P [..., 3] (NaN = background -> 0); returns [..., C] float64."""
    fg = np.isfinite(P).all(-1)
    Pz = np.where(fg[..., None], P, 0.0).astype(np.float64)
    C = prm["amp"].shape[0]
    out = np.zeros(P.shape[:-1] + (C,))
    for c in range(C):
        for j in range(3):
            out[..., c] += prm["amp"][c, j] * np.sin(
                Pz @ prm["omega"][c, j] + prm["phi"][c, j] + 2 * math.pi * prm["psi"][c, j] * tau)
    out[~fg] = 0.0
    return out


def x0_state(w: Workload, pos_lat: np.ndarray, step: int, views=None) -> np.ndarray:
    """Synthetic x0 for every asset at sampler step `step`: float32
    [B][len(views)][H][W][C] = smooth field of the surface point + per-view
    noise (std 0.05, fixed per view) + fresh per-step noise (std 0.005)."""
    B = pos_lat.shape[0]
    views = range(w.N) if views is None else list(views)
    tau = step / max(w.S, 1)
    out = np.empty((B, len(views), w.H, w.W, w.C), np.float32)
    for b in range(B):
        prm = field_params(w, b)
        for i, v in enumerate(views):
            f = clean_field(pos_lat[b, v], prm, tau)
            f += 0.05 * rng(w.cfg_id, b, PURPOSE_VIEWNOISE, v).standard_normal(f.shape)
            f += 0.005 * rng(w.cfg_id, b, PURPOSE_STEPNOISE, v, step).standard_normal(f.shape)
            out[b, i] = f
    return out


def eps_noise(w: Workload, step: int = 0) -> np.ndarray:
    """eps ~ N(0, 1), float32 [B][N][H][W][C]."""
    out = np.empty((w.B, w.N, w.H, w.W, w.C), np.float32)
    for b in range(w.B):
        out[b] = rng(w.cfg_id, b, PURPOSE_EPS, step).standard_normal(out.shape[1:])
    return out


def mix(x0: np.ndarray, eps: np.ndarray, c_signal: float, c_noise: float) -> np.ndarray:
    """c_signal * x0 + c_noise * eps in float64, returned as float32: a noisy
    state for given forward-process coefficients (supplied by the caller)."""
    return (c_signal * x0.astype(np.float64) + c_noise * eps.astype(np.float64)).astype(np.float32)


# ----------------------------------------------------------------------------
# bf16 storage helpers (storage format of the inputs; RNE)
# ----------------------------------------------------------------------------

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(np.asarray(x, np.float32))
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[nan] = 0x7FC0
    return r


def from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """float32 values -> storage array of `dtype` ("f32": float32, "bf16": uint16 bits)."""
    if dtype == "f32":
        return np.ascontiguousarray(x, np.float32)
    if dtype == "bf16":
        return to_bf16_bits(x)
    raise ValueError(dtype)


def values(s: np.ndarray, dtype: str) -> np.ndarray:
    """storage array -> float32 values."""
    if dtype == "f32":
        return np.asarray(s, np.float32)
    return from_bf16_bits(s)
