"""Workload definitions for the synthetic cross-view transport benchmarks.

These describe *inputs* (geometry, cameras, latent shapes, sampler and
schedule parameters); they contain none of the transport arithmetic.

The five workloads follow the shapes of the paper's substrates (Sec. 4.1
Setup; Sec. 3.1 six-view Hunyuan3D-2.1 Paint at 512^2; SyncMVD's ten views and
30 DDPM steps; the 50-step Euler flow sampler of MV-Adapter in Sec. 6 "Long
denoising trajectories") with synthetic stand-ins for the assets, which are
not available.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int                  # seed namespace
    B: int                       # independent assets per batch
    N: int                       # views per asset
    H: int                       # latent grid height
    W: int                       # latent grid width
    C: int                       # latent channels
    dtype: str                   # "f32" or "bf16" (latent storage)
    geometry: str                # "sphere" | "torus" | "torusknot" | "ellipsoids"
    displacement: float          # amplitude of the seeded low-frequency displacement
    camera_model: str            # "pinhole" | "ortho"
    azimuths_deg: Tuple[float, ...]
    elevations_deg: Tuple[float, ...]
    fov_deg: float = 40.0        # pinhole full field of view
    ortho_half_extent: float = 1.15
    render: Optional[int] = None  # render resolution (square); None = ray-cast at latent res
    a: int = 1                   # anchors per cached step
    K: int = 4                   # taps per anchor
    tol_frac: float = 0.01       # tolerance as a fraction of the bbox diagonal
    sampler: str = "ddim"        # "ddim" | "flow"
    S: int = 1                   # sampler steps
    full_rule: str = "periodic"  # "periodic" | "head_mid_tail" | "explicit"
    full_E: int = 0              # period for "periodic"
    full_explicit: Tuple[int, ...] = field(default_factory=tuple)
    ddim_single: Optional[Tuple[int, int]] = None  # (t, t_next) for a one-step case
    fixed_anchors: Optional[Tuple[int, ...]] = None

    @property
    def factor(self) -> int:
        return 1 if self.render is None else self.render // self.H

    @property
    def render_hw(self) -> Tuple[int, int]:
        if self.render is None:
            return self.H, self.W
        return self.render, self.render

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


def _alt(n, lo, hi):
    return tuple(lo if i % 2 == 0 else hi for i in range(n))


C1 = Workload(
    name="tiny_sphere_4v_32", cfg_id=1, B=1, N=4, H=32, W=32, C=4, dtype="f32",
    geometry="sphere", displacement=0.05, camera_model="ortho",
    azimuths_deg=(0.0, 90.0, 180.0, 270.0), elevations_deg=(0.0,) * 4,
    render=None, a=1, K=4, sampler="ddim", S=1, full_rule="explicit",
    full_explicit=(), ddim_single=(800, 760), fixed_anchors=(0,))

C2 = Workload(
    name="hunyuan_torus_6v_64", cfg_id=2, B=1, N=6, H=64, W=64, C=4, dtype="f32",
    geometry="torus", displacement=0.05, camera_model="pinhole",
    azimuths_deg=tuple(60.0 * i for i in range(6)), elevations_deg=_alt(6, 20.0, -20.0),
    render=512, a=2, K=4, sampler="ddim", S=30, full_rule="periodic", full_E=5)

C3 = Workload(
    name="torus_6v_96_b4", cfg_id=3, B=4, N=6, H=96, W=96, C=4, dtype="f32",
    geometry="torus", displacement=0.05, camera_model="pinhole",
    azimuths_deg=tuple(60.0 * i for i in range(6)), elevations_deg=_alt(6, 20.0, -20.0),
    render=768, a=2, K=4, sampler="flow", S=30, full_rule="head_mid_tail")

C4 = Workload(
    name="syncmvd_ellipsoids_10v_96", cfg_id=4, B=1, N=10, H=96, W=96, C=4, dtype="bf16",
    geometry="ellipsoids", displacement=0.05, camera_model="pinhole",
    azimuths_deg=tuple(72.0 * (i % 5) for i in range(10)),
    elevations_deg=tuple(0.0 if i < 5 else 30.0 for i in range(10)),
    render=768, a=3, K=4, sampler="ddim", S=30, full_rule="periodic", full_E=4)

C5 = Workload(
    name="stress_torusknot_12v_128x16_b8", cfg_id=5, B=8, N=12, H=128, W=128, C=16,
    dtype="bf16", geometry="torusknot", displacement=0.03, camera_model="pinhole",
    azimuths_deg=tuple(30.0 * i for i in range(12)), elevations_deg=_alt(12, 15.0, -15.0),
    render=1024, a=4, K=4, sampler="flow", S=50, full_rule="head_mid_tail")

CONFIGS = {w.name: w for w in (C1, C2, C3, C4, C5)}
BY_ID = {w.cfg_id: w for w in (C1, C2, C3, C4, C5)}


def shrink(w: Workload, **kw) -> Workload:
    """A copy of a workload with some fields replaced (smaller test cases)."""
    from dataclasses import replace
    return replace(w, **kw)
