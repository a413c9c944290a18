"""Cached denoising loop on the GPU (Sec. 3.2: loop order, batch-sliced
anchor forward, drift-bounding schedule).

Orchestration only: the step arithmetic runs in the library's kernels and the
schedule (anchor rotation, full-view steps, sampler step times) comes from
the library's host calls.  A runner keeps the loop state -- the noisy state
x_t, the store of x0 for all views, the step index k and the cached-step
counter c -- and one correspondence operator (with its visible-token index)
per anchor set, built on first use.

The denoiser is the caller's: predict(k, views) returns this step's x0 for
the listed views as a device tensor [B, len(views), H, W, C].
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional, Sequence, Tuple

import torch

from . import (GC_FULL_HEAD_MID_TAIL, GC_FULL_PERIODIC, Sampler, VisibleIndex, gc_build_correspondence,
               gc_index_correspondence, gc_posmap_bbox, gc_sampler_reconstruct, gc_sampler_step_times,
               gc_schedule_anchors, gc_schedule_full_steps, gc_transport_reconstruct, gc_transport_unipc,
               gc_unipc_coeffs, gc_unipc_update)

Predict = Callable[[int, List[int]], torch.Tensor]


class GeoCacheRunner:
    def __init__(self, pos: torch.Tensor, cams: torch.Tensor, a: int, K: int, sampler: Sampler, S: int,
                 full: Sequence[int], tol_frac: float = 0.01, use_index: bool = True, unipc_order: int = 0,
                 unipc_corrector: bool = True, stream=None):
        """pos: device float32 [B, N, H, W, 3] latent-grid position maps;
        cams: device gc_camera tensor [B, N, 68]; full[k] = 1 for full-view steps.
        unipc_order 1 or 2 runs the UniPC multistep solver on the sampler's
        DDIM noise schedule instead of the sampler's own step."""
        self.pos, self.cams, self.a, self.K = pos, cams, a, K
        self.sampler, self.S = sampler, S
        self.full = list(full)
        if len(self.full) != S:
            raise ValueError("full must have one entry per sampler step")
        self.B, self.N = pos.shape[0], pos.shape[1]
        self.use_index = use_index
        self.stream = stream
        self.bbox = gc_posmap_bbox(pos, tol_frac, stream=stream)
        self._ops: Dict[Tuple[int, ...], Tuple[torch.Tensor, torch.Tensor, Optional[VisibleIndex]]] = {}
        self.unipc_order, self.unipc_corrector = unipc_order, unipc_corrector
        self.k = 0
        self.c = 0
        self.x_t: Optional[torch.Tensor] = None
        self.x0: Optional[torch.Tensor] = None
        self.x0_km2: Optional[torch.Tensor] = None   # UniPC: x0 of step k-2
        self.x_c: Optional[torch.Tensor] = None      # UniPC: corrected sample of step k-1

    @staticmethod
    def full_steps(rule: str, S: int, E: int = 0) -> List[int]:
        return gc_schedule_full_steps(GC_FULL_PERIODIC if rule == "periodic" else GC_FULL_HEAD_MID_TAIL, S, E)

    def operator(self, anchors: Sequence[int]):
        """(corr, weights, index) of an anchor set, built on first use."""
        key = tuple(anchors)
        if key not in self._ops:
            corr, wts = gc_build_correspondence(self.pos, self.cams, list(key), self.K, self.bbox, stream=self.stream)
            idx = gc_index_correspondence(corr, stream=self.stream) if self.use_index else None
            self._ops[key] = (corr, wts, idx)
        return self._ops[key]

    def start(self, x_t: torch.Tensor) -> None:
        self.x_t, self.x0, self.k, self.c = x_t, None, 0, 0
        self.x0_km2, self.x_c = None, None

    def step(self, predict: Predict) -> List[int]:
        """Run sampler step k; returns the views the denoiser was asked for."""
        if self.x_t is None:
            raise RuntimeError("call start() first")
        k = self.k
        if self.unipc_order:
            return self._step_unipc(predict)
        t, tn = gc_sampler_step_times(self.sampler, self.S, k)
        if self.full[k] or self.x0 is None:
            views = list(range(self.N))
            x0 = predict(k, views).contiguous()
            x_next, _ = gc_sampler_reconstruct(self.x_t, x0, self.sampler, t, tn, stream=self.stream)
        else:
            views = gc_schedule_anchors(self.N, self.a, self.c)
            self.c += 1
            corr, wts, idx = self.operator(views)
            x0, x_next, _ = gc_transport_reconstruct(self.x0, predict(k, views).contiguous(), corr, wts, self.x_t,
                                                     views, self.sampler, t, tn, index=idx, stream=self.stream)
        self.x0, self.x_t = x0, x_next
        self.k += 1
        return views

    def _step_unipc(self, predict: Predict) -> List[int]:
        k = self.k
        st = gc_unipc_coeffs(self.sampler, self.S, k, self.unipc_order, self.unipc_corrector)
        m2 = self.x0_km2 if st.use_corrector and st.c_mk2 != 0.0 else None
        if self.full[k] or self.x0 is None:
            views = list(range(self.N))
            mk = predict(k, views).contiguous()
            x_c, x_next = gc_unipc_update(st, mk, x_cur=self.x_t, x_prev=self.x_c if st.use_corrector else None,
                                          m_km2=m2, m_km1=self.x0, stream=self.stream)
        else:
            views = gc_schedule_anchors(self.N, self.a, self.c)
            self.c += 1
            corr, wts, idx = self.operator(views)
            mk, x_c, x_next = gc_transport_unipc(self.x0, predict(k, views).contiguous(), corr, wts, views, st,
                                                 x_cur=self.x_t, x_prev=self.x_c if st.use_corrector else None,
                                                 m_km2=m2, index=idx, stream=self.stream)
        self.x0_km2, self.x0, self.x_c, self.x_t = self.x0, mk, x_c, x_next
        self.k += 1
        return views

    def run(self, predict: Predict, steps: Optional[int] = None) -> None:
        for _ in range(self.S - self.k if steps is None else steps):
            self.step(predict)

    def state_dict(self) -> dict:
        """Loop state for checkpoint / resume (tensors are cloned)."""
        cl = lambda t: None if t is None else t.clone()
        return {"k": self.k, "c": self.c, "x_t": cl(self.x_t), "x0": cl(self.x0), "x0_km2": cl(self.x0_km2),
                "x_c": cl(self.x_c)}

    def load_state_dict(self, st: dict) -> None:
        cl = lambda t: None if t is None else t.clone()
        self.k, self.c = int(st["k"]), int(st["c"])
        self.x_t, self.x0 = cl(st["x_t"]), cl(st["x0"])
        self.x0_km2, self.x_c = cl(st.get("x0_km2")), cl(st.get("x_c"))
