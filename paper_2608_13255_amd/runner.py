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

import contextlib
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import torch

from . import (GC_FULL_HEAD_MID_TAIL, GC_FULL_HEAD_TAIL_E, GC_FULL_PERIODIC, Sampler, VisibleIndex,
               gc_build_correspondence, gc_coverage_init, gc_coverage_pairs, gc_coverage_score, gc_coverage_select,
               gc_coverage_update, gc_coverage_update_score, gc_coverage_update_select, gc_coverage_workspace_bytes,
               gc_index_correspondence, gc_index_foreground,
               gc_posmap_bbox, gc_sampler_reconstruct, gc_sampler_step_times, gc_schedule_advance_gaps,
               gc_schedule_anchors, gc_schedule_forced_views, gc_schedule_full_steps, gc_schedule_refresh_due,
               gc_transport_reconstruct, gc_transport_reconstruct_geom, gc_transport_unipc, gc_transport_unipc_geom,
               gc_unipc_coeffs, gc_unipc_update)

Predict = Callable[[int, List[int]], torch.Tensor]


class GeoCacheRunner:
    def __init__(self, pos: torch.Tensor, cams: torch.Tensor, a: int, K: int, sampler: Sampler, S: int,
                 full: Sequence[int], tol_frac: float = 0.01, use_index: bool = True, unipc_order: int = 0,
                 unipc_corrector: bool = True, anchor_policy: str = "rotate", max_gap: int = 0,
                 refresh_tau: Optional[float] = None, refresh_R: int = 2, geom: bool = False, stream=None):
        """pos: device float32 [B, N, H, W, 3] latent-grid position maps;
        cams: device gc_camera tensor [B, N, 68]; full[k] = 1 for full-view steps.
        unipc_order 1 or 2 runs the UniPC multistep solver on the sampler's
        DDIM noise schedule instead of the sampler's own step.

        anchor_policy "coverage" picks each cached step's anchors by greedy
        weighted maximum coverage of the stale tokens (gc_coverage_select);
        views that have not been anchors for max_gap cached steps (0: off)
        are forced into the set, longest gap first.  "rotation_coverage"
        takes, among the rotation's distinct sets, the one with the largest
        weighted coverage (gc_coverage_score; ties to the earlier set).
        refresh_tau makes a step full when the fraction of foreground tokens
        stale for refresh_R or more steps exceeds it.  geom computes the
        correspondence inside each step instead of building and caching one
        per anchor set; with use_index it uses the position maps' foreground
        index (built once here)."""
        if anchor_policy not in ("rotate", "coverage", "rotation_coverage"):
            raise ValueError("anchor_policy must be 'rotate', 'coverage' or 'rotation_coverage'")
        self.pos, self.cams, self.a, self.K = pos, cams, a, K
        self.sampler, self.S = sampler, S
        self.full = list(full)
        if len(self.full) != S:
            raise ValueError("full must have one entry per sampler step")
        self.B, self.N = pos.shape[0], pos.shape[1]
        self.use_index = use_index
        if stream is not None and not isinstance(stream, torch.cuda.Stream):
            stream = torch.cuda.ExternalStream(int(stream))
        self.stream = stream
        self._ops: Dict[Tuple[int, ...], Tuple[torch.Tensor, torch.Tensor, Optional[VisibleIndex]]] = {}
        self.unipc_order, self.unipc_corrector = unipc_order, unipc_corrector
        self.anchor_policy, self.max_gap = anchor_policy, max_gap
        self.refresh_tau, self.refresh_R, self.geom = refresh_tau, refresh_R, geom
        self.tracking = anchor_policy != "rotate" or refresh_tau is not None
        self.rotation_sets: List[List[int]] = []
        for c in range(self.N):
            A = gc_schedule_anchors(self.N, a, c)
            if A not in self.rotation_sets:
                self.rotation_sets.append(A)
        with self._on_stream():
            self.bbox = gc_posmap_bbox(pos, tol_frac, stream=stream)
            self.fg_index = gc_index_foreground(pos, stream=stream) if geom and use_index else None
            self.pairs = gc_coverage_pairs(pos, cams, self.bbox, stream=stream) if self.tracking else None
            self._ws = (torch.empty(gc_coverage_workspace_bytes(), dtype=torch.uint8, device=pos.device)
                        if self.tracking else None)
        self.stale: Optional[torch.Tensor] = None
        # the next cached step's selection (device) or set scores, computed
        # with the last step's staleness update in one pass; None: compute it
        # when needed (after a restart or a resume)
        self._next: Optional[torch.Tensor] = None
        self.stats_host = None                        # per-view staleness statistics after the last step (refresh rule)
        self.gap: List[int] = [0] * self.N            # cached steps since each view was last an anchor
        self.last_full = False
        self.k = 0
        self.c = 0
        self.x_t: Optional[torch.Tensor] = None
        self.x0: Optional[torch.Tensor] = None
        self.x0_km2: Optional[torch.Tensor] = None   # UniPC: x0 of step k-2
        self.x_c: Optional[torch.Tensor] = None      # UniPC: corrected sample of step k-1

    def _on_stream(self):
        """Every device call, allocation and read-back of the runner happens
        with its stream current, so they are ordered on it (with stream=None,
        on torch's current stream)."""
        return torch.cuda.stream(self.stream) if self.stream is not None else contextlib.nullcontext()

    @staticmethod
    def full_steps(rule: str, S: int, E: int = 0) -> List[int]:
        """rule "periodic" (every E-th step), "head_mid_tail" ({0, 1, S/2, S-1}) or
        "head_tail_e" ({0, 1} and the last E steps)."""
        codes = {"periodic": GC_FULL_PERIODIC, "head_mid_tail": GC_FULL_HEAD_MID_TAIL, "head_tail_e": GC_FULL_HEAD_TAIL_E}
        if rule not in codes:
            raise ValueError(f"unknown full-step rule {rule!r}")
        return gc_schedule_full_steps(codes[rule], S, E)

    def operator(self, anchors: Sequence[int]):
        """(corr, weights, index) of an anchor set, built on first use."""
        key = tuple(anchors)
        if key not in self._ops:
            corr, wts = gc_build_correspondence(self.pos, self.cams, list(key), self.K, self.bbox, stream=self.stream)
            idx = gc_index_correspondence(corr, stream=self.stream) if self.use_index else None
            self._ops[key] = (corr, wts, idx)
        return self._ops[key]

    def start(self, x_t: torch.Tensor) -> None:
        """x_t: the initial state; work that produced it on another stream
        must be complete or ordered before this runner's stream."""
        with self._on_stream():
            self._start(x_t)

    def _start(self, x_t: torch.Tensor) -> None:
        self.x_t, self.x0, self.k, self.c = x_t, None, 0, 0
        self.x0_km2, self.x_c = None, None
        if self.tracking:
            self.stale = gc_coverage_init(self.pos, stream=self.stream)
            self.stats_host = None
        self._next = None
        self.gap = [0] * self.N
        self.last_full = False

    def _is_full(self, k: int) -> bool:
        if self.full[k] or self.x0 is None:
            return True
        return (self.refresh_tau is not None and self.stats_host is not None
                and gc_schedule_refresh_due(self.stats_host, self.refresh_tau))

    def _anchors(self) -> List[int]:
        """Anchor set of the next cached step (advances the cached-step counter)."""
        c = self.c
        self.c += 1
        if self.anchor_policy == "rotate":
            return gc_schedule_anchors(self.N, self.a, c)
        nxt, self._next = self._next, None
        if self.anchor_policy == "rotation_coverage":
            sc = nxt if nxt is not None else gc_coverage_score(self.pairs, self.stale, self.rotation_sets,
                                                               workspace=self._ws, stream=self.stream)
            sc = sc.cpu().tolist()
            return list(self.rotation_sets[sc.index(max(sc))])
        if nxt is None:
            due = gc_schedule_forced_views(self.gap, self.a, self.max_gap)
            nxt = gc_coverage_select(self.pairs, self.stale, self.a, forced=due, workspace=self._ws, stream=self.stream)
        return [int(v) for v in nxt.cpu().tolist()]

    def _after(self, views: List[int], full: bool) -> None:
        """Staleness and anchor gaps after a step with the given views."""
        self.last_full = full
        self.gap = gc_schedule_advance_gaps(self.gap, views, full)
        if self.tracking:
            # the update and the next cached step's choice in one pass over
            # the tokens (the forced views follow from the gaps just advanced);
            # unused when the next step is full
            if self.anchor_policy == "coverage":
                due = gc_schedule_forced_views(self.gap, self.a, self.max_gap)
                stats, self._next = gc_coverage_update_select(self.pairs, self.stale, views, self.refresh_R, self.a,
                                                              forced=due, workspace=self._ws, stream=self.stream)
            elif self.anchor_policy == "rotation_coverage":
                stats, self._next = gc_coverage_update_score(self.pairs, self.stale, views, self.refresh_R,
                                                             self.rotation_sets, workspace=self._ws, stream=self.stream)
            else:
                stats = gc_coverage_update(self.pairs, self.stale, views, self.refresh_R, stream=self.stream)
            # the host reads the statistics back only for the refresh rule
            self.stats_host = stats.cpu() if self.refresh_tau is not None else None

    def step(self, predict: Predict) -> List[int]:
        """Run sampler step k; returns the views the denoiser was asked for.
        predict runs with the runner's stream current."""
        if self.x_t is None:
            raise RuntimeError("call start() first")
        with self._on_stream():
            return self._step(predict)

    def _step(self, predict: Predict) -> List[int]:
        k = self.k
        if self.unipc_order:
            return self._step_unipc(predict)
        t, tn = gc_sampler_step_times(self.sampler, self.S, k)
        full = self._is_full(k)
        if full:
            views = list(range(self.N))
            x0 = predict(k, views).contiguous()
            x_next, _ = gc_sampler_reconstruct(self.x_t, x0, self.sampler, t, tn, stream=self.stream)
        else:
            views = self._anchors()
            new = predict(k, views).contiguous()
            if self.geom:
                x0, x_next, _ = gc_transport_reconstruct_geom(self.x0, new, self.pos, self.cams, self.bbox, self.x_t,
                                                              views, self.K, self.sampler, t, tn,
                                                              fg_index=self.fg_index, stream=self.stream)
            else:
                corr, wts, idx = self.operator(views)
                x0, x_next, _ = gc_transport_reconstruct(self.x0, new, corr, wts, self.x_t, views, self.sampler, t,
                                                         tn, index=idx, stream=self.stream)
        self.x0, self.x_t = x0, x_next
        self._after(views, full)
        self.k += 1
        return views

    def _step_unipc(self, predict: Predict) -> List[int]:
        k = self.k
        st = gc_unipc_coeffs(self.sampler, self.S, k, self.unipc_order, self.unipc_corrector)
        m2 = self.x0_km2 if st.use_corrector and st.c_mk2 != 0.0 else None
        full = self._is_full(k)
        if full:
            views = list(range(self.N))
            mk = predict(k, views).contiguous()
            x_c, x_next = gc_unipc_update(st, mk, x_cur=self.x_t, x_prev=self.x_c if st.use_corrector else None,
                                          m_km2=m2, m_km1=self.x0, stream=self.stream)
        else:
            views = self._anchors()
            new = predict(k, views).contiguous()
            x_prev = self.x_c if st.use_corrector else None
            if self.geom:
                mk, x_c, x_next = gc_transport_unipc_geom(self.x0, new, self.pos, self.cams, self.bbox, views, self.K,
                                                          st, x_cur=self.x_t, x_prev=x_prev, m_km2=m2,
                                                          fg_index=self.fg_index, stream=self.stream)
            else:
                corr, wts, idx = self.operator(views)
                mk, x_c, x_next = gc_transport_unipc(self.x0, new, corr, wts, views, st, x_cur=self.x_t,
                                                     x_prev=x_prev, m_km2=m2, index=idx, stream=self.stream)
        self.x0_km2, self.x0, self.x_c, self.x_t = self.x0, mk, x_c, x_next
        self._after(views, full)
        self.k += 1
        return views

    def run(self, predict: Predict, steps: Optional[int] = None) -> None:
        for _ in range(self.S - self.k if steps is None else steps):
            self.step(predict)

    def state_dict(self) -> dict:
        """Loop state for checkpoint / resume (tensors are cloned on the runner's stream)."""
        cl = lambda t: None if t is None else t.clone()
        with self._on_stream():
            return {"k": self.k, "c": self.c, "x_t": cl(self.x_t), "x0": cl(self.x0), "x0_km2": cl(self.x0_km2),
                    "x_c": cl(self.x_c), "stale": cl(self.stale), "stats": cl(self.stats_host), "gap": list(self.gap)}

    def load_state_dict(self, st: dict) -> None:
        with self._on_stream():
            self._load_state_dict(st)

    def _load_state_dict(self, st: dict) -> None:
        cl = lambda t: None if t is None else t.clone()
        self.k, self.c = int(st["k"]), int(st["c"])
        self.x_t, self.x0 = cl(st["x_t"]), cl(st["x0"])
        self.x0_km2, self.x_c = cl(st.get("x0_km2")), cl(st.get("x_c"))
        if self.tracking:
            if st.get("stale") is None:
                raise ValueError("this runner tracks staleness: the state needs 'stale'")
            self.stale = cl(st["stale"])
            self.stats_host = cl(st.get("stats"))
        self.gap = list(st.get("gap", [0] * self.N))
        self._next = None
