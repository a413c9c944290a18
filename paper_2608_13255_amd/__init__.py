"""MI355X-native GeoCache cross-view delta transport.

Python binding of libgeocache.so (hand-written HIP kernels for gfx950 behind
the C ABI declared in include/geocache.h).  Every function here has the name
of the C entry point it wraps and only marshals arguments: it checks torch
tensors (device, dtype, contiguity, shape), allocates outputs the caller did
not supply, passes raw device pointers and the current HIP stream, and turns
a negative status into GeoCacheError.  All computation runs in the library's
kernels; there is no CPU fallback, and importing the package fails if the
library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgeocache.so")
ABI_VERSION = 4   # GC_ABI_VERSION the binding is written for

# constants mirrored from include/geocache.h
GC_OK = 0
GC_F32, GC_BF16 = 0, 1
GC_DDIM, GC_FLOW_EULER = 0, 1
GC_PRED_NONE, GC_PRED_EPS, GC_PRED_V, GC_PRED_VEL = 0, 1, 2, 3
GC_FULL_PERIODIC, GC_FULL_HEAD_MID_TAIL, GC_FULL_HEAD_TAIL_E = 0, 1, 2
GC_MAX_VIEWS, GC_MAX_ANCHORS, GC_MAX_GRID = 64, 8, 4094
GC_NOALLOC_SCRATCH_BYTES = 1 << 20
ERRORS = {-1: "GC_ERR_ARG", -2: "GC_ERR_SHAPE", -3: "GC_ERR_DTYPE", -4: "GC_ERR_ALIGN",
          -5: "GC_ERR_ALIAS", -6: "GC_ERR_CAPACITY", -7: "GC_ERR_HIP"}

# gc_camera: int32 model, float R[9], float t[3], fx, fy, cx, cy (68 bytes)
CAMERA_DTYPE = np.dtype([("model", "<i4"), ("R", "<f4", (9,)), ("t", "<f4", (3,)), ("fx", "<f4"),
                         ("fy", "<f4"), ("cx", "<f4"), ("cy", "<f4")])
assert CAMERA_DTYPE.itemsize == 68


class GeoCacheError(RuntimeError):
    def __init__(self, func: str, code: int, msg: str):
        super().__init__(f"{func} failed with {ERRORS.get(code, code)}: {msg}")
        self.code = code


class _Sampler(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("pred_out", ctypes.c_int32), ("T", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("beta_start", ctypes.c_double), ("beta_end", ctypes.c_double)]


class UniPCStep(ctypes.Structure):
    """gc_unipc_step: coefficients of one UniPC step (gc_unipc_coeffs)."""
    _fields_ = [("use_corrector", ctypes.c_int32), ("corrector_order", ctypes.c_int32),
                ("predictor_order", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("c_xprev", ctypes.c_double), ("c_mk2", ctypes.c_double), ("c_mk1", ctypes.c_double),
                ("c_mk", ctypes.c_double), ("p_xc", ctypes.c_double), ("p_mk1", ctypes.c_double),
                ("p_mk", ctypes.c_double)]


@dataclass(frozen=True)
class Sampler:
    """gc_sampler: kind GC_DDIM (linear betas over T steps) or GC_FLOW_EULER."""
    kind: int = GC_DDIM
    pred_out: int = GC_PRED_NONE
    T: int = 1000
    beta_start: float = 1e-4
    beta_end: float = 0.02

    def c(self) -> _Sampler:
        return _Sampler(self.kind, self.pred_out, self.T, 0, self.beta_start, self.beta_end)


_LIB = None
_vp = ctypes.c_void_p
_i32p = ctypes.POINTER(ctypes.c_int32)
_i = ctypes.c_int
_i64 = ctypes.c_int64


def lib() -> ctypes.CDLL:
    """The loaded libgeocache.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it (python -c 'import __graft_entry__ as g; g.build()' "
                              "or make -C paper_2608_13255_amd)")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "gc_abi_version": ([], _i),
            "gc_last_error": ([], ctypes.c_char_p),
            "gc_posmap_downsample": ([_vp, _i64, _i, _i, _i, _vp, _vp], _i),
            "gc_posmap_bbox": ([_vp, _i, _i, _i, _i, ctypes.c_float, _vp, _vp], _i),
            "gc_build_correspondence": ([_vp, _vp, _i, _i, _i, _i, _i32p, _i, _i, _vp, _vp, _vp, _vp, _vp], _i),
            "gc_index_workspace_bytes": ([_i64], ctypes.c_size_t),
            "gc_index_correspondence": ([_vp, _i64, _i, _i, _i, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp], _i),
            "gc_index_correspondence_noalloc": ([_vp, _i64, _i, _i, _i, _vp, _vp, _vp, _vp], _i),
            "gc_index_foreground": ([_vp, _i64, _i, _i, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp], _i),
            "gc_transport_step": ([_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i, _i, _i, _i, _i, _i32p, _i, _i, _i, _vp,
                                   _vp], _i),
            "gc_sampler_reconstruct": ([_vp, _vp, _vp, _vp, _i64, _i, ctypes.POINTER(_Sampler), ctypes.c_double,
                                        ctypes.c_double, _vp], _i),
            "gc_transport_reconstruct": ([_vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp, _i, _i, _i, _i, _i, _i32p, _i,
                                          _i, _i, ctypes.POINTER(_Sampler), ctypes.c_double, ctypes.c_double, _vp,
                                          _vp, _vp, _vp], _i),
            "gc_unipc_coeffs": ([ctypes.POINTER(_Sampler), _i, _i, _i, _i, ctypes.POINTER(UniPCStep)], _i),
            "gc_unipc_update": ([_vp, _vp, _vp, _vp, _vp, _i64, _i, ctypes.POINTER(UniPCStep), _vp, _vp, _vp], _i),
            "gc_transport_unipc": ([_vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i32p,
                                    _i, _i, _i, ctypes.POINTER(UniPCStep), _vp, _vp, _vp, _vp], _i),
            "gc_transport_step_geom": ([_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i, _i, _i, _i, _i, _i32p, _i, _i,
                                        _i, _vp, _vp], _i),
            "gc_transport_reconstruct_geom": ([_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp, _i, _i, _i, _i, _i,
                                               _i32p, _i, _i, _i, ctypes.POINTER(_Sampler), ctypes.c_double,
                                               ctypes.c_double, _vp, _vp, _vp, _vp], _i),
            "gc_transport_unipc_geom": ([_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _i, _i, _i, _i, _i,
                                         _i32p, _i, _i, _i, ctypes.POINTER(UniPCStep), _vp, _vp, _vp, _vp], _i),
            "gc_coverage_pair_words": ([_i, _i, _i, _i], _i64),
            "gc_coverage_pairs": ([_vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp], _i),
            "gc_coverage_init": ([_vp, _i, _i, _i, _i, _vp, _vp], _i),
            "gc_coverage_update": ([_vp, _i, _i, _i, _i, _i32p, _i, _i, _vp, _vp, _vp], _i),
            "gc_coverage_workspace_bytes": ([], ctypes.c_size_t),
            "gc_coverage_select": ([_vp, _vp, _i, _i, _i, _i, _i, _i32p, _i, _vp, _vp, ctypes.c_size_t, _vp], _i),
            "gc_schedule_refresh_due": ([_vp, _i, _i, ctypes.c_double, ctypes.POINTER(ctypes.c_int)], _i),
            "gc_coverage_score": ([_vp, _vp, _i, _i, _i, _i, _i32p, _i, _i, _vp, _vp, ctypes.c_size_t, _vp], _i),
            "gc_coverage_update_select": ([_vp, _i, _i, _i, _i, _i32p, _i, _i, _vp, _vp, _i, _i32p, _i, _vp, _vp,
                                           ctypes.c_size_t, _vp], _i),
            "gc_coverage_update_score": ([_vp, _i, _i, _i, _i, _i32p, _i, _i, _vp, _vp, _i32p, _i, _i, _vp, _vp,
                                          ctypes.c_size_t, _vp], _i),
            "gc_schedule_forced_views": ([_i32p, _i, _i, _i, _i32p, ctypes.POINTER(ctypes.c_int)], _i),
            "gc_schedule_advance_gaps": ([_i32p, _i, _i32p, _i, _i], _i),
            "gc_schedule_anchors": ([_i, _i, _i64, _i32p], _i),
            "gc_schedule_full_steps": ([_i, _i, _i, ctypes.POINTER(ctypes.c_uint8)], _i),
            "gc_sampler_step_times": ([ctypes.POINTER(_Sampler), _i, _i, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_double)], _i),
            "gc_sampler_alpha_bar": ([ctypes.POINTER(_Sampler), _i, ctypes.POINTER(ctypes.c_double)], _i),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        if L.gc_abi_version() != ABI_VERSION:
            raise ImportError(f"libgeocache ABI {L.gc_abi_version()} != {ABI_VERSION}")
        _LIB = L
    return _LIB


def _check(rc: int, func: str) -> None:
    if rc != GC_OK:
        raise GeoCacheError(func, rc, lib().gc_last_error().decode(errors="replace"))


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _side_stream(stream) -> Optional[torch.cuda.Stream]:
    """The stream of an explicit `stream` argument when it is not torch's
    current stream (None otherwise)."""
    if stream is None:
        return None
    cur = torch.cuda.current_stream()
    s = stream if isinstance(stream, torch.cuda.Stream) else torch.cuda.ExternalStream(int(stream))
    return None if s.cuda_stream == cur.cuda_stream else s


def _keep(stream, tensors) -> None:
    """Tensors this binding allocated and handed to work on a side stream:
    tell torch's caching allocator, so that their memory is not given to
    current-stream work before the side stream's kernels are done with it."""
    s = _side_stream(stream)
    if s is not None:
        for t in tensors:
            t.record_stream(s)


def _after_side(stream) -> None:
    """Order torch's current stream (and so a following host read-back)
    after the work just enqueued on a side stream."""
    s = _side_stream(stream)
    if s is not None:
        torch.cuda.current_stream().wait_stream(s)


def _dev(t: torch.Tensor, name: str) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _opt(t: Optional[torch.Tensor], name: str) -> Optional[int]:
    return None if t is None else _dev(t, name)


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return GC_F32
    if t.dtype == torch.bfloat16:
        return GC_BF16
    raise ValueError(f"latents must be float32 or bfloat16 (got {t.dtype})")


def _anchors(anchors: Sequence[int]):
    arr = (ctypes.c_int32 * len(anchors))(*[int(x) for x in anchors])
    return arr, len(anchors)


def camera_tensor(cams: Dict[str, np.ndarray], device="cuda") -> torch.Tensor:
    """Pack camera arrays (keys model, R, t, fx, fy, cx, cy with a common
    leading shape, e.g. [B][N]) into a device uint8 tensor of gc_camera."""
    lead = np.shape(cams["model"])
    rec = np.zeros(lead, CAMERA_DTYPE)
    rec["model"] = cams["model"]
    rec["R"] = np.reshape(cams["R"], lead + (9,))
    rec["t"] = cams["t"]
    for k in ("fx", "fy", "cx", "cy"):
        rec[k] = cams[k]
    raw = np.ascontiguousarray(rec).view(np.uint8).reshape(lead + (68,))
    return torch.from_numpy(raw.copy()).to(device)


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def gc_posmap_downsample(pos_hi: torch.Tensor, f: int, pos_lat: torch.Tensor = None, stream=None) -> torch.Tensor:
    """pos_hi float32 [..., Hr, Wr, 3] -> pos_lat float32 [..., Hr/f, Wr/f, 3]."""
    if pos_hi.dtype != torch.float32 or pos_hi.dim() < 3 or pos_hi.shape[-1] != 3:
        raise ValueError("pos_hi must be float32 [..., Hr, Wr, 3]")
    Hr, Wr = pos_hi.shape[-3], pos_hi.shape[-2]
    lead = tuple(pos_hi.shape[:-3])
    n = int(np.prod(lead)) if lead else 1
    fresh = []
    if pos_lat is None:
        pos_lat = torch.empty(lead + (Hr // f, Wr // f, 3), dtype=torch.float32, device=pos_hi.device)
        fresh.append(pos_lat)
    _check(lib().gc_posmap_downsample(_dev(pos_hi, "pos_hi"), n, Hr, Wr, f, _dev(pos_lat, "pos_lat"),
                                      _stream(stream)), "gc_posmap_downsample")
    _keep(stream, fresh)
    return pos_lat


def gc_posmap_bbox(pos: torch.Tensor, tol_frac: float = 0.01, bbox: torch.Tensor = None, stream=None) -> torch.Tensor:
    """pos float32 [B, N, H, W, 3] -> bbox float32 [B, 8]."""
    if pos.dtype != torch.float32 or pos.dim() != 5 or pos.shape[-1] != 3:
        raise ValueError("pos must be float32 [B, N, H, W, 3]")
    B, N, H, W, _ = pos.shape
    fresh = []
    if bbox is None:
        bbox = torch.empty((B, 8), dtype=torch.float32, device=pos.device)
        fresh.append(bbox)
    _check(lib().gc_posmap_bbox(_dev(pos, "pos"), B, N, H, W, float(tol_frac), _dev(bbox, "bbox"),
                                _stream(stream)), "gc_posmap_bbox")
    _keep(stream, fresh)
    return bbox


def gc_build_correspondence(pos: torch.Tensor, cams: torch.Tensor, anchors: Sequence[int], K: int,
                            bbox: torch.Tensor, corr: torch.Tensor = None, weights: torch.Tensor = None,
                            stats: torch.Tensor = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """pos float32 [B, N, H, W, 3], cams uint8 [B, N, 68] (camera_tensor),
    bbox float32 [B, 8] -> (corr int32 [B, N-a, H, W, a], weights float32
    [B, N-a, H, W, a, K]); stats (optional) int32/uint32 [B, 4]."""
    if pos.dtype != torch.float32 or pos.dim() != 5 or pos.shape[-1] != 3:
        raise ValueError("pos must be float32 [B, N, H, W, 3]")
    B, N, H, W, _ = pos.shape
    if cams.dtype != torch.uint8 or tuple(cams.shape) != (B, N, 68):
        raise ValueError(f"cams must be uint8 [B={B}, N={N}, 68]")
    arr, a = _anchors(anchors)
    NT = N - a
    dev = pos.device
    fresh = []
    if corr is None:
        corr = torch.empty((B, NT, H, W, a), dtype=torch.int32, device=dev)
        fresh.append(corr)
    if weights is None:
        weights = torch.empty((B, NT, H, W, a, K), dtype=torch.float32, device=dev)
        fresh.append(weights)
    if tuple(corr.shape) != (B, NT, H, W, a) or corr.dtype != torch.int32:
        raise ValueError("corr must be int32 [B, N-a, H, W, a]")
    if tuple(weights.shape) != (B, NT, H, W, a, K) or weights.dtype != torch.float32:
        raise ValueError("weights must be float32 [B, N-a, H, W, a, K]")
    if stats is not None and (tuple(stats.shape) != (B, 4) or stats.element_size() != 4):
        raise ValueError("stats must be a 32-bit [B, 4] tensor")
    _check(lib().gc_build_correspondence(_dev(pos, "pos"), _dev(cams, "cams"), B, N, H, W, arr, a, K,
                                         _dev(bbox, "bbox"), _dev(corr, "corr") if corr.numel() else None,
                                         _dev(weights, "weights") if weights.numel() else None,
                                         _opt(stats, "stats"), _stream(stream)), "gc_build_correspondence")
    _keep(stream, fresh)
    return corr, weights


@dataclass
class VisibleIndex:
    """Output of gc_index_correspondence: vis_bits (int32 view of the uint32
    words), vis_list (int32) and the host count n_vis."""
    vis_bits: torch.Tensor
    vis_list: torch.Tensor
    n_vis: int


def gc_index_correspondence(corr: torch.Tensor, workspace: torch.Tensor = None, stream=None) -> VisibleIndex:
    """Visible-token index of a correspondence (corr int32 [B, N-a, H, W, a]),
    its list in tile order.  Reads the visible count back to the host (one
    synchronisation)."""
    if corr.dtype != torch.int32 or corr.dim() != 5:
        raise ValueError("corr must be int32 [B, N-a, H, W, a]")
    a = corr.shape[-1]
    n_tok = int(corr.numel() // a) if a else 0
    n_views = corr.shape[0] * corr.shape[1] if n_tok else 0
    H, W = max(corr.shape[2], 1), max(corr.shape[3], 1)
    dev = corr.device
    need = int(lib().gc_index_workspace_bytes(n_tok))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace must hold at least {need} bytes")
    bits = torch.empty(max(1, (n_tok + 31) // 32), dtype=torch.int32, device=dev)
    lst = torch.empty(max(1, n_tok), dtype=torch.int32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    _check(lib().gc_index_correspondence(_dev(corr, "corr") if n_tok else None, n_views, H, W, a,
                                         _dev(bits, "vis_bits"), _dev(lst, "vis_list"), _dev(nv, "n_vis"),
                                         _dev(workspace, "workspace"),
                                         workspace.numel() * workspace.element_size(), _stream(stream)),
           "gc_index_correspondence")
    _keep(stream, (bits, lst))
    _after_side(stream)          # the count is read on the current stream
    return VisibleIndex(bits, lst, int(nv.item()))


def gc_index_correspondence_noalloc(corr: torch.Tensor, stream=None) -> VisibleIndex:
    """gc_index_correspondence with the library's own scratch instead of a
    workspace (the C call allocates nothing; this wrapper allocates the
    outputs).  Reads the visible count back to the host."""
    if corr.dtype != torch.int32 or corr.dim() != 5:
        raise ValueError("corr must be int32 [B, N-a, H, W, a]")
    a = corr.shape[-1]
    n_tok = int(corr.numel() // a) if a else 0
    n_views = corr.shape[0] * corr.shape[1] if n_tok else 0
    H, W = max(corr.shape[2], 1), max(corr.shape[3], 1)
    dev = corr.device
    bits = torch.empty(max(1, (n_tok + 31) // 32), dtype=torch.int32, device=dev)
    lst = torch.empty(max(1, n_tok), dtype=torch.int32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    _check(lib().gc_index_correspondence_noalloc(_dev(corr, "corr") if n_tok else None, n_views, H, W, a,
                                                 _dev(bits, "vis_bits"), _dev(lst, "vis_list"), _dev(nv, "n_vis"),
                                                 _stream(stream)), "gc_index_correspondence_noalloc")
    _keep(stream, (bits, lst))
    _after_side(stream)
    return VisibleIndex(bits, lst, int(nv.item()))


@dataclass
class ForegroundIndex:
    """Output of gc_index_foreground: fg_bits (int32 view of the uint32
    words), fg_recs (int32 [capacity, 4] records {token, x, y, z}) and the
    host count n_fg."""
    fg_bits: torch.Tensor
    fg_recs: torch.Tensor
    n_fg: int


def gc_index_foreground(pos: torch.Tensor, workspace: torch.Tensor = None, stream=None) -> ForegroundIndex:
    """Foreground index of position maps (float32 [..., H, W, 3], e.g.
    [B, N, H, W, 3]), once per asset batch; its records in tile order.  Reads
    the foreground count back to the host (one synchronisation)."""
    if pos.dtype != torch.float32 or pos.dim() < 3 or pos.shape[-1] != 3:
        raise ValueError("pos must be float32 [..., H, W, 3]")
    H, W = pos.shape[-3], pos.shape[-2]
    n_tok = int(pos.numel() // 3)
    n_views = n_tok // (H * W) if H * W else 0
    dev = pos.device
    need = int(lib().gc_index_workspace_bytes(n_tok))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace must hold at least {need} bytes")
    bits = torch.empty(max(1, (n_tok + 31) // 32), dtype=torch.int32, device=dev)
    recs = torch.empty((max(1, n_tok), 4), dtype=torch.int32, device=dev)
    nf = torch.empty(1, dtype=torch.int32, device=dev)
    _check(lib().gc_index_foreground(_dev(pos, "pos") if n_tok else None, n_views, max(H, 1), max(W, 1),
                                     _dev(bits, "fg_bits"),
                                     _dev(recs, "fg_recs"), _dev(nf, "n_fg"), _dev(workspace, "workspace"),
                                     workspace.numel() * workspace.element_size(), _stream(stream)),
           "gc_index_foreground")
    _keep(stream, (bits, recs))
    _after_side(stream)          # the count is read on the current stream
    return ForegroundIndex(bits, recs, int(nf.item()))


def _fg_args(fg_index: Optional[ForegroundIndex]):
    if fg_index is None:
        return None, None, 0
    return _dev(fg_index.fg_bits, "fg_bits"), _dev(fg_index.fg_recs, "fg_recs"), int(fg_index.n_fg)


def _index_args(index: Optional[VisibleIndex]):
    if index is None:
        return None, None, 0
    return _dev(index.vis_bits, "vis_bits"), _dev(index.vis_list, "vis_list"), int(index.n_vis)


def _latent_shape(x0_prev: torch.Tensor):
    if x0_prev.dim() != 5:
        raise ValueError("latents must be [B, N, H, W, C]")
    return tuple(x0_prev.shape)


def gc_transport_step(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, corr: torch.Tensor,
                      weights: torch.Tensor, anchors: Sequence[int], x0_out: torch.Tensor = None,
                      index: VisibleIndex = None, stream=None) -> torch.Tensor:
    """Eq. 1 over one cached step; returns x0_out [B, N, H, W, C].  `index`
    (gc_index_correspondence of corr) selects the split launch."""
    B, N, H, W, C = _latent_shape(x0_prev)
    arr, a = _anchors(anchors)
    if tuple(x0_anchor_new.shape) != (B, a, H, W, C) or x0_anchor_new.dtype != x0_prev.dtype:
        raise ValueError(f"x0_anchor_new must be [B, a={a}, H, W, C] of the same dtype as x0_prev")
    K = weights.shape[-1]
    if x0_out is None:
        x0_out = torch.empty_like(x0_prev)
    _check(lib().gc_transport_step(_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
                                   _dev(corr, "corr") if corr.numel() else None,
                                   _dev(weights, "weights") if weights.numel() else None, *_index_args(index),
                                   B, N, H, W, C, arr, a, K, dtype_code(x0_prev), _dev(x0_out, "x0_out"),
                                   _stream(stream)), "gc_transport_step")
    _keep(stream, (x0_out,))
    return x0_out


def gc_sampler_reconstruct(x_t: torch.Tensor, x0: torch.Tensor, sampler: Sampler, t: float, t_next: float,
                           x_next: torch.Tensor = None, model_out: torch.Tensor = None, stream=None):
    """Elementwise sampler step from x0; returns (x_next, model_out or None)."""
    if x0.shape != x_t.shape or x0.dtype != x_t.dtype:
        raise ValueError("x_t and x0 must have the same shape and dtype")
    if x_next is None:
        x_next = torch.empty_like(x_t)
    if sampler.pred_out != GC_PRED_NONE and model_out is None:
        model_out = torch.empty_like(x_t)
    smp = sampler.c()
    _check(lib().gc_sampler_reconstruct(_dev(x_t, "x_t"), _dev(x0, "x0"), _dev(x_next, "x_next"),
                                        _opt(model_out, "model_out"), x_t.numel(), dtype_code(x_t),
                                        ctypes.byref(smp), float(t), float(t_next), _stream(stream)),
           "gc_sampler_reconstruct")
    _keep(stream, [t for t in (x_next, model_out) if t is not None])
    return x_next, model_out


def gc_transport_reconstruct(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, corr: torch.Tensor,
                             weights: torch.Tensor, x_t: torch.Tensor, anchors: Sequence[int], sampler: Sampler,
                             t: float, t_next: float, x0_out: torch.Tensor = None, x_next: torch.Tensor = None,
                             model_out: torch.Tensor = None, index: VisibleIndex = None, stream=None):
    """Fused Eq. 1 + reconstruction; returns (x0_out, x_next, model_out or None).
    `index` (gc_index_correspondence of corr) selects the split launch."""
    B, N, H, W, C = _latent_shape(x0_prev)
    arr, a = _anchors(anchors)
    if tuple(x0_anchor_new.shape) != (B, a, H, W, C) or x0_anchor_new.dtype != x0_prev.dtype:
        raise ValueError(f"x0_anchor_new must be [B, a={a}, H, W, C] of the same dtype as x0_prev")
    if x_t.shape != x0_prev.shape or x_t.dtype != x0_prev.dtype:
        raise ValueError("x_t must match x0_prev in shape and dtype")
    K = weights.shape[-1]
    if x0_out is None:
        x0_out = torch.empty_like(x0_prev)
    if x_next is None:
        x_next = torch.empty_like(x_t)
    if sampler.pred_out != GC_PRED_NONE and model_out is None:
        model_out = torch.empty_like(x_t)
    smp = sampler.c()
    _check(lib().gc_transport_reconstruct(_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
                                          _dev(corr, "corr") if corr.numel() else None,
                                          _dev(weights, "weights") if weights.numel() else None,
                                          *_index_args(index), _dev(x_t, "x_t"), B, N, H, W, C, arr, a, K,
                                          dtype_code(x0_prev),
                                          ctypes.byref(smp), float(t), float(t_next), _dev(x0_out, "x0_out"),
                                          _dev(x_next, "x_next"), _opt(model_out, "model_out"), _stream(stream)),
           "gc_transport_reconstruct")
    _keep(stream, [t for t in (x0_out, x_next, model_out) if t is not None])
    return x0_out, x_next, model_out


def _geom_inputs(x0_prev, x0_anchor_new, pos, cams, bbox, anchors):
    B, N, H, W, C = _latent_shape(x0_prev)
    arr, a = _anchors(anchors)
    if tuple(x0_anchor_new.shape) != (B, a, H, W, C) or x0_anchor_new.dtype != x0_prev.dtype:
        raise ValueError(f"x0_anchor_new must be [B, a={a}, H, W, C] of the same dtype as x0_prev")
    if pos.dtype != torch.float32 or tuple(pos.shape) != (B, N, H, W, 3):
        raise ValueError(f"pos must be float32 [B={B}, N={N}, H={H}, W={W}, 3]")
    if cams.dtype != torch.uint8 or tuple(cams.shape) != (B, N, 68):
        raise ValueError(f"cams must be uint8 [B={B}, N={N}, 68]")
    if bbox.dtype != torch.float32 or tuple(bbox.shape) != (B, 8):
        raise ValueError(f"bbox must be float32 [B={B}, 8]")
    return (B, N, H, W, C), arr, a


def gc_transport_step_geom(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, pos: torch.Tensor,
                           cams: torch.Tensor, bbox: torch.Tensor, anchors: Sequence[int], K: int,
                           x0_out: torch.Tensor = None, fg_index: ForegroundIndex = None, stream=None) -> torch.Tensor:
    """Eq. 1 with G_{A->v} computed on the fly from the position maps
    (pos float32 [B, N, H, W, 3], cams from camera_tensor, bbox from
    gc_posmap_bbox); equals gc_build_correspondence + gc_transport_step.
    `fg_index` (gc_index_foreground of pos) selects the foreground launch."""
    (B, N, H, W, C), arr, a = _geom_inputs(x0_prev, x0_anchor_new, pos, cams, bbox, anchors)
    if x0_out is None:
        x0_out = torch.empty_like(x0_prev)
    fb, fr, nf = _fg_args(fg_index)
    _check(lib().gc_transport_step_geom(_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
                                        _dev(pos, "pos"), _dev(cams, "cams"), _dev(bbox, "bbox"), fb, fr, nf, B, N, H,
                                        W, C, arr, a, K, dtype_code(x0_prev), _dev(x0_out, "x0_out"),
                                        _stream(stream)),
           "gc_transport_step_geom")
    _keep(stream, (x0_out,))
    return x0_out


def gc_transport_reconstruct_geom(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, pos: torch.Tensor,
                                  cams: torch.Tensor, bbox: torch.Tensor, x_t: torch.Tensor, anchors: Sequence[int],
                                  K: int, sampler: Sampler, t: float, t_next: float, x0_out: torch.Tensor = None,
                                  x_next: torch.Tensor = None, model_out: torch.Tensor = None,
                                  fg_index: ForegroundIndex = None, stream=None):
    """gc_transport_reconstruct with G_{A->v} computed on the fly; returns
    (x0_out, x_next, model_out or None).  `fg_index` (gc_index_foreground of
    pos) selects the foreground launch."""
    (B, N, H, W, C), arr, a = _geom_inputs(x0_prev, x0_anchor_new, pos, cams, bbox, anchors)
    if x_t.shape != x0_prev.shape or x_t.dtype != x0_prev.dtype:
        raise ValueError("x_t must match x0_prev in shape and dtype")
    if x0_out is None:
        x0_out = torch.empty_like(x0_prev)
    if x_next is None:
        x_next = torch.empty_like(x_t)
    if sampler.pred_out != GC_PRED_NONE and model_out is None:
        model_out = torch.empty_like(x_t)
    smp = sampler.c()
    fb, fr, nf = _fg_args(fg_index)
    _check(lib().gc_transport_reconstruct_geom(_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
                                               _dev(pos, "pos"), _dev(cams, "cams"), _dev(bbox, "bbox"), fb, fr, nf,
                                               _dev(x_t, "x_t"), B, N, H, W, C, arr, a, K, dtype_code(x0_prev),
                                               ctypes.byref(smp), float(t), float(t_next), _dev(x0_out, "x0_out"),
                                               _dev(x_next, "x_next"), _opt(model_out, "model_out"),
                                               _stream(stream)), "gc_transport_reconstruct_geom")
    _keep(stream, [t for t in (x0_out, x_next, model_out) if t is not None])
    return x0_out, x_next, model_out


class BoundCall:
    """A gc_transport_reconstruct call with every argument but (t, t_next)
    already marshalled: calling it issues exactly one ctypes call.  For
    step loops where per-call Python checks would cost more host time than
    the kernel takes on the GPU."""
    __slots__ = ("_fn", "_pre", "_post", "_smp", "keep")

    def __init__(self, fn, pre, smp, post, keep):
        self._fn, self._pre, self._smp, self._post, self.keep = fn, pre, smp, post, keep

    def __call__(self, t: float, t_next: float) -> None:
        rc = self._fn(*self._pre, ctypes.byref(self._smp), t, t_next, *self._post)
        if rc != GC_OK:
            _check(rc, "gc_transport_reconstruct")


def bind_transport_reconstruct(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, corr: torch.Tensor,
                               weights: torch.Tensor, x_t: torch.Tensor, anchors: Sequence[int], sampler: Sampler,
                               x0_out: torch.Tensor, x_next: torch.Tensor, model_out: torch.Tensor = None,
                               index: VisibleIndex = None, stream=None) -> BoundCall:
    """Marshal gc_transport_reconstruct's buffer arguments once (same checks
    as gc_transport_reconstruct); the returned object takes (t, t_next).
    The tensors must stay alive and unmoved while the object is used."""
    B, N, H, W, C = _latent_shape(x0_prev)
    arr, a = _anchors(anchors)
    if tuple(x0_anchor_new.shape) != (B, a, H, W, C) or x0_anchor_new.dtype != x0_prev.dtype:
        raise ValueError(f"x0_anchor_new must be [B, a={a}, H, W, C] of the same dtype as x0_prev")
    for name, t in (("x_t", x_t), ("x0_out", x0_out), ("x_next", x_next)):
        if t.shape != x0_prev.shape or t.dtype != x0_prev.dtype:
            raise ValueError(f"{name} must match x0_prev in shape and dtype")
    if (sampler.pred_out != GC_PRED_NONE) != (model_out is not None):
        raise ValueError("model_out must be given iff the sampler has a prediction output")
    K = weights.shape[-1]
    pre = (_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
           _dev(corr, "corr") if corr.numel() else None, _dev(weights, "weights") if weights.numel() else None,
           *_index_args(index), _dev(x_t, "x_t"), B, N, H, W, C, arr, a, K, dtype_code(x0_prev))
    post = (_dev(x0_out, "x0_out"), _dev(x_next, "x_next"), _opt(model_out, "model_out"), _stream(stream))
    return BoundCall(lib().gc_transport_reconstruct, pre, sampler.c(), post,
                     (x0_prev, x0_anchor_new, corr, weights, x_t, x0_out, x_next, model_out, arr, index))


def gc_unipc_coeffs(sampler: Sampler, S: int, k: int, order: int = 2, corrector: bool = True) -> UniPCStep:
    st = UniPCStep()
    smp = sampler.c()
    _check(lib().gc_unipc_coeffs(ctypes.byref(smp), S, k, order, int(corrector), ctypes.byref(st)),
           "gc_unipc_coeffs")
    return st


def gc_unipc_update(st: UniPCStep, m_k: torch.Tensor, x_cur: torch.Tensor = None, x_prev: torch.Tensor = None,
                    m_km2: torch.Tensor = None, m_km1: torch.Tensor = None, x_c: torch.Tensor = None,
                    x_next: torch.Tensor = None, stream=None):
    """UniPC update over all elements (a full step); returns (x_c, x_next)."""
    if x_c is None:
        x_c = torch.empty_like(m_k)
    if x_next is None:
        x_next = torch.empty_like(m_k)
    for name, t in (("x_cur", x_cur), ("x_prev", x_prev), ("m_km2", m_km2), ("m_km1", m_km1)):
        if t is not None and (t.shape != m_k.shape or t.dtype != m_k.dtype):
            raise ValueError(f"{name} must match m_k in shape and dtype")
    _check(lib().gc_unipc_update(_opt(x_cur, "x_cur"), _opt(x_prev, "x_prev"), _opt(m_km2, "m_km2"),
                                 _opt(m_km1, "m_km1"), _dev(m_k, "m_k"), m_k.numel(), dtype_code(m_k),
                                 ctypes.byref(st), _dev(x_c, "x_c"), _dev(x_next, "x_next"), _stream(stream)),
           "gc_unipc_update")
    _keep(stream, (x_c, x_next))
    return x_c, x_next


def gc_transport_unipc(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, corr: torch.Tensor,
                       weights: torch.Tensor, anchors: Sequence[int], st: UniPCStep, x_cur: torch.Tensor = None,
                       x_prev: torch.Tensor = None, m_km2: torch.Tensor = None, x0_out: torch.Tensor = None,
                       x_c: torch.Tensor = None, x_next: torch.Tensor = None, index: VisibleIndex = None,
                       stream=None):
    """Fused Eq. 1 + UniPC update; returns (x0_out, x_c, x_next)."""
    B, N, H, W, C = _latent_shape(x0_prev)
    arr, a = _anchors(anchors)
    if tuple(x0_anchor_new.shape) != (B, a, H, W, C) or x0_anchor_new.dtype != x0_prev.dtype:
        raise ValueError(f"x0_anchor_new must be [B, a={a}, H, W, C] of the same dtype as x0_prev")
    for name, t in (("x_cur", x_cur), ("x_prev", x_prev), ("m_km2", m_km2)):
        if t is not None and (t.shape != x0_prev.shape or t.dtype != x0_prev.dtype):
            raise ValueError(f"{name} must match x0_prev in shape and dtype")
    K = weights.shape[-1]
    x0_out = torch.empty_like(x0_prev) if x0_out is None else x0_out
    x_c = torch.empty_like(x0_prev) if x_c is None else x_c
    x_next = torch.empty_like(x0_prev) if x_next is None else x_next
    _check(lib().gc_transport_unipc(_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
                                    _dev(corr, "corr") if corr.numel() else None,
                                    _dev(weights, "weights") if weights.numel() else None, *_index_args(index),
                                    _opt(x_cur, "x_cur"), _opt(x_prev, "x_prev"), _opt(m_km2, "m_km2"),
                                    B, N, H, W, C, arr, a, K, dtype_code(x0_prev), ctypes.byref(st),
                                    _dev(x0_out, "x0_out"), _dev(x_c, "x_c"), _dev(x_next, "x_next"),
                                    _stream(stream)), "gc_transport_unipc")
    _keep(stream, (x0_out, x_c, x_next))
    return x0_out, x_c, x_next


def gc_transport_unipc_geom(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, pos: torch.Tensor,
                            cams: torch.Tensor, bbox: torch.Tensor, anchors: Sequence[int], K: int, st: UniPCStep,
                            x_cur: torch.Tensor = None, x_prev: torch.Tensor = None, m_km2: torch.Tensor = None,
                            x0_out: torch.Tensor = None, x_c: torch.Tensor = None, x_next: torch.Tensor = None,
                            fg_index: ForegroundIndex = None, stream=None):
    """gc_transport_unipc with G_{A->v} computed on the fly; returns
    (x0_out, x_c, x_next).  `fg_index` (gc_index_foreground of pos) selects
    the foreground launch."""
    (B, N, H, W, C), arr, a = _geom_inputs(x0_prev, x0_anchor_new, pos, cams, bbox, anchors)
    for name, t in (("x_cur", x_cur), ("x_prev", x_prev), ("m_km2", m_km2)):
        if t is not None and (t.shape != x0_prev.shape or t.dtype != x0_prev.dtype):
            raise ValueError(f"{name} must match x0_prev in shape and dtype")
    x0_out = torch.empty_like(x0_prev) if x0_out is None else x0_out
    x_c = torch.empty_like(x0_prev) if x_c is None else x_c
    x_next = torch.empty_like(x0_prev) if x_next is None else x_next
    fb, fr, nf = _fg_args(fg_index)
    _check(lib().gc_transport_unipc_geom(_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
                                         _dev(pos, "pos"), _dev(cams, "cams"), _dev(bbox, "bbox"), fb, fr, nf,
                                         _opt(x_cur, "x_cur"), _opt(x_prev, "x_prev"), _opt(m_km2, "m_km2"),
                                         B, N, H, W, C, arr, a, K, dtype_code(x0_prev), ctypes.byref(st),
                                         _dev(x0_out, "x0_out"), _dev(x_c, "x_c"), _dev(x_next, "x_next"),
                                         _stream(stream)), "gc_transport_unipc_geom")
    _keep(stream, (x0_out, x_c, x_next))
    return x0_out, x_c, x_next


class BoundUniPC:
    """A gc_transport_unipc call with its buffer arguments marshalled; the
    object takes the step's coefficients and issues exactly one ctypes call."""
    __slots__ = ("_fn", "_pre", "_post", "keep")

    def __init__(self, fn, pre, post, keep):
        self._fn, self._pre, self._post, self.keep = fn, pre, post, keep

    def __call__(self, st: UniPCStep) -> None:
        rc = self._fn(*self._pre, ctypes.byref(st), *self._post)
        if rc != GC_OK:
            _check(rc, "gc_transport_unipc")


def bind_transport_unipc(x0_prev: torch.Tensor, x0_anchor_new: torch.Tensor, corr: torch.Tensor,
                         weights: torch.Tensor, anchors: Sequence[int], x0_out: torch.Tensor, x_c: torch.Tensor,
                         x_next: torch.Tensor, x_cur: torch.Tensor = None, x_prev: torch.Tensor = None,
                         m_km2: torch.Tensor = None, index: VisibleIndex = None, stream=None) -> BoundUniPC:
    """Marshal gc_transport_unipc's buffer arguments once (same shape checks
    as gc_transport_unipc); the returned object takes a UniPCStep.  The
    tensors must stay alive and unmoved while the object is used."""
    B, N, H, W, C = _latent_shape(x0_prev)
    arr, a = _anchors(anchors)
    if tuple(x0_anchor_new.shape) != (B, a, H, W, C) or x0_anchor_new.dtype != x0_prev.dtype:
        raise ValueError(f"x0_anchor_new must be [B, a={a}, H, W, C] of the same dtype as x0_prev")
    for name, t in (("x_cur", x_cur), ("x_prev", x_prev), ("m_km2", m_km2), ("x0_out", x0_out), ("x_c", x_c),
                    ("x_next", x_next)):
        if t is not None and (t.shape != x0_prev.shape or t.dtype != x0_prev.dtype):
            raise ValueError(f"{name} must match x0_prev in shape and dtype")
    K = weights.shape[-1]
    pre = (_dev(x0_prev, "x0_prev"), _dev(x0_anchor_new, "x0_anchor_new"),
           _dev(corr, "corr") if corr.numel() else None, _dev(weights, "weights") if weights.numel() else None,
           *_index_args(index), _opt(x_cur, "x_cur"), _opt(x_prev, "x_prev"), _opt(m_km2, "m_km2"),
           B, N, H, W, C, arr, a, K, dtype_code(x0_prev))
    post = (_dev(x0_out, "x0_out"), _dev(x_c, "x_c"), _dev(x_next, "x_next"), _stream(stream))
    return BoundUniPC(lib().gc_transport_unipc, pre, post,
                      (x0_prev, x0_anchor_new, corr, weights, x_cur, x_prev, m_km2, x0_out, x_c, x_next, arr, index))


# --------------------------------------------------------------------------
# token staleness and the coverage-driven schedule
# --------------------------------------------------------------------------

def gc_coverage_pairs(pos: torch.Tensor, cams: torch.Tensor, bbox: torch.Tensor, out: torch.Tensor = None,
                      stream=None) -> torch.Tensor:
    """Single-anchor visibility bits: int32 [N, B, N, ceil(H*W/32)] (uint32
    words; bit p % 32 of word p / 32 of row (u, b, v): anchor u sees token p
    of view v)."""
    if pos.dtype != torch.float32 or pos.dim() != 5 or pos.shape[-1] != 3:
        raise ValueError("pos must be float32 [B, N, H, W, 3]")
    B, N, H, W, _ = pos.shape
    if cams.dtype != torch.uint8 or tuple(cams.shape) != (B, N, 68):
        raise ValueError(f"cams must be uint8 [B={B}, N={N}, 68]")
    wpr = (H * W + 31) // 32
    if out is None:
        out = torch.empty((N, B, N, wpr), dtype=torch.int32, device=pos.device)
    if tuple(out.shape) != (N, B, N, wpr) or out.element_size() != 4:
        raise ValueError(f"out must be a 32-bit [{N}, {B}, {N}, {wpr}] tensor")
    _check(lib().gc_coverage_pairs(_dev(pos, "pos"), _dev(cams, "cams"), _dev(bbox, "bbox"), B, N, H, W,
                                   _dev(out, "pair_bits"), _stream(stream)), "gc_coverage_pairs")
    _keep(stream, (out,))
    return out


def gc_coverage_init(pos: torch.Tensor, out: torch.Tensor = None, stream=None) -> torch.Tensor:
    """Staleness uint8 [B, N, H, W]: 0 for foreground tokens, 255 for background."""
    B, N, H, W, _ = pos.shape
    if out is None:
        out = torch.empty((B, N, H, W), dtype=torch.uint8, device=pos.device)
    _check(lib().gc_coverage_init(_dev(pos, "pos"), B, N, H, W, _dev(out, "stale"), _stream(stream)),
           "gc_coverage_init")
    _keep(stream, (out,))
    return out


def gc_coverage_update(pair_bits: torch.Tensor, stale: torch.Tensor, anchors: Sequence[int], R: int,
                       stats: torch.Tensor = None, stream=None) -> torch.Tensor:
    """One step with anchor set `anchors` (every view for a full step):
    staleness updated in place; returns stats int32 [B, N, 4] (foreground,
    staleness >= R, sum, max)."""
    if stale.dtype != torch.uint8 or stale.dim() != 4:
        raise ValueError("stale must be uint8 [B, N, H, W]")
    B, N, H, W = stale.shape
    arr = (ctypes.c_int32 * len(anchors))(*anchors)
    if stats is None:
        stats = torch.empty((B, N, 4), dtype=torch.int32, device=stale.device)
    if tuple(stats.shape) != (B, N, 4) or stats.element_size() != 4:
        raise ValueError(f"stats must be a 32-bit [{B}, {N}, 4] tensor")
    _check(lib().gc_coverage_update(_dev(pair_bits, "pair_bits"), B, N, H, W, arr, len(anchors), R,
                                    _dev(stale, "stale"), _dev(stats, "stats"), _stream(stream)),
           "gc_coverage_update")
    _keep(stream, (stats,))
    return stats


def gc_coverage_workspace_bytes() -> int:
    return int(lib().gc_coverage_workspace_bytes())


def gc_coverage_select(pair_bits: torch.Tensor, stale: torch.Tensor, a: int, forced: Sequence[int] = (),
                       out: torch.Tensor = None, workspace: torch.Tensor = None, stream=None) -> torch.Tensor:
    """Anchor set of the next cached step (greedy weighted maximum coverage):
    device int32 [a], ascending.  Enqueued only: read it after a sync."""
    B, N, H, W = stale.shape
    if out is None:
        out = torch.empty(a, dtype=torch.int32, device=stale.device)
    if workspace is None:
        workspace = torch.empty(gc_coverage_workspace_bytes(), dtype=torch.uint8, device=stale.device)
    farr = (ctypes.c_int32 * max(len(forced), 1))(*forced)
    _check(lib().gc_coverage_select(_dev(pair_bits, "pair_bits"), _dev(stale, "stale"), B, N, H, W, a, farr,
                                    len(forced), _dev(out, "anchors_out"), _dev(workspace, "workspace"),
                                    workspace.numel() * workspace.element_size(), _stream(stream)),
           "gc_coverage_select")
    _keep(stream, (out, workspace))
    return out


def gc_coverage_score(pair_bits: torch.Tensor, stale: torch.Tensor, sets: Sequence[Sequence[int]],
                      out: torch.Tensor = None, workspace: torch.Tensor = None, stream=None) -> torch.Tensor:
    """Weighted coverage of each candidate set: device int64 [M] (uint64 values)."""
    B, N, H, W = stale.shape
    M, a = len(sets), len(sets[0])
    if any(len(S) != a for S in sets):
        raise ValueError("candidate sets must have the same size")
    flat = (ctypes.c_int32 * (M * a))(*[int(u) for S in sets for u in S])
    if out is None:
        out = torch.empty(M, dtype=torch.int64, device=stale.device)
    if workspace is None:
        workspace = torch.empty(gc_coverage_workspace_bytes(), dtype=torch.uint8, device=stale.device)
    _check(lib().gc_coverage_score(_dev(pair_bits, "pair_bits"), _dev(stale, "stale"), B, N, H, W, flat, M, a,
                                   _dev(out, "scores"), _dev(workspace, "workspace"),
                                   workspace.numel() * workspace.element_size(), _stream(stream)),
           "gc_coverage_score")
    _keep(stream, (out, workspace))
    return out


def _stats_out(stale: torch.Tensor, stats: Optional[torch.Tensor]) -> torch.Tensor:
    B, N = stale.shape[:2]
    if stats is None:
        stats = torch.empty((B, N, 4), dtype=torch.int32, device=stale.device)
    if tuple(stats.shape) != (B, N, 4) or stats.element_size() != 4:
        raise ValueError(f"stats must be a 32-bit [{B}, {N}, 4] tensor")
    return stats


def gc_coverage_update_select(pair_bits: torch.Tensor, stale: torch.Tensor, anchors: Sequence[int], R: int,
                              a_next: int, forced: Sequence[int] = (), stats: torch.Tensor = None,
                              out: torch.Tensor = None, workspace: torch.Tensor = None, stream=None):
    """gc_coverage_update with `anchors`, then gc_coverage_select of `a_next`
    views on the updated staleness, in one pass over the tokens; returns
    (stats int32 [B, N, 4], selection device int32 [a_next])."""
    if stale.dtype != torch.uint8 or stale.dim() != 4:
        raise ValueError("stale must be uint8 [B, N, H, W]")
    B, N, H, W = stale.shape
    arr = (ctypes.c_int32 * len(anchors))(*anchors)
    stats = _stats_out(stale, stats)
    if out is None:
        out = torch.empty(a_next, dtype=torch.int32, device=stale.device)
    if workspace is None:
        workspace = torch.empty(gc_coverage_workspace_bytes(), dtype=torch.uint8, device=stale.device)
    farr = (ctypes.c_int32 * max(len(forced), 1))(*forced)
    _check(lib().gc_coverage_update_select(_dev(pair_bits, "pair_bits"), B, N, H, W, arr, len(anchors), R,
                                           _dev(stale, "stale"), _dev(stats, "stats"), a_next, farr, len(forced),
                                           _dev(out, "anchors_out"), _dev(workspace, "workspace"),
                                           workspace.numel() * workspace.element_size(), _stream(stream)),
           "gc_coverage_update_select")
    _keep(stream, (stats, out, workspace))
    return stats, out


def gc_coverage_update_score(pair_bits: torch.Tensor, stale: torch.Tensor, anchors: Sequence[int], R: int,
                             sets: Sequence[Sequence[int]], stats: torch.Tensor = None, out: torch.Tensor = None,
                             workspace: torch.Tensor = None, stream=None):
    """gc_coverage_update with `anchors`, then gc_coverage_score of `sets` on
    the updated staleness, in one pass over the tokens; returns (stats int32
    [B, N, 4], scores device int64 [M])."""
    if stale.dtype != torch.uint8 or stale.dim() != 4:
        raise ValueError("stale must be uint8 [B, N, H, W]")
    B, N, H, W = stale.shape
    arr = (ctypes.c_int32 * len(anchors))(*anchors)
    M, a_set = len(sets), len(sets[0])
    if any(len(S) != a_set for S in sets):
        raise ValueError("candidate sets must have the same size")
    flat = (ctypes.c_int32 * (M * a_set))(*[int(u) for S in sets for u in S])
    stats = _stats_out(stale, stats)
    if out is None:
        out = torch.empty(M, dtype=torch.int64, device=stale.device)
    if workspace is None:
        workspace = torch.empty(gc_coverage_workspace_bytes(), dtype=torch.uint8, device=stale.device)
    _check(lib().gc_coverage_update_score(_dev(pair_bits, "pair_bits"), B, N, H, W, arr, len(anchors), R,
                                          _dev(stale, "stale"), _dev(stats, "stats"), flat, M, a_set,
                                          _dev(out, "scores"), _dev(workspace, "workspace"),
                                          workspace.numel() * workspace.element_size(), _stream(stream)),
           "gc_coverage_update_score")
    _keep(stream, (stats, out, workspace))
    return stats, out


def gc_schedule_refresh_due(stats_host, tau: float) -> bool:
    """stats as returned by gc_coverage_update, on the host (numpy or CPU tensor)."""
    import numpy as np
    st = np.ascontiguousarray(stats_host.numpy() if isinstance(stats_host, torch.Tensor) else stats_host)
    if st.dtype.itemsize != 4 or st.ndim != 3 or st.shape[2] != 4:
        raise ValueError("stats must be 32-bit [B, N, 4]")
    due = ctypes.c_int()
    _check(lib().gc_schedule_refresh_due(st.ctypes.data, st.shape[0], st.shape[1], float(tau), ctypes.byref(due)),
           "gc_schedule_refresh_due")
    return bool(due.value)


def gc_schedule_forced_views(gap: Sequence[int], a: int, max_gap: int) -> List[int]:
    """Views whose anchor gap reached max_gap, longest gap first (ties: lower view), at most a."""
    N = len(gap)
    g = (ctypes.c_int32 * max(N, 1))(*[int(x) for x in gap])
    out = (ctypes.c_int32 * max(a, 1))()
    n = ctypes.c_int()
    _check(lib().gc_schedule_forced_views(g, N, a, max_gap, out, ctypes.byref(n)), "gc_schedule_forced_views")
    return list(out[:n.value])


def gc_schedule_advance_gaps(gap: Sequence[int], views: Sequence[int], full: bool) -> List[int]:
    """The anchor gaps after a step that predicted `views` (all views if full)."""
    N = len(gap)
    g = (ctypes.c_int32 * max(N, 1))(*[int(x) for x in gap])
    arr, n = _anchors(views)
    _check(lib().gc_schedule_advance_gaps(g, N, arr, n, int(bool(full))), "gc_schedule_advance_gaps")
    return list(g[:N])


def gc_schedule_anchors(N: int, a: int, c: int) -> List[int]:
    out = (ctypes.c_int32 * a)()
    _check(lib().gc_schedule_anchors(N, a, c, out), "gc_schedule_anchors")
    return list(out)


def gc_schedule_full_steps(rule: int, S: int, E: int = 0) -> List[int]:
    out = (ctypes.c_uint8 * S)()
    _check(lib().gc_schedule_full_steps(rule, S, E, out), "gc_schedule_full_steps")
    return list(out)


def gc_sampler_step_times(sampler: Sampler, S: int, k: int) -> Tuple[float, float]:
    t, tn = ctypes.c_double(), ctypes.c_double()
    smp = sampler.c()
    _check(lib().gc_sampler_step_times(ctypes.byref(smp), S, k, ctypes.byref(t), ctypes.byref(tn)),
           "gc_sampler_step_times")
    return t.value, tn.value


def gc_sampler_alpha_bar(sampler: Sampler, t: int) -> float:
    out = ctypes.c_double()
    smp = sampler.c()
    _check(lib().gc_sampler_alpha_bar(ctypes.byref(smp), int(t), ctypes.byref(out)), "gc_sampler_alpha_bar")
    return out.value


lib()
