"""C-ABI checks that need no GPU: the library loads, exports exactly what
include/geocache.h declares, rejects bad arguments on the host before any
launch, and its host schedule agrees with the oracle's."""
import ctypes
import math
import os
import re
import shutil
import subprocess
import sys

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "geocache.h")
LIBSO = os.path.join(ROOT, "paper_2608_13255_amd", "libgeocache.so")

# fake, never-dereferenced device addresses: every call below fails validation
# before anything is launched
A0, A1, A2, A3, A4, A5, A6, A7 = (0x10000000 * (i + 1) for i in range(8))


def header_abi_version():
    return int(re.search(r"#define GC_ABI_VERSION (\d+)", open(HEADER).read()).group(1))


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int64_t|int|size_t|const char\*)\s+(gc_\w+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def gc():
    import paper_2608_13255_amd as gc
    return gc


@pytest.fixture(scope="module")
def L(gc):
    assert gc.ABI_VERSION == header_abi_version()
    return gc.lib()


def test_exports_match_header(L):
    declared = header_functions()
    assert len(declared) >= 12
    out = subprocess.run(["nm", "-D", "--defined-only", LIBSO], capture_output=True, text=True, check=True).stdout
    exported = sorted(set(re.findall(r"\sT\s+(gc_\w+)$", out, flags=re.M)))
    assert exported == declared
    for name in declared:
        assert getattr(L, name) is not None
    assert L.gc_abi_version() == header_abi_version()


def test_binding_types_every_entry_point(L):
    """The Python binding declares argument and result types for every
    function the header declares (ctypes would otherwise pass them untyped)."""
    for name in header_functions():
        f = getattr(L, name)
        assert f.argtypes is not None, name
        assert f.restype is not None, name


def test_struct_layouts(gc):
    assert gc.CAMERA_DTYPE.itemsize == 68
    assert ctypes.sizeof(gc._Sampler) == 32


def _err(L):
    return L.gc_last_error().decode()


def test_transport_validation(gc, L):
    anchors = (ctypes.c_int32 * 2)(0, 3)

    def call(x0_prev=A0, new=A1, corr=A2, w=A3, B=1, N=6, H=8, W=8, C=16, anc=anchors, a=2, K=4, dt=1, out=A4,
             bits=None, lst=None, nv=0):
        return L.gc_transport_step(x0_prev, new, corr, w, bits, lst, nv, B, N, H, W, C, anc, a, K, dt, out, None)

    assert call(x0_prev=None) == -1 and "null" in _err(L)
    assert call(a=0) == -1
    assert call(a=7) == -1
    assert call(K=5) == -1 and "K=5" in _err(L)
    assert call(K=0) == -1
    assert call(C=6) == -2
    assert call(C=260) == -6
    assert call(N=65, a=2) == -6
    assert call(H=4095) == -6
    assert call(dt=7) == -3
    assert call(x0_prev=A0 + 8) == -4
    assert call(out=A0 + 16) == -5            # x0_out overlaps x0_prev
    dup = (ctypes.c_int32 * 2)(3, 3)
    assert call(anc=dup) == -1 and "twice" in _err(L)
    bad = (ctypes.c_int32 * 2)(0, 6)
    assert call(anc=bad) == -1
    assert call(corr=None) == -1               # targets exist, so the operator is required
    nine = (ctypes.c_int32 * 9)(*range(9))
    assert call(anc=nine, a=9, N=12) == -6
    assert call(bits=A5) == -1                  # an index needs both the bits and the list
    assert call(bits=A5, lst=A5 + 4096, nv=-1) == -1
    assert call(bits=A5, lst=A5 + 4096, nv=1 * 4 * 64 + 1) == -1   # more visible tokens than targets
    assert call(bits=A5 + 4, lst=A5 + 4096, nv=3) == -4


def test_index_checked_below_the_split_bound():
    """A step smaller than the split launch's bound (2^18 work items by
    default) takes the plain launch, but its index is still validated on the
    host: run in a process that keeps the library's default bound (the test
    suite lowers it to 0)."""
    code = f"""
import ctypes
L = ctypes.CDLL({LIBSO!r})
L.gc_last_error.restype = ctypes.c_char_p
anchors = (ctypes.c_int32 * 2)(0, 3)
def call(bits, lst, nv):
    return L.gc_transport_step(ctypes.c_void_p({A0}), ctypes.c_void_p({A1}), ctypes.c_void_p({A2}),
                               ctypes.c_void_p({A3}), ctypes.c_void_p(bits), ctypes.c_void_p(lst),
                               ctypes.c_int64(nv), 1, 6, 8, 8, 16, anchors, 2, 4, 1, ctypes.c_void_p({A4}), None)
assert call({A5}, None, 0) == -1, L.gc_last_error()
assert call({A5}, {A5} + 4096, -1) == -1, L.gc_last_error()
assert call({A5}, {A5} + 4096, 1 * 4 * 64 + 1) == -1, L.gc_last_error()
assert call({A5} + 4, {A5} + 4096, 3) == -4, L.gc_last_error()
print("index checked")
"""
    env = {k: v for k, v in os.environ.items() if k != "GC_SPLIT_MIN_ITEMS"}
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and "index checked" in r.stdout, r.stdout + r.stderr


def test_fused_validation(gc, L):
    anchors = (ctypes.c_int32 * 2)(0, 3)
    smp = gc.Sampler(kind=gc.GC_FLOW_EULER).c()
    n = 1 * 6 * 8 * 8 * 16 * 2

    def call(xt=A5, smpp=ctypes.byref(smp), t=0.5, tn=0.4, out=A4, xn=A5 + n, mo=None):
        return L.gc_transport_reconstruct(A0, A1, A2, A3, None, None, 0, xt, 1, 6, 8, 8, 16, anchors, 2, 4, 1,
                                          smpp, t, tn, out, xn, mo, None)

    assert call(t=0.0) == -1                   # sigma_t must be > 0
    assert call(tn=0.6) == -1                  # sigma_next must not exceed sigma_t
    assert call(smpp=None) == -1
    assert call(mo=A5 + 4 * n) == -1           # pred NONE but model_out given
    assert call(xn=A4) == -5                   # x_next == x0_out
    bad = gc.Sampler(kind=gc.GC_DDIM, pred_out=gc.GC_PRED_VEL).c()
    assert call(smpp=ctypes.byref(bad), t=500, tn=400) == -1
    ddim = gc.Sampler(kind=gc.GC_DDIM).c()
    assert call(smpp=ctypes.byref(ddim), t=500.5, tn=400) == -1
    assert call(smpp=ctypes.byref(ddim), t=1000, tn=400) == -1


def test_reconstruct_and_build_validation(gc, L):
    smp = gc.Sampler(kind=gc.GC_DDIM, pred_out=gc.GC_PRED_EPS).c()
    assert L.gc_sampler_reconstruct(A0, A1, A2, None, 64, 0, ctypes.byref(smp), 500, 400, None) == -1
    assert L.gc_sampler_reconstruct(A0, A1, A2, A3, 66, 0, ctypes.byref(smp), 500, 400, None) == -2
    assert L.gc_sampler_reconstruct(A0, A1, A0 + 16, A3, 64, 0, ctypes.byref(smp), 500, 400, None) == -5
    anchors = (ctypes.c_int32 * 1)(0)
    assert L.gc_build_correspondence(A0, A1, 1, 4, 8, 8, anchors, 1, 0, A2, A3, A4, None, None) == -1
    assert L.gc_build_correspondence(A0, A1, 1, 4, 8, 8, anchors, 1, 4, A2, A0, A4, None, None) == -5
    assert L.gc_build_correspondence(A0, A1, 1, 4, 5000, 8, anchors, 1, 4, A2, A3, A4, None, None) == -6
    assert L.gc_posmap_downsample(A0, 2, 30, 32, 8, A1, None) == -2
    assert L.gc_posmap_downsample(A0, 2, 32, 32, 8, A0 + 64, None) == -5
    assert L.gc_posmap_bbox(A0, 1, 4, 8, 8, 0.0, A1, None) == -1
    assert L.gc_posmap_bbox(A0, 1, 4, 8, 8, 0.01, A1 + 4, None) == -4
    need = L.gc_index_workspace_bytes(1 << 20)
    assert need >= 2 * 4 * 1024 and need % 256 == 0
    # visible-token index: 64 views of 128 x 128 tokens = 2^20
    assert L.gc_index_correspondence(A0, 64, 128, 128, 4, A1, A2, A3, A4, need - 1, None) == -6
    assert L.gc_index_correspondence(A0, 64, 128, 128, 9, A1, A2, A3, A4, need, None) == -1
    assert L.gc_index_correspondence(A0, 64, 128, 128, 4, A1, A0 + 64, A3, A4, need, None) == -5
    assert L.gc_index_correspondence(A0, -1, 128, 128, 4, A1, A2, A3, A4, need, None) == -2
    assert L.gc_index_correspondence(A0, 64, 0, 128, 4, A1, A2, A3, A4, need, None) == -2
    assert L.gc_index_correspondence(A0, 64, 128, 5000, 4, A1, A2, A3, A4, need, None) == -6
    assert L.gc_index_correspondence(A0, 1 << 17, 128, 128, 4, A1, A2, A3, A4, need, None) == -6   # 2^31 tokens
    # foreground index of position maps: pos, bits, records, count, workspace
    assert L.gc_index_foreground(A0, 64, 128, 128, A1, A2, A3, A4, need - 1, None) == -6
    assert L.gc_index_foreground(A0, 64, 128, 128, A1, A2, None, A4, need, None) == -1
    assert L.gc_index_foreground(None, 64, 128, 128, A1, A2, A3, A4, need, None) == -1
    assert L.gc_index_foreground(A0, -1, 128, 128, A1, A2, A3, A4, need, None) == -2
    assert L.gc_index_foreground(A0, 64, 128, 0, A1, A2, A3, A4, need, None) == -2
    assert L.gc_index_foreground(A0, 1 << 31, 1, 1, A1, A2, A3, A4, need, None) == -6
    assert L.gc_index_foreground(A0, 64, 128, 128, A1, A2 + 8, A3, A4, need, None) == -4
    assert L.gc_index_foreground(A0, 64, 128, 128, A1, A0 + 64, A3, A4, need, None) == -5   # records overlap the maps
    assert L.gc_index_foreground(A0, 64, 128, 128, A1, A2, A2 + 16, A4, need, None) == -5   # count inside the records
    assert L.gc_index_foreground(A0, 64, 128, 128, A1, A2, A3, A1 + 16, need, None) == -5   # workspace over the bits


def test_host_schedule_matches_oracle(gc):
    for N, a in [(4, 1), (6, 2), (10, 3), (12, 4), (7, 3), (6, 6)]:
        for c in range(2 * N + 3):
            assert gc.gc_schedule_anchors(N, a, c) == oracle.anchors(N, a, c)
        win = math.ceil(N / a)
        for c0 in range(N):
            seen = set()
            for c in range(c0, c0 + win):
                seen |= set(gc.gc_schedule_anchors(N, a, c))
            assert seen == set(range(N))
    for rule, name, S, E in [(0, "periodic", 30, 5), (0, "periodic", 30, 4), (1, "head_mid_tail", 30, 0),
                             (1, "head_mid_tail", 50, 0), (1, "head_mid_tail", 10, 0), (0, "periodic", 1, 3),
                             (2, "head_tail_e", 10, 5), (2, "head_tail_e", 30, 1), (2, "head_tail_e", 8, 0),
                             (2, "head_tail_e", 6, 6), (2, "head_tail_e", 1, 1)]:
        assert gc.gc_schedule_full_steps(rule, S, E) == oracle.full_steps(name, S, E)
    ddim = gc.Sampler(kind=gc.GC_DDIM)
    flow = gc.Sampler(kind=gc.GC_FLOW_EULER)
    for S in (1, 10, 30, 50):
        for k in range(S):
            assert gc.gc_sampler_step_times(ddim, S, k) == oracle.step_times("ddim", S, k)
            t, tn = gc.gc_sampler_step_times(flow, S, k)
            ot, otn = oracle.step_times("flow", S, k)
            assert abs(t - ot) < 1e-15 and abs(tn - otn) < 1e-15
    for t in (-1, 0, 32, 500, 999):
        assert abs(gc.gc_sampler_alpha_bar(ddim, t) - oracle.alpha_bar(t)) <= 1e-15
    with pytest.raises(gc.GeoCacheError):
        gc.gc_schedule_anchors(6, 7, 0)
    with pytest.raises(gc.GeoCacheError):
        gc.gc_schedule_full_steps(5, 10, 1)
    with pytest.raises(gc.GeoCacheError):
        gc.gc_schedule_full_steps(2, 10, 11)


def test_product_fails_loudly_without_library(tmp_path):
    pkg = tmp_path / "paper_2608_13255_amd"
    pkg.mkdir()
    shutil.copy(os.path.join(ROOT, "paper_2608_13255_amd", "__init__.py"), pkg / "__init__.py")
    r = subprocess.run([sys.executable, "-c", "import paper_2608_13255_amd"], cwd=tmp_path,
                       capture_output=True, text=True)
    assert r.returncode != 0 and "libgeocache.so is missing" in r.stderr


def test_product_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2608_13255_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h", "Makefile")) or f == "Makefile":
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"\boracle\b|\borc_\w+|liboracle|\bsynth\b", text), f


def test_unipc_validation(gc, L):
    ddim = gc.Sampler(kind=gc.GC_DDIM).c()
    st = gc.UniPCStep()
    assert ctypes.sizeof(st) == 72
    flow = gc.Sampler(kind=gc.GC_FLOW_EULER).c()
    assert L.gc_unipc_coeffs(ctypes.byref(flow), 10, 0, 2, 1, ctypes.byref(st)) == -1
    assert L.gc_unipc_coeffs(ctypes.byref(ddim), 10, 0, 3, 1, ctypes.byref(st)) == -1
    assert L.gc_unipc_coeffs(ctypes.byref(ddim), 10, 10, 2, 1, ctypes.byref(st)) == -1
    assert L.gc_unipc_coeffs(ctypes.byref(ddim), 10, 5, 2, 1, None) == -1
    assert L.gc_unipc_coeffs(ctypes.byref(ddim), 10, 5, 2, 1, ctypes.byref(st)) == 0
    assert st.use_corrector == 1 and st.corrector_order == 2 and st.predictor_order == 2
    assert st.c_mk2 != 0.0 and st.p_mk1 != 0.0
    n = 64
    nb = 4 * n

    def upd(x_cur=A0, x_prev=A1, m2=A2, m1=A3, mk=A4, n_el=n, dt=0, stp=ctypes.byref(st), xc=A5, xn=A5 + nb):
        return L.gc_unipc_update(x_cur, x_prev, m2, m1, mk, n_el, dt, stp, xc, xn, None)

    assert upd(stp=None) == -1
    assert upd(x_prev=None) == -1 and "x_prev" in _err(L)
    assert upd(m2=None) == -1 and "m_{k-2}" in _err(L)
    assert upd(m1=None) == -1
    assert upd(n_el=66) == -2
    assert upd(dt=7) == -3
    assert upd(m2=A2 + 8) == -4
    assert upd(xc=A4) == -5                     # x_c on m_k
    assert upd(xn=A5 + 16) == -5                # x_next overlaps x_c
    assert upd(n_el=0, xc=A1, xn=A0) == 0       # in place (x_c on x_prev, x_next on x_cur); n = 0 launches nothing
    assert L.gc_unipc_coeffs(ctypes.byref(ddim), 10, 0, 2, 1, ctypes.byref(st)) == 0
    assert st.use_corrector == 0 and st.predictor_order == 1 and st.p_mk1 == 0.0
    assert upd(x_cur=None) == -1 and "x_cur" in _err(L)
    anchors = (ctypes.c_int32 * 2)(0, 3)
    big = 1 * 6 * 8 * 8 * 16 * 4

    def fused(xc=A5, xn=A5 + big, x_cur=A4 + big, out=A4 + 2 * big):
        return L.gc_transport_unipc(A0, A1, A2, A3, None, None, 0, x_cur, None, None, 1, 6, 8, 8, 16, anchors, 2, 4,
                                    0, ctypes.byref(st), out, xc, xn, None)

    assert fused(xc=None) == -1
    assert fused(x_cur=None) == -1
    assert fused(xn=A5 + 64) == -5              # x_next overlaps x_c
    assert fused(out=A0 + 64) == -5             # x0_out overlaps x0_prev


def test_geom_validation(gc, L):
    anchors = (ctypes.c_int32 * 2)(0, 3)
    n = 1 * 6 * 8 * 8 * 16 * 2

    def step(prev=A0, new=A1, pos=A2, cams=A3, bbox=A4, C=16, a=2, K=4, dt=1, out=A5, anc=anchors, fb=None, fr=None,
             nf=0):
        return L.gc_transport_step_geom(prev, new, pos, cams, bbox, fb, fr, nf, 1, 6, 8, 8, C, anc, a, K, dt, out,
                                        None)

    assert step(pos=None) == -1 and "null" in _err(L)
    assert step(cams=None) == -1
    assert step(K=0) == -1
    assert step(a=9) == -1
    assert step(C=6) == -2
    assert step(dt=5) == -3
    assert step(pos=A2 + 4) == -4
    assert step(out=A0 + 32) == -5                # x0_out overlaps x0_prev
    assert step(out=A2 + 64) == -5                # x0_out overlaps the position maps
    dup = (ctypes.c_int32 * 2)(1, 1)
    assert step(anc=dup) == -1 and "twice" in _err(L)
    # the optional foreground index (6 * 8 * 8 = 384 tokens)
    assert step(fr=A6) == -1 and "without fg_bits" in _err(L)
    assert step(nf=3) == -1
    assert step(fb=A6, nf=385) == -1 and "n_fg" in _err(L)
    assert step(fb=A6, nf=-1) == -1
    assert step(fb=A6, nf=5) == -1 and "fg_recs" in _err(L)
    assert step(fb=A6 + 4, fr=A7, nf=5) == -4
    assert step(fb=A6, fr=A7 + 8, nf=5) == -4
    assert step(fb=A6, fr=A7, nf=5, out=A7 - 64) == -5     # x0_out overlaps the records
    assert step(fb=A6, fr=A7, nf=5, out=A6 - 64) == -5     # x0_out overlaps the bits
    smp = gc.Sampler(kind=gc.GC_FLOW_EULER).c()

    def fused(xt=A5 + 4 * n, xn=A5 + 8 * n, mo=None, t=0.5, tn=0.4, fb=None, fr=None, nf=0):
        return L.gc_transport_reconstruct_geom(A0, A1, A2, A3, A4, fb, fr, nf, xt, 1, 6, 8, 8, 16, anchors, 2, 4, 1,
                                               ctypes.byref(smp), t, tn, A5, xn, mo, None)

    assert fused(xt=None) == -1
    assert fused(t=0.0) == -1
    assert fused(mo=A5 + 12 * n) == -1            # model_out without a prediction output
    assert fused(xn=A5 + 64) == -5                # x_next overlaps x0_out
    assert fused(xt=A5 + 64) == -5                # x_t overlaps x0_out
    assert fused(fb=A6, fr=A7, nf=5, xn=A7 - 64) == -5   # x_next overlaps the records
    assert fused(fb=A6, nf=2) == -1


def test_unipc_geom_validation(gc, L):
    anchors = (ctypes.c_int32 * 2)(0, 3)
    n = 1 * 6 * 8 * 8 * 16 * 2
    st = gc.UniPCStep()
    rc = L.gc_unipc_coeffs(ctypes.byref(gc.Sampler(kind=gc.GC_DDIM).c()), 10, 4, 2, 1, ctypes.byref(st))
    assert rc == 0 and st.use_corrector == 1 and st.c_mk2 != 0.0

    def call(xcur=A5 + 4 * n, xprev=A5 + 8 * n, m2=A5 + 12 * n, xc=A5 + 16 * n, xn=A5 + 20 * n, out=A5, s=st,
             fb=None, fr=None, nf=0, pos=A2):
        return L.gc_transport_unipc_geom(A0, A1, pos, A3, A4, fb, fr, nf, xcur, xprev, m2, 1, 6, 8, 8, 16, anchors, 2,
                                         4, 1, ctypes.byref(s) if s is not None else None, out, xc, xn, None)

    assert call(s=None) == -1 and "coefficients" in _err(L)
    assert call(xprev=None) == -1 and "corrector" in _err(L)
    assert call(m2=None) == -1 and "m_{k-2}" in _err(L)
    assert call(xc=None) == -1
    assert call(pos=None) == -1
    assert call(xc=A5 + 16 * n + 4) == -4
    assert call(xn=A0 + 64) == -5               # x_next overlaps x0_prev
    assert call(xc=A5 + 4 * n) == -5            # x_c over x_cur (only x_prev allowed)
    assert call(xn=A5 + 8 * n) == -5            # x_next over x_prev (only x_cur allowed)
    assert call(xc=A5 + 20 * n) == -5           # x_c over x_next
    assert call(out=A2) == -5                   # x0_out over the position maps
    assert call(fb=A6, nf=3) == -1              # records missing
    assert call(fb=A6, fr=A7, nf=5, xn=A7 - 64) == -5


def test_error_message_is_per_thread(gc, L):
    """gc_last_error() reports the calling thread's last failure, also while
    another thread fails differently at the same time."""
    import threading
    bad = {}
    barrier = threading.Barrier(2)
    anchors = (ctypes.c_int32 * 2)(0, 3)

    def worker(name, K, dt, rc_want, text):
        barrier.wait()
        for _ in range(500):
            rc = L.gc_transport_step(A0, A1, A2, A3, None, None, 0, 1, 6, 8, 8, 16, anchors, 2, K, dt, A4, None)
            msg = L.gc_last_error().decode()
            if rc != rc_want or text not in msg:
                bad[name] = (rc, msg)

    t1 = threading.Thread(target=worker, args=("K", 5, 1, -1, "K=5"))
    t2 = threading.Thread(target=worker, args=("dtype", 4, 7, -3, "dtype"))
    t1.start(); t2.start(); t1.join(); t2.join()
    assert not bad, bad


def test_index_lane_counts_fit_32_bits(gc, L):
    """The split launches number their gather / list lanes in 32 bits; index
    sizes whose lane count would exceed 2^31 - 1 are rejected on the host
    (GC_ERR_CAPACITY) before anything is launched, and sizes at the limit
    pass that check (the calls below then stop at a missing x_t instead)."""
    P = [(i + 1) << 40 for i in range(10)]       # fake addresses, 1 TiB apart: nothing overlaps
    one = (ctypes.c_int32 * 1)(0)
    # float32, C = 256: 64 channel vectors per token; 4 views of 4094^2 tokens, one anchor
    B, N, H, W, C = 1, 4, 4094, 4094, 256
    smp = gc.Sampler(kind=gc.GC_FLOW_EULER).c()

    def step(nv):
        return L.gc_transport_step(P[0], P[1], P[2], P[3], P[4], P[5], nv, B, N, H, W, C, one, 1, 4, 0, P[6], None)

    def fused(nv):
        return L.gc_transport_reconstruct(P[0], P[1], P[2], P[3], P[4], P[5], nv, None, B, N, H, W, C, one, 1, 4, 0,
                                          ctypes.byref(smp), 0.5, 0.4, P[6], P[7], None, None)

    assert step(2 ** 25) == -6 and "2^31" in _err(L)          # 2^25 * 64 lanes
    assert step(2 ** 25 - 31) == -6                            # rounds up to 2^31 lanes
    assert fused(2 ** 25 - 31) == -6
    assert fused(2 ** 25 - 32) == -1 and "x_t" in _err(L)      # 2^31 - 2048 lanes: accepted
    # the foreground launch: 8 lanes per record (C = 32 float32), 32 records per block
    B, N, H, W, C = 19, 31, 1019, 3578, 32
    n_tok = B * N * H * W
    assert 2 ** 31 - 256 < n_tok < 2 ** 31

    def geom(nf):
        return L.gc_transport_reconstruct_geom(P[0], P[1], P[2], P[3], P[4], P[5], P[6], nf, None, B, N, H, W, C,
                                               one, 1, 4, 0, ctypes.byref(smp), 0.5, 0.4, P[7], P[8], None, None)

    assert geom(n_tok) == -6 and "n_fg" in _err(L)
    assert geom(2 ** 31 - 256) == -1 and "x_t" in _err(L)


def test_forced_views_and_gaps_host_calls(gc, L):
    """The library's forced-view rule and gap counter (the runner's only
    source for them) on the hand-derived toy cases, against the oracle's own
    rule on random gaps, and their argument checks."""
    assert gc.gc_schedule_forced_views([0, 1, 1], 1, 1) == [1]
    assert gc.gc_schedule_forced_views([1, 0, 2], 3, 1) == [2, 0]
    assert gc.gc_schedule_forced_views([3, 3, 3], 2, 2) == [0, 1]
    assert gc.gc_schedule_forced_views([5, 5, 5], 3, 0) == []
    assert gc.gc_schedule_advance_gaps([1, 0, 2], [2], False) == [2, 1, 0]
    assert gc.gc_schedule_advance_gaps([1, 0, 2], [], True) == [0, 0, 0]
    assert gc.gc_schedule_advance_gaps([2 ** 31 - 1, 0], [1], False) == [2 ** 31 - 1, 0]
    rs = np.random.default_rng(3)
    for _ in range(300):
        N = int(rs.integers(1, 13))
        a = int(rs.integers(1, N + 1))
        gap = [int(x) for x in rs.integers(0, 5, N)]
        mg = int(rs.integers(0, 4))
        assert gc.gc_schedule_forced_views(gap, a, mg) == oracle.forced_views(gap, a, mg)
        views = sorted(set(int(x) for x in rs.integers(0, N, int(rs.integers(0, N + 1)))))
        full = bool(rs.integers(0, 2))
        assert gc.gc_schedule_advance_gaps(gap, views, full) == oracle.advance_gaps(gap, views, full)
    g = (ctypes.c_int32 * 3)(0, 1, 2)
    out = (ctypes.c_int32 * 3)()
    n = ctypes.c_int()
    assert L.gc_schedule_forced_views(None, 3, 1, 1, out, ctypes.byref(n)) == -1
    assert L.gc_schedule_forced_views(g, 3, 4, 1, out, ctypes.byref(n)) == -1
    assert L.gc_schedule_forced_views(g, 65, 1, 1, out, ctypes.byref(n)) == -6
    assert L.gc_schedule_forced_views(g, 3, 1, -1, out, ctypes.byref(n)) == -1
    neg = (ctypes.c_int32 * 3)(0, -1, 2)
    assert L.gc_schedule_forced_views(neg, 3, 1, 1, out, ctypes.byref(n)) == -1
    v = (ctypes.c_int32 * 1)(3)
    assert L.gc_schedule_advance_gaps(g, 3, v, 1, 0) == -1 and "view 3" in _err(L)
    assert L.gc_schedule_advance_gaps(g, 3, None, 1, 0) == -1
    assert L.gc_schedule_advance_gaps(g, 3, v, 4, 0) == -1
    assert list(g) == [0, 1, 2]                 # a rejected call leaves the gaps alone


def test_noalloc_index_validation(gc, L):
    """gc_index_correspondence_noalloc checks its arguments and its scratch
    limit (GC_NOALLOC_SCRATCH_BYTES: 2 * ceil(n / 1024) int32, so at most
    134217728 tokens) on the host, before it touches a device."""
    nv = (ctypes.c_int32 * 1)()

    def call(corr=A0, n=4096, a=4, bits=A1, lst=A2, nvp=A3):
        # n tokens as n views of one token (the order does not matter here)
        return L.gc_index_correspondence_noalloc(corr, n, 1, 1, a, bits, lst, nvp, None)

    assert gc.GC_NOALLOC_SCRATCH_BYTES == 1 << 20
    big = 134217728
    far = [(i + 1) << 40 for i in range(4)]     # 1 TiB apart: nothing overlaps
    assert call(corr=far[0], bits=far[1], lst=far[2], nvp=far[3], n=big + 1) == -6 and "scratch" in _err(L)
    assert int(L.gc_index_workspace_bytes(big)) == 1 << 20
    assert call(nvp=None) == -1
    assert call(a=9) == -1
    assert call(n=-1) == -2
    assert call(corr=A0 + 4) == -4
    assert call(lst=A1 + 64) == -5             # list overlaps the bits
    assert call(n=2 ** 31) == -6


def test_tile_order_definition():
    """The tests' definition of the index lists' order on a hand example: a
    3 x 18 grid is one band of two tiles, 16 columns then 2; row-major inside
    each; a second view follows the first."""
    from conftest import tile_order
    first = [y * 18 + x for y in range(3) for x in range(16)] + [y * 18 + x for y in range(3) for x in (16, 17)]
    assert tile_order(1, 3, 18).tolist() == first
    assert tile_order(2, 3, 18).tolist() == first + [54 + t for t in first]
    # 17 rows: a full band of 16 rows, then a band of one row
    t = tile_order(1, 17, 4).tolist()
    assert t == list(range(64)) + [64, 65, 66, 67]
    assert sorted(tile_order(3, 37, 53).tolist()) == list(range(3 * 37 * 53))


def test_coverage_validation(gc, L):
    """The coverage calls check their arguments on the host and fail before
    any launch: update, selection, scoring and the fused update + selection /
    scoring (whose stats must not overlap the workspace or the result)."""
    B, N, H, W = 1, 4, 8, 8
    ws = int(L.gc_coverage_workspace_bytes())
    assert ws % 256 == 0 and ws >= 8 * (1 << N)

    def ints(*v):
        return (ctypes.c_int32 * max(len(v), 1))(*v)

    A = ints(0, 2)
    # update: pair_bits, B, N, H, W, anchors, a, R, stale, stats
    assert L.gc_coverage_update(None, B, N, H, W, A, 2, 2, A1, A2, None) == -1
    assert L.gc_coverage_update(A0, B, N, H, W, ints(0, 4), 2, 2, A1, A2, None) == -1     # anchor outside [0, N)
    assert L.gc_coverage_update(A0, B, N, H, W, ints(1, 1), 2, 2, A1, A2, None) == -1     # anchor twice
    assert L.gc_coverage_update(A0, B, N, H, W, A, 2, 0, A1, A2, None) == -1              # R < 1
    assert L.gc_coverage_update(A0, B, 65, H, W, A, 2, 2, A1, A2, None) == -6             # N > GC_MAX_VIEWS
    assert L.gc_coverage_update(A0, B, N, H, W, A, 2, 2, A1, A2 + 4, None) == -4          # stats misaligned
    assert L.gc_coverage_update(A0, B, N, H, W, A, 2, 2, A0 + 16, A2, None) == -5         # stale over the pairs
    # selection: pair_bits, stale, B, N, H, W, a, forced, n_forced, anchors_out, workspace, ws_bytes
    sel = lambda a=2, f=ints(), nf=0, out=A2, wsp=A3, wsb=ws: L.gc_coverage_select(A0, A1, B, N, H, W, a, f, nf,
                                                                                     out, wsp, wsb, None)
    assert sel(a=0) == -1
    assert sel(f=ints(3, 3), nf=2) == -1                                                  # forced twice
    assert sel(f=ints(4), nf=1) == -1                                                     # forced outside [0, N)
    assert sel(nf=3) == -1                                                                # more forced than a
    assert sel(wsb=ws - 1) == -6
    assert sel(wsp=A3 + 8) == -4
    assert sel(out=A3 + 16) == -5                                                         # result in the workspace
    assert L.gc_coverage_select(A0, A1, B, 12, H, W, 9, ints(), 0, A2, A3, ws, None) == -6   # a > GC_MAX_ANCHORS
    # scoring: pair_bits, stale, B, N, H, W, sets, M, a, scores, workspace, ws_bytes
    S = ints(0, 1, 2, 3)
    assert L.gc_coverage_score(A0, A1, B, N, H, W, S, 0, 2, A2, A3, ws, None) == -6       # M outside [1, 64]
    assert L.gc_coverage_score(A0, A1, B, N, H, W, ints(0, 5, 2, 3), 2, 2, A2, A3, ws, None) == -1
    assert L.gc_coverage_score(A0, A1, B, N, H, W, S, 2, 2, A2 + 4, A3, ws, None) == -4   # scores misaligned
    assert L.gc_coverage_score(A0, A1, B, N, H, W, S, 2, 2, A3 + 64, A3, ws, None) == -5  # scores in the workspace
    # fused: the update's checks, the selection's / scoring's, and stats apart from both
    us = lambda st=A4, a_next=2, out=A2, wsp=A3: L.gc_coverage_update_select(A0, B, N, H, W, A, 2, 2, A1, st, a_next,
                                                                            ints(), 0, out, wsp, ws, None)
    assert us(a_next=0) == -1
    assert us(st=A4 + 4) == -4
    assert us(st=A3 + 256) == -5                                                          # stats in the workspace
    assert us(st=A2) == -5                                                                # stats over the result
    assert L.gc_coverage_update_select(A0, B, N, H, W, ints(0, 0), 2, 2, A1, A4, 2, ints(), 0, A2, A3, ws,
                                       None) == -1
    sc = lambda st=A4, out=A2: L.gc_coverage_update_score(A0, B, N, H, W, A, 2, 2, A1, st, S, 2, 2, out, A3, ws, None)
    assert sc(st=A3 + 256) == -5
    assert sc(st=A2) == -5                                                                # stats over the scores
    assert L.gc_coverage_update_score(A0, B, N, H, W, A, 2, 0, A1, A4, S, 2, 2, A2, A3, ws, None) == -1   # R < 1
