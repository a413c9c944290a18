"""Benchmark of the per-step cross-view transport on one MI355X.

One timed step is one cached denoising step of the workload: the host
schedule picks the step's anchor set (gc_schedule_anchors) and its
precomputed correspondence, then gc_transport_reconstruct runs Eq. 1 and the
sampler-consistent Euler/DDIM update over every view of every asset.  Inputs
are resident in HBM; each step uses the next of several buffer sets so that
the 256 MB last-level cache cannot serve a step from the previous one.

Reported (one JSON line):
  value      transported view-pixels per second, B * (N - a) * H * W per step
  roofline   the fused kernel's algorithmic bytes per launch (the latents read
             and written, a correspondence word per (target token, anchor) and
             the K weights of every visible pair) over its average launch
             duration (HIP events on the launch stream bracketing the K
             back-to-back launches of the timed region), against 8 TB/s; beside
             it the practical ceiling, a plain nontemporal 16-byte copy kernel
             (ceiling/)
  cpu_baseline  the oracle's transport + reconstruction on one asset, timed
             single-threaded on the host
The once-per-asset rows (area downsample, bbox, correspondence builds), the
unfused pair, the plain copy / read / write kernels and the other workloads
(cache-resident, and from HBM after a flush) are timed too and reported
under "rows".  --cold WORKLOAD runs only that workload's from-HBM steps.
"""
import argparse
import ctypes
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
FUSED_KERNEL = "k_transport<1, 8, 1, true>"   # bf16, 16-byte vectors, fused reconstruction, split launch


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="stress_torusknot_12v_128x16_b8")
    ap.add_argument("--ring", type=int, default=3, help="buffer sets cycled through (defeats the LLC)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-coverage", action="store_true", help="skip the coverage-schedule rows")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (reference kernel for counter scaling)")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--no-small", action="store_true", help="skip the rows of the other workloads")
    ap.add_argument("--cold", metavar="WORKLOAD",
                    help="only the from-HBM steps of one workload's row (each after an L2 / LLC flush); for "
                         "kernel traces and counter passes of that workload's fused kernel")
    return ap.parse_args()


def log(args, *a):
    if not args.quiet:
        print(*a, file=sys.stderr, flush=True)


def load_ceiling():
    """ceiling/libceiling.so: plain copy / read / write kernels with the
    per-step kernels' access shape (built by build())."""
    path = os.path.join(ROOT, "ceiling", "libceiling.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it (python -c 'import __graft_entry__ as g; g.build()')")
    L = ctypes.CDLL(path)
    vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.ceil_copy.argtypes = [vp, vp, i64, ci, vp]
    L.ceil_read.argtypes = [vp, i64, vp, ci, vp]
    L.ceil_write.argtypes = [vp, i64, ctypes.c_uint32, ci, vp]
    for f in (L.ceil_copy, L.ceil_read, L.ceil_write):
        f.restype = ci
    return L


class Flush:
    """Evicts earlier data from L2 and the 256 MB last-level cache: one plain
    read of a 1 GiB buffer, on the given stream (outside any timed region)."""

    def __init__(self, torch, dev):
        self.L = load_ceiling()
        self.n16 = (1 << 30) // 16
        self.buf = torch.ones(1 << 28, dtype=torch.int32, device=dev)
        self.sink = torch.empty(((self.n16 + 255) // 256) * 4, dtype=torch.int32, device=dev)

    def __call__(self, stream_handle):
        rc = self.L.ceil_read(self.buf.data_ptr(), self.n16, self.sink.data_ptr(), 0, stream_handle)
        if rc != 0:
            raise RuntimeError(f"ceil_read failed ({rc})")


def ceiling_rows(torch, dev):
    """GB/s (bytes read + written) of the plain streaming kernels over 1 GiB,
    cached and nontemporal, ten back-to-back launches each: the practical
    ceiling the per-step kernels are compared with."""
    L = load_ceiling()
    n16 = (1 << 30) // 16
    a = torch.ones(1 << 28, dtype=torch.int32, device=dev)
    b = torch.zeros_like(a)
    sink = torch.empty(((n16 + 255) // 256) * 4, dtype=torch.int32, device=dev)
    s = torch.cuda.current_stream().cuda_stream

    def timed(call, n=10):
        for _ in range(2):
            if call() != 0:
                raise RuntimeError("ceiling kernel launch failed")
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            call()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    out = {}
    for nt, tag in ((0, ""), (1, "_nt")):
        out["copy" + tag + "_GBps"] = 2 * (1 << 30) / (timed(lambda: L.ceil_copy(a.data_ptr(), b.data_ptr(), n16, nt, s)) * 1e-3) / 1e9
        out["read" + tag + "_GBps"] = (1 << 30) / (timed(lambda: L.ceil_read(a.data_ptr(), n16, sink.data_ptr(), nt, s)) * 1e-3) / 1e9
        out["write" + tag + "_GBps"] = (1 << 30) / (timed(lambda: L.ceil_write(b.data_ptr(), n16, 7, nt, s)) * 1e-3) / 1e9
    ms = timed(lambda: (b.copy_(a), 0)[1])
    out["torch_copy_GBps"] = 2 * (1 << 30) / (ms * 1e-3) / 1e9
    del a, b, sink
    return out


def kernel_source_hash():
    h = hashlib.sha256()
    # the step kernel's sources and the index builder, whose list order shapes the step's memory traffic
    for f in ("gc_transport.hip", "gc_latent.h", "gc_common.h", "gc_index.hip"):
        h.update(open(os.path.join(ROOT, "paper_2608_13255_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(workload):
    """HBM bytes per launch of the fused kernel from the committed rocprofv3
    counter summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"fused_transport_reconstruct_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and line.split(":")[0].strip() in ("source_hash", "hbm_bytes_per_launch"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_hash") != kernel_source_hash() or "hbm_bytes_per_launch" not in vals:
        return None
    return float(vals["hbm_bytes_per_launch"])


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported (assets shard across GPUs with "
              f"no communication; run one process per GPU)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_13255_amd as gc
    import synth

    if args.cold:
        torch.cuda.set_device(0)
        if args.copy_probe:
            copy_probe(torch, torch.device("cuda:0"))
        row = config_row(gc, synth, args.cold, cold_steps=max(args.steps, 10), warm=False)
        print(json.dumps({"workload": args.cold, "cold_steps": max(args.steps, 10), **row}), flush=True)
        return

    w = synth.CONFIGS[args.config]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    tdtype = torch.float32 if w.dtype == "f32" else torch.bfloat16
    B, N, H, W, C, a, K = w.B, w.N, w.H, w.W, w.C, w.a, w.K
    HW = H * W
    es = 4 if w.dtype == "f32" else 2

    # ---- inputs (seeded, synthetic) --------------------------------------
    t0 = time.time()
    hi = synth.render_position_maps(w)
    cams_np = synth.batch_cameras(w)
    log(args, f"[bench] rendered {hi.shape} in {time.time() - t0:.1f}s")
    hi_d = torch.from_numpy(hi).to(dev)
    # the oracle's baseline takes asset 0's render and computes everything
    # else itself (nothing it reads comes from the HIP path)
    hi0 = None if args.no_cpu_baseline else hi[:1].copy()
    del hi
    cams = gc.camera_tensor(cams_np, dev)

    smp = gc.Sampler(kind=gc.GC_DDIM if w.sampler == "ddim" else gc.GC_FLOW_EULER)
    full = gc.gc_schedule_full_steps(gc.GC_FULL_PERIODIC if w.full_rule == "periodic" else gc.GC_FULL_HEAD_MID_TAIL,
                                     w.S, w.full_E)
    cached_steps = [k for k in range(w.S) if not full[k]]
    anchor_sets = []
    for c in range(N):
        A = tuple(gc.gc_schedule_anchors(N, a, c))
        if A not in anchor_sets:
            anchor_sets.append(A)

    def ev():
        return torch.cuda.Event(enable_timing=True)

    # device warm-up: about 100 ms of plain fills, so that the once-per-asset
    # rows below are not timed while the GPU's clocks ramp up from idle
    spin = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    for i in range(100):
        spin.fill_(float(i))
    torch.cuda.synchronize()
    del spin

    # ---- once per asset: downsample, bbox, correspondence builds ------------
    rows = {}
    for rep in range(3):
        e0, e1, e2, e3 = ev(), ev(), ev(), ev()
        e0.record()
        if w.factor > 1:
            pos = gc.gc_posmap_downsample(hi_d, w.factor)
        else:
            pos = hi_d.clone()
        e1.record()
        bbox = gc.gc_posmap_bbox(pos, w.tol_frac)
        e2.record()
        ops = {}
        stats = {}
        for A in anchor_sets:
            st = torch.empty((B, 4), dtype=torch.int32, device=dev)
            ops[A] = gc.gc_build_correspondence(pos, cams, list(A), K, bbox, stats=st)
            stats[A] = st
        e3.record()
        torch.cuda.synchronize()
    if w.factor > 1:
        # ten back-to-back launches into a preallocated output (the render maps
        # are larger than the last-level cache, so every launch reads HBM)
        ds_out = torch.empty_like(pos)
        torch.cuda.synchronize()
        d0, d1 = ev(), ev()
        d0.record()
        for _ in range(10):
            gc.gc_posmap_downsample(hi_d, w.factor, pos_lat=ds_out)
        d1.record()
        torch.cuda.synchronize()
        assert torch.equal(ds_out.view(torch.int32), pos.view(torch.int32))
        rows["downsample_ms"] = d0.elapsed_time(d1) / 10
        rows["downsample_GBps"] = (hi_d.numel() + pos.numel()) * 4 / (rows["downsample_ms"] * 1e-3) / 1e9
        del ds_out
    else:
        rows["downsample_ms"] = e0.elapsed_time(e1)
        rows["downsample_GBps"] = None
    rows["bbox_ms"] = e1.elapsed_time(e2)
    # builds: ten back-to-back launches per anchor set into the buffers above
    torch.cuda.synchronize()
    b0, b1 = ev(), ev()
    b0.record()
    for _ in range(10):
        for A in anchor_sets:
            gc.gc_build_correspondence(pos, cams, list(A), K, bbox, corr=ops[A][0], weights=ops[A][1], stats=stats[A])
    b1.record()
    torch.cuda.synchronize()
    rows["build_ms_per_anchor_set"] = b0.elapsed_time(b1) / (10 * len(anchor_sets))   # with the counters
    b0.record()
    for _ in range(10):
        for A in anchor_sets:
            gc.gc_build_correspondence(pos, cams, list(A), K, bbox, corr=ops[A][0], weights=ops[A][1])
    b1.record()
    torch.cuda.synchronize()
    rows["build_no_counters_ms_per_anchor_set"] = b0.elapsed_time(b1) / (10 * len(anchor_sets))
    # (target token, anchor) pairs the builder decides per second
    n_pairs = B * (N - a) * HW * a
    rows["build_pairs_per_s"] = n_pairs / (rows["build_no_counters_ms_per_anchor_set"] * 1e-3)
    rows["build_with_counters_pairs_per_s"] = n_pairs / (rows["build_ms_per_anchor_set"] * 1e-3)
    rows["anchor_sets"] = len(anchor_sets)
    index = {}
    e4, e5 = ev(), ev()
    e4.record()
    for A in anchor_sets:
        index[A] = gc.gc_index_correspondence(ops[A][0])
    e5.record()
    torch.cuda.synchronize()
    # the binding allocates the index and reads the visible count back (one
    # synchronisation); the device part alone: ten back-to-back launches per
    # set into preallocated buffers
    rows["index_with_readback_ms_per_anchor_set"] = e4.elapsed_time(e5) / len(anchor_sets)
    corr0 = ops[anchor_sets[0]][0]
    n_tok = corr0.numel() // corr0.shape[-1]
    ws = torch.empty(int(gc.lib().gc_index_workspace_bytes(n_tok)), dtype=torch.uint8, device=dev)
    bits_i = torch.empty((n_tok + 31) // 32, dtype=torch.int32, device=dev)
    lst_i = torch.empty(n_tok, dtype=torch.int32, device=dev)
    nv_i = torch.empty(1, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    e4.record()
    for _ in range(10):
        for A in anchor_sets:
            rc = gc.lib().gc_index_correspondence(ops[A][0].data_ptr(), corr0.shape[0] * corr0.shape[1],
                                                  corr0.shape[2], corr0.shape[3], corr0.shape[-1], bits_i.data_ptr(),
                                                  lst_i.data_ptr(), nv_i.data_ptr(), ws.data_ptr(), ws.numel(),
                                                  torch.cuda.current_stream().cuda_stream)
            assert rc == 0, gc.lib().gc_last_error()
    e5.record()
    torch.cuda.synchronize()
    rows["index_device_ms_per_anchor_set"] = e4.elapsed_time(e5) / (10 * len(anchor_sets))
    del ws, bits_i, lst_i, nv_i
    vis_pairs = {A: int(stats[A][:, 0].sum().item()) for A in anchor_sets}
    cover = {A: float(stats[A][:, 1].sum().item()) / max(1, float(stats[A][:, 2].sum().item())) for A in anchor_sets}
    del hi_d
    torch.cuda.empty_cache()

    # ---- latent buffers: a ring of sets ------------------------------------
    t0 = time.time()
    x0_prev_np = synth.x0_state(w, pos.cpu().numpy(), cached_steps[0] - 1)
    eps_np = synth.eps_noise(w, 0)
    log(args, f"[bench] synthetic latents in {time.time() - t0:.1f}s")

    def dev_lat(x):
        return torch.from_numpy(x).to(dev).to(tdtype)

    base_prev = dev_lat(x0_prev_np)
    base_eps = dev_lat(eps_np)
    ring = []
    for r in range(args.ring):
        x0_prev = base_prev.clone()
        x_t = (base_prev.float() * 0.5 + base_eps.float() * 0.5).to(tdtype)
        x0_new = (base_prev[:, :a].float() + 0.01 * (r + 1)).to(tdtype).contiguous()
        ring.append(dict(x0_prev=x0_prev, x0_new=x0_new, x_t=x_t, x0_out=torch.empty_like(x0_prev),
                         x_next=torch.empty_like(x0_prev)))
    del base_prev, base_eps
    torch.cuda.synchronize()

    latent_view = HW * C * es
    V = B * (N - a) * HW

    n_tok = B * (N - a) * HW

    def algo_bytes(A):
        # what one cached step must move (the definition of the per-step unit): read
        # x0_prev, x0_anchor_new, x_t, write x0_out, x_next; a correspondence word per
        # (target token, anchor); the K weights of every visible (token, anchor) pair
        return B * (4 * N + a) * latent_view + 4 * n_tok * a + 4 * K * vis_pairs[A]

    def index_bytes(A):
        # what the split launch reads of the operator instead of every word: a bit per
        # target token, the list of visible tokens and their words
        nv = index[A].n_vis
        return (B * (4 * N + a) * latent_view + 4 * ((n_tok + 31) // 32) + 4 * nv + 4 * a * nv
                + 4 * K * vis_pairs[A])

    # every (buffer set, anchor set) pair gets its call marshalled once, so the
    # host issues one ctypes call per step and stays ahead of the GPU
    plans = {}
    for r, buf in enumerate(ring):
        for A in anchor_sets:
            corr, wts = ops[A]
            plans[(r, A)] = gc.bind_transport_reconstruct(buf["x0_prev"], buf["x0_new"], corr, wts, buf["x_t"],
                                                          list(A), smp, buf["x0_out"], buf["x_next"],
                                                          index=index[A])

    def step(i):
        A = tuple(gc.gc_schedule_anchors(N, a, i))        # host schedule: cached step i
        t, tn = gc.gc_sampler_step_times(smp, w.S, cached_steps[i % len(cached_steps)])
        plans[(i % len(ring), A)](t, tn)
        return A

    # device warm-up before the W warmup steps: about 90 ms of the same step,
    # so that the GPU's clocks have left their idle state (the first tens of
    # milliseconds after an idle host phase run measurably slower)
    for i in range(2000):
        step(i)
    torch.cuda.synchronize()
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # ---- timed region -------------------------------------------------------
    # Only the step launches run between the two events: the average launch
    # duration is the region's time over K (the kernel plus its dispatch gap
    # when launches run back to back).
    used = []
    start, end = ev(), ev()
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        used.append(step(args.warmup + i))
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps
    avg_kernel_ms = ms_per_step
    bytes_per_launch = float(np.mean([algo_bytes(A) for A in used]))
    achieved = bytes_per_launch / (avg_kernel_ms * 1e-3) / 1e9
    rows["index_bytes_per_launch"] = float(np.mean([index_bytes(A) for A in used]))
    rows["index_bytes_GBps"] = rows["index_bytes_per_launch"] / (avg_kernel_ms * 1e-3) / 1e9

    # ---- per-step distribution (outside the timed region) ---------------------
    # each step between its own pair of events; the events' own cost widens
    # the gaps a little, so the median sits slightly above the timed mean
    n_dist = min(100, max(10, args.steps))
    evs = [ev() for _ in range(n_dist + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    for i in range(n_dist):
        step(args.warmup + args.steps + i)
        evs[i + 1].record()
    torch.cuda.synchronize()
    per_step_us = np.array([evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(n_dist)])
    rows["step_us_p10_p50_p90"] = [round(float(np.percentile(per_step_us, q)), 2) for q in (10, 50, 90)]
    # the same steps on one buffer set (262 MB, about the size of the last-level
    # cache): what the LLC can serve of a step that re-reads the last one's
    # buffers, against the ring's every-step-from-HBM figure above
    torch.cuda.synchronize()
    r0, r1 = ev(), ev()
    r0.record()
    for i in range(args.steps):
        A = tuple(gc.gc_schedule_anchors(N, a, i))
        plans[(0, A)](*gc.gc_sampler_step_times(smp, w.S, cached_steps[i % len(cached_steps)]))
    r1.record()
    torch.cuda.synchronize()
    rows["step_us_one_buffer_set"] = r0.elapsed_time(r1) / args.steps * 1e3

    # ---- unfused pair and full step, for the record -------------------------
    def timed(fn, n=40, batches=7, warm=200):
        # the same call back to back first (about 10 ms of device work), so
        # that the clocks have left the host-side setup's idle state; then the
        # median over batches of n back-to-back calls, each batch between its
        # own pair of events
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        per = []
        for _ in range(batches):
            s, e = ev(), ev()
            s.record()
            for _ in range(n):
                fn()
            e.record()
            torch.cuda.synchronize()
            per.append(s.elapsed_time(e) / n)
        return float(np.median(per))

    A0 = list(anchor_sets[0])
    corr0, wts0 = ops[anchor_sets[0]]
    buf = ring[0]
    kc = cached_steps[0]
    tt, ttn = gc.gc_sampler_step_times(smp, w.S, kc)
    rows["transport_only_ms"] = timed(lambda: gc.gc_transport_step(buf["x0_prev"], buf["x0_new"], corr0, wts0, A0,
                                                                   x0_out=buf["x0_out"], index=index[anchor_sets[0]]))
    rows["reconstruct_only_ms"] = timed(lambda: gc.gc_sampler_reconstruct(buf["x_t"], buf["x0_out"], smp, tt, ttn,
                                                                          x_next=buf["x_next"]))
    rows["unfused_pair_ms"] = rows["transport_only_ms"] + rows["reconstruct_only_ms"]

    # multistep variant: UniPC-2 with the corrector (DDIM noise schedule) fused with
    # Eq. 1; it also reads x_prev and m_{k-2} and writes x_c (no x_t read)
    ust = gc.gc_unipc_coeffs(gc.Sampler(kind=gc.GC_DDIM), w.S, kc, 2, True)
    uplans = []
    for b in ring[:2]:
        uplans.append(gc.bind_transport_unipc(b["x0_prev"], b["x0_new"], corr0, wts0, A0, b["x0_out"],
                                              torch.empty_like(b["x0_prev"]), b["x_next"], x_prev=b["x_t"].clone(),
                                              m_km2=b["x0_prev"].clone(), index=index[anchor_sets[0]]))
    uc = iter(range(1 << 30))
    rows["unipc_fused_ms"] = timed(lambda: uplans[next(uc) % len(uplans)](ust))
    nv0 = index[anchor_sets[0]].n_vis
    ubytes = (B * (6 * N + a) * latent_view + 4 * ((n_tok + 31) // 32) + 4 * nv0 + 4 * a * nv0
              + 4 * K * vis_pairs[anchor_sets[0]])
    rows["unipc_fused_GBps"] = ubytes / (rows["unipc_fused_ms"] * 1e-3) / 1e9
    del uplans

    # the same cached step with G_{A->v} computed on the fly (no stored operator);
    # algorithmic bytes: the latents as above, 12 B of position per target token,
    # the anchors' position maps once
    L = gc.lib()
    smp_c = smp.c()
    arr0 = (ctypes.c_int32 * a)(*A0)
    # the foreground index of the position maps (once per asset batch)
    torch.cuda.synchronize()
    f0, f1 = ev(), ev()
    f0.record()
    fgi = gc.gc_index_foreground(pos)
    f1.record()
    torch.cuda.synchronize()
    rows["foreground_index_with_readback_ms"] = f0.elapsed_time(f1)
    rows["foreground_tokens"] = fgi.n_fg

    def geom_args(fg):
        out = []
        for b in ring[:2]:
            out.append((b["x0_prev"].data_ptr(), b["x0_new"].data_ptr(), pos.data_ptr(), cams.data_ptr(),
                        bbox.data_ptr(), fg.fg_bits.data_ptr() if fg else None, fg.fg_recs.data_ptr() if fg else None,
                        fg.n_fg if fg else 0, b["x_t"].data_ptr(), B, N, H, W, C, arr0, a, K,
                        gc.dtype_code(b["x0_prev"]), ctypes.byref(smp_c), tt, ttn, b["x0_out"].data_ptr(),
                        b["x_next"].data_ptr(), None, torch.cuda.current_stream().cuda_stream))
        return out

    gi = iter(range(1 << 30))

    def geom_call(gargs):
        rc = L.gc_transport_reconstruct_geom(*gargs[next(gi) % len(gargs)])
        if rc != 0:
            raise RuntimeError(L.gc_last_error().decode())

    # the blocked launch, then the foreground launch
    gargs = geom_args(None)
    rows["geom_fused_ms"] = timed(lambda: geom_call(gargs))
    gbytes = B * (4 * N + a) * latent_view + 12 * n_tok + 12 * B * a * HW
    rows["geom_fused_GBps"] = gbytes / (rows["geom_fused_ms"] * 1e-3) / 1e9
    gargs_fg = geom_args(fgi)
    rows["geom_fg_fused_ms"] = timed(lambda: geom_call(gargs_fg))
    # a bit per target token and a 16-byte record per foreground target token
    # in place of every target token's 12-byte position
    targets0 = [v for v in range(N) if v not in A0]
    fg_targets = int(torch.isfinite(pos[:, targets0]).all(-1).sum().item())
    gbytes_fg = B * (4 * N + a) * latent_view + n_tok // 8 + 16 * fg_targets + 12 * B * a * HW
    rows["geom_fg_fused_GBps"] = gbytes_fg / (rows["geom_fg_fused_ms"] * 1e-3) / 1e9
    # the on-the-fly UniPC-2 step (foreground launch), the multistep row's inputs
    ubufs = [(b, b["x_t"].clone(), b["x0_prev"].clone(), torch.empty_like(b["x0_prev"])) for b in ring[:2]]
    ui = iter(range(1 << 30))

    def unipc_geom_call():
        b, xp, m2, xc = ubufs[next(ui) % len(ubufs)]
        gc.gc_transport_unipc_geom(b["x0_prev"], b["x0_new"], pos, cams, bbox, A0, K, ust, x_prev=xp, m_km2=m2,
                                   x0_out=b["x0_out"], x_c=xc, x_next=b["x_next"], fg_index=fgi)

    rows["unipc_geom_fg_fused_ms"] = timed(unipc_geom_call)
    ugbytes = B * (6 * N + a) * latent_view + n_tok // 8 + 16 * fg_targets + 12 * B * a * HW
    rows["unipc_geom_fg_fused_GBps"] = ugbytes / (rows["unipc_geom_fg_fused_ms"] * 1e-3) / 1e9
    del ubufs
    # K = 1 (the paper's ablation finds one tap as good as four): the same step
    # with a one-tap operator
    corr1, wts1 = gc.gc_build_correspondence(pos, cams, A0, 1, bbox)
    idx1 = gc.gc_index_correspondence(corr1)
    k1 = [gc.bind_transport_reconstruct(b["x0_prev"], b["x0_new"], corr1, wts1, b["x_t"], A0, smp, b["x0_out"],
                                        b["x_next"], index=idx1) for b in ring[:2]]
    ki = iter(range(1 << 30))
    rows["k1_fused_ms"] = timed(lambda: k1[next(ki) % len(k1)](tt, ttn))
    rows["k1_view_pixels_per_s"] = B * (N - a) * HW / (rows["k1_fused_ms"] * 1e-3)
    del k1, corr1, wts1, idx1
    rows["coverage_per_anchor_set"] = [round(cover[A], 4) for A in anchor_sets]
    rows["visible_pairs_per_anchor_set"] = [vis_pairs[A] for A in anchor_sets]
    rows["visible_tokens_per_anchor_set"] = [index[A].n_vis for A in anchor_sets]
    # target tokens by the number of anchors that see them (0 .. a), per anchor set
    rows["n_vis_histogram_per_anchor_set"] = [
        torch.bincount((ops[A][0] != 0).sum(-1).flatten(), minlength=a + 1).tolist() for A in anchor_sets]

    if args.copy_probe:
        copy_probe(torch, dev)
    # the practical ceiling: plain streaming kernels with the step's access shape
    rows["ceiling"] = ceiling_rows(torch, dev)

    # ---- the other workloads: eager vs HIP-graph replay ------------------------
    if not args.no_small:
        for name in synth.CONFIGS:
            if name != w.name:
                rows[f"config_{name}"] = config_row(gc, synth, name,
                                                    oracle_seconds=None if args.no_cpu_baseline else 1.0)

    # ---- coverage-driven schedule: staleness under each anchor policy --------
    if not args.no_coverage:
        rows["coverage"] = coverage_rows(gc, w, pos, cams, bbox, full)

    # ---- CPU baseline: the oracle on one asset ------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, hi0, cams_np, cached_steps[0] - 1, args.cpu_seconds)

    traffic = read_traffic(w.name)
    out = {
        "metric": "transported view-pixels/s per denoising step; achieved HBM GB/s vs peak",
        "value": V / (ms_per_step * 1e-3),
        "unit": "view-pixels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded torus-knot renders, synthetic x0 fields)",
        "config": {"workload": w.name, "assets": B, "views": N, "latent": [H, W, C], "anchors": a, "K": K,
                   "sampler": w.sampler, "steps_S": w.S, "render": w.render, "ring_buffers": args.ring,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS,
                     "traffic": traffic, "kernel": FUSED_KERNEL, "algorithmic_bytes_per_launch": bytes_per_launch,
                     "avg_launch_us": avg_kernel_ms * 1e3,
                     "copy_ceiling_GBps": rows["ceiling"]["copy_nt_GBps"],
                     "frac_of_copy_ceiling": achieved / rows["ceiling"]["copy_nt_GBps"]},
        "cpu_baseline": cpu,
        "rows": rows,
    }
    print(json.dumps(out), flush=True)


def copy_probe(torch, dev):
    """A plain 1 GiB device-to-device copy (torch's), the reference dispatch
    whose FETCH_SIZE / WRITE_SIZE readings scale the counters of the other
    kernels in the same rocprofv3 run."""
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(11):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def coverage_rows(gc, w, pos, cams, bbox, full, R=2):
    """One whole trajectory of the schedule alone (no latents) per anchor
    policy: per-step staleness of the foreground tokens after the step
    (mean, fraction stale for >= R steps, max) and the policy's cost per
    cached step two ways: the wall time of the trajectory's step (the
    staleness update fused with the next step's selection or scoring, and
    the host read-backs of the anchors and counters), and the device time of
    the same launches captured in a HIP graph and replayed back to back (what
    they cost the GPU when the host is not in the way)."""
    import numpy as np
    import torch
    N, a = w.N, w.a
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    pairs = gc.gc_coverage_pairs(pos, cams, bbox)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    # device time: the kernel alone, into the same buffer
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    gc.gc_coverage_pairs(pos, cams, bbox, out=pairs)
    e1.record()
    torch.cuda.synchronize()
    n_dec = N * w.B * N * w.H * w.W
    out = {"pairs_ms": e0.elapsed_time(e1), "pairs_first_call_wall_ms": wall_ms,
           "pair_decisions_per_s": n_dec / (e0.elapsed_time(e1) * 1e-3), "R": R}
    rot_sets = []
    for c in range(N):
        A = gc.gc_schedule_anchors(N, a, c)
        if A not in rot_sets:
            rot_sets.append(A)
    ws = torch.empty(gc.gc_coverage_workspace_bytes(), dtype=torch.uint8, device=pos.device)
    max_gap = -(-N // a)
    for policy in ("rotate", "rotation_coverage", "coverage"):
        stale = gc.gc_coverage_init(pos)
        gap, c, rec, cost, nxt = [0] * N, 0, [], [], None
        for k in range(w.S):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            if full[k] or k == 0:
                A = list(range(N))
            elif policy == "rotate":
                A = gc.gc_schedule_anchors(N, a, c)
            elif policy == "rotation_coverage":
                sc = nxt.cpu().tolist()   # scored by the last step's fused update
                A = rot_sets[sc.index(max(sc))]
            else:
                A = nxt.cpu().tolist()    # chosen by the last step's fused update
            gap = gc.gc_schedule_advance_gaps(gap, A, bool(full[k] or k == 0))
            # the update, fused with the next cached step's choice (unused if that step is full)
            if policy == "rotation_coverage":
                st, nxt = gc.gc_coverage_update_score(pairs, stale, A, R, rot_sets, workspace=ws)
            elif policy == "coverage":
                st, nxt = gc.gc_coverage_update_select(pairs, stale, A, R, a,
                                                       forced=gc.gc_schedule_forced_views(gap, a, max_gap),
                                                       workspace=ws)
            else:
                st = gc.gc_coverage_update(pairs, stale, A, R)
            st = st.cpu().numpy().astype(np.int64)
            if not (full[k] or k == 0):
                cost.append(time.perf_counter() - t0)
                c += 1
            fg = st[..., 0].sum()
            rec.append((st[..., 2].sum() / fg, st[..., 1].sum() / fg, st[..., 3].max()))
        r = np.array(rec, np.float64)
        # the policy's launches for one cached step, captured and replayed back to back
        sgr = torch.cuda.Stream()
        stats_buf = torch.empty((w.B, N, 4), dtype=torch.int32, device=pos.device)
        sel_buf = torch.empty(a, dtype=torch.int32, device=pos.device)
        score_buf = torch.empty(len(rot_sets), dtype=torch.int64, device=pos.device)
        A0 = rot_sets[0]
        torch.cuda.synchronize()

        def policy_step():
            if policy == "rotation_coverage":
                gc.gc_coverage_update_score(pairs, stale, A0, R, rot_sets, stats=stats_buf, out=score_buf,
                                            workspace=ws, stream=sgr)
            elif policy == "coverage":
                gc.gc_coverage_update_select(pairs, stale, A0, R, a, stats=stats_buf, out=sel_buf, workspace=ws,
                                             stream=sgr)
            else:
                gc.gc_coverage_update(pairs, stale, A0, R, stats=stats_buf, stream=sgr)

        reps = 20
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=sgr):
            for _ in range(reps):
                policy_step()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(sgr):    # replay() launches on the current stream: the events' stream
            graph.replay()
            torch.cuda.synchronize()
            g0.record(sgr)
            for _ in range(5):
                graph.replay()
            g1.record(sgr)
        torch.cuda.synchronize()
        out[policy] = {"mean_staleness": round(float(r[:, 0].mean()), 5),
                       "frac_stale_ge_R": round(float(r[:, 1].mean()), 5), "max_staleness": int(r[:, 2].max()),
                       "ms_per_cached_step": round(float(np.median(cost)) * 1e3, 4),
                       "device_ms_per_cached_step": round(g0.elapsed_time(g1) / (5 * reps), 4)}
        del graph
    return out


GRAPH_STEPS = 24   # cached steps captured per graph (rounded up to whole rotations)


def config_row(gc, synth, name, steps=300, oracle_seconds=None, cold_steps=30, warm=True):
    """One cached step of another workload, three ways: launched eagerly and
    replayed from a HIP graph holding a run of consecutive steps (one per
    anchor set of the rotation, repeated) -- these working sets fit in the
    256 MB last-level cache and are re-read every step, so those GB/s are
    cache-resident figures and the smaller workloads are launch-bound -- and
    from HBM: each of cold_steps steps between its own pair of events after a
    1 GiB read that evicts the step's data from L2 and the LLC (the events
    add their own cost to these short steps).  Algorithmic bytes per step are
    the latents, a correspondence word per (target token, anchor) and the
    weights of the visible pairs.  With oracle_seconds, the oracle's cached
    step on the same workload is timed beside it (one host thread, from the
    seeded render on its own).  warm=False runs the HBM steps only."""
    import numpy as np
    import torch
    w = synth.CONFIGS[name]
    dev = torch.device("cuda:0")
    hi_np = synth.render_position_maps(w)
    hi = torch.from_numpy(hi_np).to(dev)
    pos = gc.gc_posmap_downsample(hi, w.factor) if w.factor > 1 else hi
    cams = gc.camera_tensor(synth.batch_cameras(w), dev)
    bbox = gc.gc_posmap_bbox(pos, w.tol_frac)
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    if w.fixed_anchors:
        sets = [list(w.fixed_anchors)]
    else:
        sets = []
        for c in range(w.N):
            A = gc.gc_schedule_anchors(w.N, w.a, c)
            if A not in sets:
                sets.append(A)
    smp = gc.Sampler(kind=gc.GC_DDIM if w.sampler == "ddim" else gc.GC_FLOW_EULER)
    t, tn = w.ddim_single if w.ddim_single else gc.gc_sampler_step_times(smp, w.S, 2)
    g = torch.Generator(device=dev).manual_seed(0)
    shape = (w.B, w.N, w.H, w.W, w.C)
    x0 = torch.randn(shape, generator=g, device=dev).to(tdt)
    xt = torch.randn(shape, generator=g, device=dev).to(tdt)
    s = torch.cuda.Stream()
    calls = []
    es = 4 if w.dtype == "f32" else 2
    n_tok = w.B * (w.N - len(sets[0])) * w.H * w.W
    step_bytes = []
    for A in sets:
        st = torch.zeros((w.B, 4), dtype=torch.int32, device=dev)
        corr, wts = gc.gc_build_correspondence(pos, cams, A, w.K, bbox, stats=st)
        idx = gc.gc_index_correspondence(corr)
        pairs = int(st[:, 0].sum().item())
        step_bytes.append(w.B * (4 * w.N + len(A)) * w.H * w.W * w.C * es + 4 * n_tok * len(A) + 4 * w.K * pairs)
        new = torch.randn((w.B, len(A), w.H, w.W, w.C), generator=g, device=dev).to(tdt)
        calls.append(gc.bind_transport_reconstruct(x0, new, corr, wts, xt, A, smp, torch.empty_like(x0),
                                                   torch.empty_like(x0), index=idx, stream=s))
    torch.cuda.synchronize()
    V = n_tok
    mean_bytes = sum(step_bytes) / len(step_bytes)
    row = {"view_pixels_per_step": V, "algorithmic_bytes_per_step": mean_bytes}
    reps = max(1, steps // len(calls))

    def timed(fn, n):
        # with s current: the bound calls launch on s, and graph.replay() on the
        # current stream, so the events on s bracket the launches either way
        with torch.cuda.stream(s):
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(n):
                fn()
            e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    def eager():
        for c in calls:
            c(t, tn)
    if warm:
        eager_ms = timed(eager, reps) / len(calls)
        # A captured denoising loop holds many consecutive steps; a graph of one
        # step per replay would time the replay call's own host overhead instead.
        rounds = -(-GRAPH_STEPS // len(calls))
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            for _ in range(rounds):
                eager()
        graph_ms = timed(graph.replay, max(1, reps // rounds)) / (len(calls) * rounds)
        best = min(eager_ms, graph_ms)
        row.update({"eager_us_per_step": eager_ms * 1e3, "graph_us_per_step": graph_ms * 1e3,
                    "view_pixels_per_s": V / (best * 1e-3),
                    "cache_resident_algorithmic_GBps": mean_bytes / (best * 1e-3) / 1e9})
    # from HBM: each step after a flush of L2 and the LLC, between its own events
    flush = Flush(torch, dev)
    calls[0](t, tn)
    torch.cuda.synchronize()
    cold = []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for i in range(cold_steps):
        flush(s.cuda_stream)
        e0.record(s)
        calls[i % len(calls)](t, tn)
        e1.record(s)
        torch.cuda.synchronize()
        cold.append(e0.elapsed_time(e1))
    p50 = float(np.median(cold))
    row.update({"hbm_us_per_step_p10_p50_p90": [round(float(np.percentile(cold, q)) * 1e3, 2) for q in (10, 50, 90)],
                "hbm_view_pixels_per_s": V / (p50 * 1e-3),
                "hbm_algorithmic_GBps": mean_bytes / (p50 * 1e-3) / 1e9,
                "hbm_frac_of_peak": mean_bytes / (p50 * 1e-3) / 1e9 / PEAK_HBM_GBS})
    del flush
    if oracle_seconds:
        vps = oracle_step_rate(w, hi_np, oracle_seconds)
        row["oracle_view_pixels_per_s"] = vps
        row["gpu_over_oracle"] = row.get("view_pixels_per_s", row["hbm_view_pixels_per_s"]) / vps
    return row


def oracle_step_rate(w, hi_np, seconds):
    """The oracle's cached step (transport + reconstruction) over all assets
    of a workload, single-threaded, repeated for about `seconds` seconds:
    transported view-pixels/s.  Every input is computed from the seeded
    render by the oracle and the generators."""
    import numpy as np

    import oracle
    import synth
    A = list(w.fixed_anchors) if w.fixed_anchors else oracle.anchors(w.N, w.a, 0)
    t, tn = w.ddim_single if w.ddim_single else oracle.step_times(w.sampler, w.S, 2)
    pos = oracle.downsample(hi_np, w.factor) if w.factor > 1 else hi_np
    cams = synth.batch_cameras(w)
    corr, wts, _ = oracle.build(pos, cams, list(A), w.K, oracle.bbox(pos, w.tol_frac))
    rs = np.random.default_rng(7)
    prev = synth.storage(rs.standard_normal((w.B, w.N, w.H, w.W, w.C)).astype(np.float32), w.dtype)
    new = synth.storage(rs.standard_normal((w.B, len(A), w.H, w.W, w.C)).astype(np.float32), w.dtype)
    xt = synth.storage(rs.standard_normal((w.B, w.N, w.H, w.W, w.C)).astype(np.float32), w.dtype)
    reps = 0
    with one_core():
        t0 = time.perf_counter()
        while True:
            _, st = oracle.transport(prev, new, corr, wts, list(A), w.dtype)
            oracle.reconstruct(xt, st, w.dtype, w.sampler, t, tn)
            reps += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                break
    return reps * w.B * (w.N - len(A)) * w.H * w.W / el


class one_core:
    """Pins the calling thread to one host core while the oracle is timed
    (the oracle is single-threaded); restores the previous affinity."""

    def __enter__(self):
        self.saved = None
        if hasattr(os, "sched_getaffinity"):
            self.saved = os.sched_getaffinity(0)
            os.sched_setaffinity(0, {min(self.saved)})
        return self

    def __exit__(self, *exc):
        if self.saved is not None:
            os.sched_setaffinity(0, self.saved)
        return False


def cpu_baseline(w, hi0, cams_np, step, seconds):
    """The oracle's cached step (transport + reconstruction) on one asset,
    single-threaded, repeated for about `seconds` seconds.  hi0: asset 0's
    render-resolution position maps; the oracle downsamples them itself."""
    import numpy as np

    import oracle
    import synth

    pos1 = oracle.downsample(hi0, w.factor) if w.factor > 1 else hi0
    x0_prev1 = synth.x0_state(w, pos1, step)
    cams1 = {k: v[:1] for k, v in cams_np.items()}
    A = oracle.anchors(w.N, w.a, 0)
    bb = oracle.bbox(pos1, w.tol_frac)
    corr, wts, _ = oracle.build(pos1, cams1, A, w.K, bb)
    prev = synth.storage(x0_prev1, w.dtype)
    new = synth.storage(x0_prev1[:, A] + np.float32(0.01), w.dtype)
    xt = synth.storage(0.5 * x0_prev1, w.dtype)
    t, tn = oracle.step_times(w.sampler, w.S, 2)
    reps = 0
    with one_core():
        t0 = time.perf_counter()
        while True:
            _, st = oracle.transport(prev, new, corr, wts, A, w.dtype)
            oracle.reconstruct(xt, st, w.dtype, w.sampler, t, tn)
            reps += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                break
    vp = reps * (w.N - w.a) * w.H * w.W
    model = "unknown CPU"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    visible = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"value": vp / el, "unit": "view-pixels/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} cached steps of 1 of {w.B} assets ({w.N} views, {w.H}x{w.W}x{w.C} {w.dtype}, "
                      f"a={w.a}, K={w.K}), transport + reconstruction, {el:.1f}s on one host thread pinned to one core",
            "host": f"{model}; {visible} CPUs visible to the process"}


if __name__ == "__main__":
    main()
