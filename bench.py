#!/usr/bin/env python3
"""Throughput of the co-batched multi-LoRA layer (forward + LoRA backward) on one MI355X.

One step = one pass of the whole path over one synthetic batch: pack the segment
table (dsv_segments_build, host + one copy to the device, on a side stream so that it
overlaps the previous step's kernels, double-buffered), then for every
projection of the workload the co-batched forward (shrink, gathered low-rank
terms, base GEMM with the low-rank prologue, training-row h saved) and the LoRA
backward of the training rows (g, dB, dA, dX).  Inputs are resident in HBM
before the timed region starts.

Default workload: the Llama-3-8B layer set (q, k, v, o 4096x4096/1024, gate/up
4096x14336, down 14336x4096) in bf16, 8 prefill segments of 512 tokens on
adapters drawn from 32 rank-16 adapters plus 2 fine-tuning sequences of 1024
tokens on adapter 0 (T = 6144, T_t = 2048).

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2607_28848_amd import workloads as wl  # noqa: E402

METRIC = "co-batched multi-LoRA fwd+bwd TFLOP/s and % of bf16 MFMA peak, 1 GPU"
PEAK_BF16_TFLOPS = 2516.6   # 256 CUs x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU
WORKLOADS = {
    "llama8b": wl.llama8b_mixed,
    "decode": wl.decode_heavy,
    "llama70b": wl.llama70b,
    "sweep0": lambda: wl.load_sweep(0.0),
    "sweep25": lambda: wl.load_sweep(0.25),
    "sweep50": lambda: wl.load_sweep(0.5),
    "sweep75": lambda: wl.load_sweep(0.75),
    "sweep100": lambda: wl.load_sweep(1.0),
}


LAUNCH_NOTES = {
    "set": ("one grouped call per direction over all projections: their synthetic inputs are independent, "
            "so this is the same work, but in a model o waits for attention and down for the MLP product; "
            "an upper bound of a real layer's launches (extras.launch_modes_ms_per_step.layer is the "
            "realisable grouping)"),
    "layer": ("grouped calls over the projections a transformer layer can run together: q/k/v, o, "
              "gate/up, down"),
    "single": "one call per projection",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algo_flops(w, proj):
    """(fwd, bwd) algorithmic FLOPs of one projection, true ranks only:
    fwd 2 T K N + sum_seg 2 len r_a (K + N); bwd 2 T_t K N + sum_train 4 len r_a (K + N)."""
    K, N = proj.K, proj.N
    fwd = 2.0 * w.n_tokens * K * N
    bwd = 2.0 * w.train_tokens * K * N
    for (_, l, a, t) in w.segments:
        r = int(w.ranks[a])
        fwd += 2.0 * l * r * (K + N)
        if t:
            bwd += 4.0 * l * r * (K + N)
    return fwd, bwd


def gemm_fwd_flops(w, proj, gathered_rows):
    """Algorithmic FLOPs of the forward GEMM launch: the base product plus the
    low-rank expand of the rows whose term rides the tile (not the gathered ones)."""
    row_rank = np.zeros(w.n_tokens, np.int64)
    for (s, l, a, _) in w.segments:
        row_rank[s:s + l] = int(w.ranks[a])
    expand = 2.0 * proj.N * float(row_rank.sum() - row_rank[gathered_rows].sum())
    return 2.0 * w.n_tokens * proj.K * proj.N + expand


def gemm_bwd_flops(w, proj):
    """dX GEMM: 2 T_t N K + 2 sum_train len r_a K."""
    f = 2.0 * w.train_tokens * proj.K * proj.N
    for (_, l, a, t) in w.segments:
        if t:
            f += 2.0 * l * int(w.ranks[a]) * proj.K
    return f


def measured_traffic():
    """HBM bytes per forward-GEMM launch from the committed counter summary, if it was
    taken with the kernel source as it is now (else None)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_fwd_gemm_llama8b_mixed.json")
    try:
        doc = json.load(open(path))
        src = open(os.path.join(ROOT, doc["kernel_source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != doc.get("kernel_source_sha256"):
        return None
    return float(doc["traffic_bytes_per_launch"])


def strided_rows(t, code):
    """t with its rows at the stride dsv_row_stride recommends: t itself when that is
    its row length, else the [R][C] view of a [R][stride] buffer holding t's values."""
    import torch
    from paper_2607_28848_amd import dsv
    R, C = t.shape
    st = dsv.row_stride(C, code)
    if st == C:
        return t
    buf = torch.zeros((R, st), dtype=t.dtype, device=t.device)
    buf[:, :C] = t
    return buf[:, :C]


def layout_note(w, code, layout):
    """The caller buffers' row strides of the timed step."""
    if layout == "dense":
        return "dense: every row exactly K or N elements"
    from paper_2607_28848_amd import dsv
    lens = sorted({n for p in w.projections for n in (p.K, p.N) if dsv.row_stride(n, code) != n})
    if not lens:
        return "strided (dsv_row_stride): every recommended stride is the row length, so dense"
    return ("strided: rows of %s elements (X, W, Y, dY, dX, W transposed) stored %s elements apart "
            "(dsv_row_stride), all other rows dense; the same values and FLOPs "
            "(extras.launch_modes_ms_per_step.set_dense is the same step on dense buffers)"
            % ("/".join(map(str, lens)), "/".join(str(dsv.row_stride(n, code)) for n in lens)))


def launch_groups(w, launch, dropout):
    """[(lo, hi)] ranges of w.projections run by one grouped call each, or None for
    one call per projection.  `layer` groups the projections whose inputs exist at
    the same point of a transformer layer: those sharing the layer input (q, k, v),
    the attention output (o), the MLP input (gate, up) and the MLP product (down).
    A workload of one projection is a group of one outside `single` mode, so its dX
    GEMM reads the transposed weight as in the grouped modes."""
    if launch == "single":
        return None
    if launch == "set" or len(w.projections) == 1:
        return [(0, len(w.projections))]
    names = [p.name for p in w.projections]
    order = [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]]
    if names != [n for g in order for n in g]:
        return [(i, i + 1) for i in range(len(names))]
    out, lo = [], 0
    for g in order:
        out.append((lo, lo + len(g)))
        lo += len(g)
    return out


def _gen(args):
    name, p = args
    w = WORKLOADS[name]()
    t = w.tensors(p, pad=0.0)
    return t.store


def cpu_baseline(w, stores, n_fwd_rows, n_dx_rows, seed=0):
    """The fp64 reference timed on the host cores over a bounded sample of the same
    workload: every projection's forward on n_fwd_rows sampled rows and its backward
    (g, dA, dB in full, dX on n_dx_rows sampled training rows)."""
    import oracle
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(w.n_tokens, n_fwd_rows, replace=False)).astype(np.int32)
    Tt = w.train_tokens
    dxr = np.sort(rng.choice(Tt, min(n_dx_rows, Tt), replace=False)).astype(np.int32) if Tt else None
    flops, secs = 0.0, 0.0
    row_rank = np.zeros(w.n_tokens, np.int64)
    for (s, l, a, _) in w.segments:
        row_rank[s:s + l] = int(w.ranks[a])
    tr_rank = row_rank[[t for (s, l, a, tt) in w.segments if tt for t in range(s, s + l)]]
    for p, proj in enumerate(w.projections):
        st = stores[p]
        cvt = (lambda b: wl.bf16_bits_to_f64(b)) if w.dtype == "bf16" else (lambda b: b.astype(np.float64))
        X, W, A, B, dY = (cvt(st[k]) for k in ("X", "W", "A", "B", "dY"))
        K, N = proj.K, proj.N
        t0 = time.perf_counter()
        oracle.forward(w.segments, w.ranks, w.scales, w.r_max, X, W, A, B, rows)
        if Tt:
            oracle.backward(w.segments, w.ranks, w.scales, w.r_max, X, W, A, B, dY, dx_rows=dxr)
        secs += time.perf_counter() - t0
        flops += float(sum(2.0 * K * N + 2.0 * row_rank[r] * (K + N) for r in rows))
        if Tt:
            rsum = float(tr_rank.sum())
            flops += 2.0 * rsum * N * 2 + 2.0 * rsum * K          # g, dB, dA
            flops += len(dxr) * 2.0 * N * K + 2.0 * K * float(tr_rank[dxr].sum())  # dX rows
        log("  cpu baseline %s: %.1f s so far" % (proj.name, secs))
    return flops, secs


def cpu_model():
    """The host CPU's model name (first entry of /proc/cpuinfo), or None."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def library_gemm_context(w, P, stream, reps=20):
    """The same GEMM shapes through torch (hipBLASLt / rocBLAS on ROCm) on the same
    resident bf16 data, as context for the roofline: each projection's forward base
    product X W^T ([T][K] x [N][K]^T) and dX product dY W ([T_t][N] x [N][K]), without
    the low-rank terms.  Timed as whole loops of the 7 + 7 products (the clock settles
    as it does in the bench's step), then one shape at a time."""
    import torch
    import torch.nn.functional as F
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    Tt = w.train_tokens
    outs = [(torch.empty((w.n_tokens, p.N), dtype=torch.bfloat16, device=P[i]["X"].device),
             torch.empty((max(Tt, 1), p.K), dtype=torch.bfloat16, device=P[i]["X"].device))
            for i, p in enumerate(w.projections)]

    def fwd(i):
        torch.matmul(P[i]["X"], P[i]["W"].t(), out=outs[i][0])

    def dx(i):
        torch.matmul(P[i]["dY"], P[i]["W"], out=outs[i][1])

    def timed(fn, n):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    ff = [2.0 * w.n_tokens * p.K * p.N for p in w.projections]
    fb = [2.0 * Tt * p.K * p.N for p in w.projections]
    n = len(w.projections)
    out = {"library": str(torch.backends.cuda.preferred_blas_library()),
           "note": "torch.matmul on the bench's resident bf16 operands, base products only"}
    t_fwd = timed(lambda: [fwd(i) for i in range(n)], reps)
    out["fwd_all_us"] = round(t_fwd, 1)
    out["fwd_all_tflops"] = round(sum(ff) / (t_fwd * 1e-6) / 1e12, 1)
    if Tt:
        t_bwd = timed(lambda: [dx(i) for i in range(n)], reps)
        out["dx_all_us"] = round(t_bwd, 1)
        out["dx_all_tflops"] = round(sum(fb) / (t_bwd * 1e-6) / 1e12, 1)
        t_both = timed(lambda: [fwd(i) for i in range(n)] + [dx(i) for i in range(n)], reps)
        out["fwd_plus_dx_us"] = round(t_both, 1)
        out["fwd_plus_dx_tflops"] = round((sum(ff) + sum(fb)) / (t_both * 1e-6) / 1e12, 1)
    per = {}
    for i, p in enumerate(w.projections):
        t = timed(lambda: fwd(i), reps)
        d = {"fwd_us": round(t, 1), "fwd_tflops": round(ff[i] / (t * 1e-6) / 1e12, 1)}
        if Tt:
            t = timed(lambda: dx(i), reps)
            d.update(dx_us=round(t, 1), dx_tflops=round(fb[i] / (t * 1e-6) / 1e12, 1))
        per["%s %dx%d" % (p.name, p.K, p.N)] = d
    out["per_projection"] = per
    del outs
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--time-every", type=int, default=5,
                    help="attach the HIP events that time the GEMM launches to every K-th timed step (a "
                         "dispatch that carries events starts several microseconds after the kernel before it "
                         "and delays the kernel after it; the other steps run without them)")
    ap.add_argument("--workload", default="llama8b", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=48, help="forward rows per projection in the CPU sample")
    ap.add_argument("--cpu-dx-rows", type=int, default=24)
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the timings after the main loop (AdamW, recomputed h, dropout, co-batching "
                         "overhead, launch modes)")
    ap.add_argument("--extras", default="all", choices=("all", "overhead", "library"),
                    help="overhead: of the timings after the main loop, only the co-batching overhead; "
                         "library: only the library-GEMM context")
    ap.add_argument("--launch", default="set", choices=("single", "layer", "set"),
                    help="single: one call per projection; layer: grouped calls over the projections a "
                         "transformer layer can run together (q/k/v, o, gate/up, down); set: one grouped call "
                         "over the whole set")
    ap.add_argument("--layout", default="strided", choices=("strided", "dense"),
                    help="strided: the grouped calls' caller buffers (X, W, Y, dY, dX, the transposed weight) "
                         "hold their rows at the stride dsv_row_stride recommends (rows of 14336 bf16 elements "
                         "64 elements apart more); dense: rows of exactly K or N elements.  The single-projection "
                         "calls (--launch single) take dense buffers")
    ap.add_argument("--no-wt", action="store_true",
                    help="grouped backward without the transposed copy of the frozen weights (the dX GEMM "
                         "then transposes W in the kernel)")
    ap.add_argument("--dropout", type=float, default=0.0, metavar="P",
                    help="LoRA dropout P on the training rows in the timed step (fresh mask per step)")
    ap.add_argument("--upload", default="side", choices=("side", "inorder"),
                    help="side: each step's plan metadata is uploaded on a side stream into alternating "
                         "buffers, overlapping the previous step; inorder: on the compute stream")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first run 3 plain device copies of MIB MiB (reference for HBM byte counters)")
    args = ap.parse_args()

    if args.time_every < 1:
        ap.error("--time-every must be at least 1")
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    w = WORKLOADS[args.workload]()
    log("workload %s: T=%d T_t=%d projections=%s" % (
        w.name, w.n_tokens, w.train_tokens, [(p.name, p.K, p.N) for p in w.projections]))
    t0 = time.time()
    with ProcessPoolExecutor(max_workers=min(8, len(w.projections))) as ex:
        stores = list(ex.map(_gen, [(args.workload, p) for p in range(len(w.projections))]))
    log("inputs drawn in %.1f s" % (time.time() - t0))

    import torch
    from paper_2607_28848_amd import dsv

    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    bf = w.dtype == "bf16"

    def up(a):
        if bf:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)

    if args.calibrate_copy > 0:
        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration: 3 copies of %d MiB" % args.calibrate_copy)
        del src, dst

    tdt = torch.bfloat16 if bf else torch.float32
    code = dsv.BF16 if bf else dsv.F32
    probe = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max)
    Tt = probe.train_tokens
    P = []
    for p, proj in enumerate(w.projections):
        st = stores[p]
        d = dict(X=up(st["X"]), W=up(st["W"]), A=up(st["A"]), B=up(st["B"]), dY=up(st["dY"]))
        K, N = proj.K, proj.N
        d["Y"] = torch.empty((w.n_tokens, N), dtype=tdt, device=dev)
        d["H"] = torch.empty((max(Tt, 1), w.r_max), dtype=tdt, device=dev)
        d["dX"] = torch.empty((max(Tt, 1), K), dtype=tdt, device=dev)
        d["dA"] = torch.zeros((w.n_adapters, w.r_max, K), dtype=torch.float32, device=dev)
        d["dB"] = torch.zeros((w.n_adapters, N, w.r_max), dtype=torch.float32, device=dev)
        # the frozen weight kept a second time, transposed, for the dX GEMM (set up once, like W)
        d["Wt"] = d["W"].t().contiguous()
        d["wsf"] = torch.empty(max(dsv.fwd_workspace_bytes(probe, code, K, N), 256), dtype=torch.uint8, device=dev)
        d["wsb"] = torch.empty(max(dsv.bwd_workspace_bytes(probe, code, K, N, dropout=args.dropout > 0), 256),
                               dtype=torch.uint8, device=dev)
        # the dropout mask of the step, drawn by the forward and read by the backward
        d["mask"] = torch.empty(max(dsv.dropout_mask_words(probe, K), 1), dtype=torch.int32, device=dev)
        # the same values in rows of the recommended stride (the grouped calls' strided layout)
        d["s"] = {k: strided_rows(d[k], code) for k in ("X", "W", "Y", "dY", "dX", "Wt")}
        P.append(d)
    torch.cuda.synchronize()
    log("inputs resident on %s" % torch.cuda.get_device_name(dev))

    lib = dsv.lib_handle()
    seg = np.ascontiguousarray(np.asarray(w.segments, np.int32).reshape(-1, 4))
    ranks = np.ascontiguousarray(w.ranks, np.int32)
    scales = np.ascontiguousarray(w.scales, np.float32)
    import ctypes
    i32p = ctypes.POINTER(ctypes.c_int32)
    f32p = ctypes.POINTER(ctypes.c_float)
    meta_bytes = ctypes.c_size_t(probe.meta_bytes)
    metas = [torch.empty(max(probe.meta_bytes, 256), dtype=torch.uint8, device=dev) for _ in range(2)]
    sh = ctypes.c_void_p(int(stream.cuda_stream))
    # A step's plan is uploaded on a side stream (default priority), so the copy of
    # step i's metadata overlaps step i-1's kernels instead of sitting between them.
    # The metadata is double-buffered: buffer b is rewritten only after the step that
    # last read it has finished (meta_free[b], recorded on the compute stream), and the
    # compute stream waits for the upload (meta_ready[b]) before its first kernel.
    up_stream = torch.cuda.Stream(dev)
    uh = ctypes.c_void_p(int(up_stream.cuda_stream))
    meta_free = [torch.cuda.Event() for _ in range(2)]
    meta_ready = [torch.cuda.Event() for _ in range(2)]
    ptr = lambda t: ctypes.c_void_p(int(t.data_ptr()))  # noqa: E731
    ld = lambda t: 0 if t.is_contiguous() else int(t.stride(0))  # noqa: E731
    plan_ms = []
    def make_step(launch, use_wt=not args.no_wt, layout=args.layout):
        """The step function of one launch mode, and its projection groups."""
        groups = launch_groups(w, launch, args.dropout)
        if groups is not None:
            shapes = [(proj.K, proj.N) for proj in w.projections]
            fproj = (dsv.FwdProj * len(P))()
            bproj = (dsv.BwdProj * len(P))()
            for p, (K, N) in enumerate(shapes):
                d = P[p]
                o = d["s"] if layout == "strided" else d
                fproj[p] = dsv.FwdProj(K, N, ptr(o["X"]), ptr(o["W"]), ptr(d["A"]), ptr(d["B"]), ptr(o["Y"]), ptr(d["H"]),
                                       ld(o["X"]), ld(o["W"]), ld(o["Y"]))
                bproj[p] = dsv.BwdProj(K, N, ptr(o["X"]), ptr(o["W"]), ptr(d["A"]), ptr(d["B"]), ptr(d["H"]), ptr(o["dY"]),
                                       ptr(d["dA"]), ptr(d["dB"]), ptr(o["dX"]), ptr(o["Wt"]) if use_wt else None,
                                       ld(o["X"]), ld(o["W"]), ld(o["dY"]), ld(o["dX"]), ld(o["Wt"]) if use_wt else 0)
            fgroup = [(dsv.FwdProj * (hi - lo))(*fproj[lo:hi]) for lo, hi in groups]
            bgroup = [(dsv.BwdProj * (hi - lo))(*bproj[lo:hi]) for lo, hi in groups]
            gws_f = [torch.empty(max(dsv.fwd_grouped_workspace_bytes(probe, code, shapes[lo:hi]), 256),
                                 dtype=torch.uint8, device=dev) for lo, hi in groups]
            gws_b = [torch.empty(max(dsv.bwd_grouped_workspace_bytes(probe, code, shapes[lo:hi]), 256),
                                 dtype=torch.uint8, device=dev) for lo, hi in groups]

        def step(i):
            h = ctypes.c_void_p()
            b = i & 1
            side = args.upload == "side"
            if side:
                up_stream.wait_event(meta_free[b])
            tp = time.perf_counter()
            rc = lib.dsv_segments_build(seg.ctypes.data_as(i32p), seg.shape[0], w.n_tokens,
                                        ranks.ctypes.data_as(i32p), scales.ctypes.data_as(f32p),
                                        ranks.shape[0], w.r_max, ptr(metas[b]), ctypes.byref(meta_bytes),
                                        uh if side else sh, ctypes.byref(h))
            plan_ms.append((time.perf_counter() - tp) * 1e3)
            if rc != 0:
                raise RuntimeError("dsv_segments_build failed: %d" % rc)
            if side:
                meta_ready[b].record(up_stream)
                stream.wait_event(meta_ready[b])
            if groups is not None:
                drs = None
                if args.dropout > 0:  # one mask stream per projection and step
                    drs = [(dsv.Dropout * (hi - lo))(*[dsv.Dropout(args.dropout, 1234, i * len(w.projections) + p,
                                                                   ptr(P[p]["mask"]))
                                                        for p in range(lo, hi)]) for lo, hi in groups]
                for gi, (lo, hi) in enumerate(groups):
                    if drs is None:
                        rc = lib.dsv_cobatch_fwd_grouped(h, code, hi - lo, fgroup[gi], ptr(gws_f[gi]),
                                                         gws_f[gi].numel(), sh)
                    else:
                        rc = lib.dsv_cobatch_fwd_grouped_dropout(h, code, hi - lo, fgroup[gi], drs[gi],
                                                                 ptr(gws_f[gi]), gws_f[gi].numel(), sh)
                    if rc != 0:
                        raise RuntimeError("dsv_cobatch_fwd_grouped failed: %d" % rc)
                for gi, (lo, hi) in enumerate(groups):
                    if drs is None:
                        rc = lib.dsv_lora_bwd_grouped(h, code, hi - lo, bgroup[gi], 0, ptr(gws_b[gi]),
                                                      gws_b[gi].numel(), sh)
                    else:
                        rc = lib.dsv_lora_bwd_grouped_dropout(h, code, hi - lo, bgroup[gi], 0, drs[gi],
                                                              ptr(gws_b[gi]), gws_b[gi].numel(), sh)
                    if rc != 0:
                        raise RuntimeError("dsv_lora_bwd_grouped failed: %d" % rc)
                if side:
                    meta_free[b].record(stream)
                lib.dsv_plan_free(h)
                return
            for p, proj in enumerate(w.projections):
                d = P[p]
                K, N = proj.K, proj.N
                if args.dropout > 0:
                    # one mask stream per projection and step: offset = step * projections + p
                    dr = ctypes.byref(dsv.Dropout(args.dropout, 1234, i * len(w.projections) + p, ptr(d["mask"])))
                    rc = lib.dsv_cobatch_fwd_dropout(h, code, K, N, ptr(d["X"]), ptr(d["W"]), ptr(d["A"]),
                                                     ptr(d["B"]), ptr(d["Y"]), ptr(d["H"]), dr, ptr(d["wsf"]),
                                                     d["wsf"].numel(), sh)
                else:
                    rc = lib.dsv_cobatch_fwd(h, code, K, N, ptr(d["X"]), ptr(d["W"]), ptr(d["A"]), ptr(d["B"]),
                                             ptr(d["Y"]), ptr(d["H"]), ptr(d["wsf"]), d["wsf"].numel(), sh)
                if rc != 0:
                    raise RuntimeError("dsv_cobatch_fwd failed: %d" % rc)
                if args.dropout > 0:
                    rc = lib.dsv_lora_bwd_dropout(h, code, K, N, ptr(d["X"]), ptr(d["W"]), ptr(d["A"]), ptr(d["B"]),
                                                  ptr(d["H"]), ptr(d["dY"]), ptr(d["dA"]), ptr(d["dB"]), ptr(d["dX"]),
                                                  0, dr, ptr(d["wsb"]), d["wsb"].numel(), sh)
                else:
                    rc = lib.dsv_lora_bwd(h, code, K, N, ptr(d["X"]), ptr(d["W"]), ptr(d["A"]), ptr(d["B"]),
                                          ptr(d["H"]), ptr(d["dY"]), ptr(d["dA"]), ptr(d["dB"]), ptr(d["dX"]),
                                          0, ptr(d["wsb"]), d["wsb"].numel(), sh)
                if rc != 0:
                    raise RuntimeError("dsv_lora_bwd failed: %d" % rc)
            if side:
                meta_free[b].record(stream)
            lib.dsv_plan_free(h)  # waits for the blob's upload; the device metadata stays valid
        return step, groups

    step, groups = make_step(args.launch)

    # No garbage-collector pass inside the timed loops: a full pass over the heap
    # (tens of ms) stalls the host, which stays only one step ahead of the GPU.
    gc.collect()
    gc.disable()
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log("warmup done (%d steps)" % args.warmup)
    plan_ms.clear()
    # The library times the GEMM launches of every time_every-th timed step with
    # HIP events that ride the launches' own dispatches; such a dispatch waits
    # several microseconds after the kernel before it, so the other steps run
    # without events.
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        dsv.timing_enable(i % args.time_every == 0)
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    dsv.timing_enable(False)
    plan_med = round(float(np.median(plan_ms)), 4) if plan_ms else None
    gpu_ms = ev0.elapsed_time(ev1)
    fwd_ms, fwd_n, bwd_ms, bwd_n = dsv.timing_read()
    elapsed_s = max(wall, gpu_ms / 1e3)
    ms_per_step = elapsed_s * 1e3 / args.steps

    step_flops = sum(sum(algo_flops(w, proj)) for proj in w.projections)
    value = step_flops * args.steps / elapsed_s / 1e12
    gathered = probe.gathered_rows().astype(np.int64)
    fwd_gemm_flops = sum(gemm_fwd_flops(w, proj, gathered) for proj in w.projections)
    bwd_gemm_flops = sum(gemm_bwd_flops(w, proj) for proj in w.projections)
    fwd_avg_ms = fwd_ms / max(fwd_n, 1)
    per_step = len(groups) if groups is not None else len(w.projections)  # timed GEMM launches per step
    achieved = fwd_gemm_flops * (fwd_n / per_step) / (fwd_ms / 1e3) / 1e12 if fwd_ms > 0 else None
    bwd_achieved = bwd_gemm_flops * (bwd_n / per_step) / (bwd_ms / 1e3) / 1e12 if bwd_ms > 0 else None
    log("timed %d steps: %.3f ms/step, %.1f TFLOP/s; fwd GEMM %.1f TFLOP/s avg %.1f us; dX GEMM %s TFLOP/s"
        % (args.steps, ms_per_step, value, achieved or 0, fwd_avg_ms * 1e3,
           "%.1f" % bwd_achieved if bwd_achieved else "n/a"))

    # The step after the backward: one fused AdamW update of the training adapter of
    # every projection (not part of `value`).  HBM bytes per updated element: gradient,
    # master, m and v read (16), master, m and v written (12), bf16 copy written (2).
    extras = None
    if not args.no_extras and bf:
        extras = {}
        full = args.extras == "all"
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        probe_dev = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device=dev)
        gl = groups if groups is not None else [(p, p + 1) for p in range(len(w.projections))]
        shapes = [(proj.K, proj.N) for proj in w.projections]
        if full:
            hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
            opt = []
            for p, proj in enumerate(w.projections):
                d = P[p]
                st = [d["A"].float(), d["B"].float()]
                opt.append(st + [torch.zeros_like(st[0]), torch.zeros_like(st[0]),
                                 torch.zeros_like(st[1]), torch.zeros_like(st[1])])
            torch.cuda.synchronize()

            opt_step = dsv.adamw_grouped_prepared(
                probe_dev, [(P[p]["dA"], P[p]["dB"], *opt[p], P[p]["A"], P[p]["B"]) for p in range(len(w.projections))],
                stream=stream, **hp)
            for t in range(1, 6):
                opt_step(t)
            torch.cuda.synchronize()
            n_opt = 50
            e0.record(stream)
            for t in range(6, 6 + n_opt):
                opt_step(t)
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / n_opt
            tr = [a for a in range(w.n_adapters) if any(s[2] == a and s[3] and s[1] for s in w.segments)]
            elems = sum(int(w.ranks[a]) * (proj.K + proj.N) for a in tr for proj in w.projections)
            nbytes = 30 * elems
            extras["adamw"] = {"kernel": "adamw_kernel (fused AdamW of the training adapters' A and B, "
                                         "every projection in one launch)",
                               "launches_per_step": 1, "us_per_step": round(us, 2),
                               "bytes_per_step": nbytes, "achieved_GBps": round(nbytes / (us * 1e-6) / 1e9, 1),
                               "peak_GBps": 8000.0, "frac": round(nbytes / (us * 1e-6) / 8e12, 4),
                               "bound": "hbm"}
            log("adamw: %.2f us per step (one launch), %.1f GB/s" % (us, nbytes / (us * 1e-6) / 1e9))

            # Residual-only retention: the backward of every projection with h recomputed
            # from X (H_save not kept) against the backward that reads the kept H_save.
            def bwd_all(keep):
                for p, proj in enumerate(w.projections):
                    d = P[p]
                    dsv.lora_bwd(probe_dev, d["X"], d["W"], d["A"], d["B"], d["H"] if keep else None, d["dY"],
                                 dA=d["dA"], dB=d["dB"], dX=d["dX"], workspace=d["wsb"], stream=stream)
            bt = {}
            for keep in (True, False, True, False):
                bwd_all(keep)
                torch.cuda.synchronize()
                e0.record(stream)
                for _ in range(10):
                    bwd_all(keep)
                e1.record(stream)
                torch.cuda.synchronize()
                bt[keep] = e0.elapsed_time(e1) * 1e3 / 10
            extras["recompute_h"] = {"bwd_us_per_step_kept_h": round(bt[True], 2),
                                     "bwd_us_per_step_recomputed_h": round(bt[False], 2),
                                     "h_bytes_not_kept_per_step": int(sum(w.train_tokens * w.r_max * 2
                                                                          for _ in w.projections))}
            log("backward with kept h %.1f us, with recomputed h %.1f us per step" % (bt[True], bt[False]))

            # LoRA dropout 0.05 on the training rows (the fine-tuning setting of Sec. 4.1):
            # the whole step (forward + backward of every projection, in the bench's launch
            # mode) with and without it; the backward reads the mask the forward drew.
            wsf_d = [torch.empty(max(dsv.fwd_grouped_workspace_bytes(probe, code, shapes[lo:hi]), 256),
                                 dtype=torch.uint8, device=dev) for lo, hi in gl]
            wsb_d = [torch.empty(max(dsv.bwd_grouped_workspace_bytes(probe, code, shapes[lo:hi]), 256),
                                 dtype=torch.uint8, device=dev) for lo, hi in gl]

            def step_all(drop):
                for gi, (lo, hi) in enumerate(gl):
                    ds = [P[p] for p in range(lo, hi)]
                    drops = None if drop is None else [(drop, 1234, p, P[p]["mask"]) for p in range(lo, hi)]
                    dsv.cobatch_fwd_grouped(probe_dev, [(d["X"], d["W"], d["A"], d["B"], d["Y"], d["H"]) for d in ds],
                                            workspace=wsf_d[gi], stream=stream, dropouts=drops)
                for gi, (lo, hi) in enumerate(gl):
                    ds = [P[p] for p in range(lo, hi)]
                    drops = None if drop is None else [(drop, 1234, p, P[p]["mask"]) for p in range(lo, hi)]
                    dsv.lora_bwd_grouped(probe_dev, [(d["X"], d["W"], d["A"], d["B"], d["H"], d["dY"], d["dA"], d["dB"],
                                                      d["dX"]) for d in ds],
                                         workspace=wsb_d[gi], stream=stream, dropouts=drops,
                                         wts=None if args.no_wt else [d["Wt"] for d in ds])
            dt_ = {}
            for key in ("off", "p0.05", "off", "p0.05"):
                drop = None if key == "off" else 0.05
                step_all(drop)
                torch.cuda.synchronize()
                e0.record(stream)
                for _ in range(10):
                    step_all(drop)
                e1.record(stream)
                torch.cuda.synchronize()
                dt_[key] = e0.elapsed_time(e1) * 1e3 / 10
            extras["dropout"] = {"p": 0.05, "step_us_without": round(dt_["off"], 2),
                                 "step_us_with": round(dt_["p0.05"], 2),
                                 "overhead_frac": round(dt_["p0.05"] / dt_["off"] - 1.0, 4)}
            log("step without dropout %.1f us, with dropout 0.05 %.1f us" % (dt_["off"], dt_["p0.05"]))
            del wsf_d, wsb_d

        # The same base products through torch's GEMM library, as context.
        if args.extras in ("all", "library"):
            extras["library_gemm"] = library_gemm_context(w, P, stream)
            log("library GEMMs: %s" % {k: v for k, v in extras["library_gemm"].items() if k != "per_projection"})

        # Co-batching overhead: the forward of the batch as it is against the forward of
        # the same segment table with every is_train flag cleared (no H_save rows, no
        # training-row bookkeeping), both in the bench's launch mode.
        if w.train_tokens > 0 and args.extras in ("all", "overhead"):
            inf_segs = [(s, l, a, 0) for (s, l, a, _) in w.segments]
            plan_inf = dsv.segments_build(inf_segs, w.n_tokens, w.ranks, w.scales, w.r_max, device=dev)
            wsf_o = [torch.empty(max(dsv.fwd_grouped_workspace_bytes(probe, code, shapes[lo:hi]), 256),
                                 dtype=torch.uint8, device=dev) for lo, hi in gl]

            def fwd_all(plan_, keep):
                for gi, (lo, hi) in enumerate(gl):
                    ds = [P[p] for p in range(lo, hi)]
                    dsv.cobatch_fwd_grouped(plan_, [(d["X"], d["W"], d["A"], d["B"], d["Y"], d["H"] if keep else None)
                                                    for d in ds], workspace=wsf_o[gi], stream=stream, keep_h=keep)
            ft = {}
            for key in ("mixed", "inference", "mixed", "inference"):
                pl, keep = (probe_dev, True) if key == "mixed" else (plan_inf, False)
                fwd_all(pl, keep)
                torch.cuda.synchronize()
                e0.record(stream)
                for _ in range(20):
                    fwd_all(pl, keep)
                e1.record(stream)
                torch.cuda.synchronize()
                ft[key] = e0.elapsed_time(e1) * 1e3 / 20
            extras["cobatch_overhead"] = {
                "fwd_us_mixed": round(ft["mixed"], 2), "fwd_us_is_train_cleared": round(ft["inference"], 2),
                "overhead_frac": round(ft["mixed"] / ft["inference"] - 1.0, 4)}
            log("forward: mixed batch %.1f us, is_train cleared %.1f us" % (ft["mixed"], ft["inference"]))
            del wsf_o, plan_inf

        if full:
            # The same step in the other launch modes (10 timed steps each); "<mode>_no_wt":
            # the grouped backward without the transposed weights.
            modes = {args.launch + ("_no_wt" if args.no_wt else ""): round(ms_per_step, 4)}
            other = "dense" if args.layout == "strided" else "strided"
            for m in ("single", "layer", "set", "layer_no_wt", "set_no_wt", "set_" + other):
                if m in modes or (m == args.launch and not args.no_wt):
                    continue
                st, _ = make_step(m.split("_")[0], use_wt=not m.endswith("_no_wt"),
                                  layout=other if m.endswith("_" + other) else args.layout)
                for i in range(3):
                    st(i)
                torch.cuda.synchronize()
                e0.record(stream)
                for i in range(10):
                    st(i)
                e1.record(stream)
                torch.cuda.synchronize()
                modes[m] = round(e0.elapsed_time(e1) / 10, 4)
            extras["launch_modes_ms_per_step"] = modes
            log("ms per step by launch mode: %s" % modes)

    def cfg_str(c):
        if not c["tile_m"]:
            return None
        s = "%dx%d tiles, %dx%d" % (c["tile_m"], c["tile_n"], c["row_tiles"], c["col_tiles"])
        if c["split_tiles"]:
            s += ", %d split %d ways" % (c["split_tiles"], c["split_ways"])
        return s
    gemm_launches = {proj.name: {"fwd": cfg_str(dsv.gemm_config(probe, code, proj.K, proj.N, 0)),
                                 "dx": cfg_str(dsv.gemm_config(probe, code, proj.K, proj.N, 1))}
                     for proj in w.projections}
    roof_kernel = ("gemm16_kernel (256x256 tiles; gemm_lora_kernel for 128x128) + split_fixup_kernel<NT> "
                   "(forward base GEMM with the low-rank prologue; the fixup sums contraction-split tiles)")
    if groups is not None and any(hi - lo > 1 for lo, hi in groups):
        pc = probe.counts()
        for lo, hi in groups:
            if hi - lo < 2:
                continue
            ps = w.projections[lo:hi]
            gemm_launches["+".join(p.name for p in ps)] = {
                "fwd": "256x256 tiles, %d in one launch" % sum(pc["fwd_tiles"] * ((p.N + 255) // 256) for p in ps),
                "dx": "256x256 tiles, %d in one launch" % sum(pc["bwd_tiles"] * ((p.K + 255) // 256) for p in ps)}
            for p in ps:
                gemm_launches.pop(p.name, None)
        roof_kernel = ("gemm16_group_kernel<false> (the forward base GEMMs with their low-rank prologues, every "
                       "projection of a group in one launch; with --launch set, one launch per step)")

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline: fp64 reference on a sample (%d rows/projection fwd, %d dX rows)"
            % (args.cpu_rows, args.cpu_dx_rows))
        fl, secs = cpu_baseline(w, stores, args.cpu_rows, args.cpu_dx_rows)
        import oracle
        cpu = {"value": fl / secs / 1e12, "unit": "TFLOP/s", "cores": oracle.threads(), "kind": "oracle",
               "cpu_model": cpu_model(), "affinity_cpus": len(os.sched_getaffinity(0)),
               "sample": "every projection: forward of %d sampled rows, backward g/dA/dB over all %d "
                         "training rows and dX of %d sampled training rows; %.2f GFLOP in %.1f s"
                         % (args.cpu_rows, w.train_tokens, args.cpu_dx_rows, fl / 1e9, secs)}

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf else "f32",
        "data": "synthetic",
        "pct_of_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "config": {
            "workload": w.name,
            "tokens": w.n_tokens,
            "train_tokens": w.train_tokens,
            "projections_KxN": [[p.name, p.K, p.N] for p in w.projections],
            "adapters": w.n_adapters,
            "ranks": sorted(set(int(r) for r in w.ranks)),
            "algorithmic_gflop_per_step": round(step_flops / 1e9, 2),
            "plan_build_ms": plan_med,
            "lora_dropout": args.dropout,
            "metadata_upload": args.upload,
            "launch": args.launch,
            "launch_note": LAUNCH_NOTES[args.launch],
            "dx_weight": "W transposed (kept once, like W)" if groups is not None and not args.no_wt else "W",
            "layout": layout_note(w, code, args.layout if groups is not None else "dense"),
            "launch_groups": ([[p.name for p in w.projections[lo:hi]] for lo, hi in groups] if groups is not None
                              else [[p.name] for p in w.projections]),
        },
        "roofline": {
            "kernel": roof_kernel,
            "bound": "mfma",
            "achieved": round(achieved, 2) if achieved else None,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4) if achieved else None,
            # the counter record is of the one-launch forward of the default run (the
            # 8B set in one grouped call on row-strided buffers)
            "traffic": (round(measured_traffic()) if measured_traffic() and args.workload == "llama8b"
                        and args.launch == "set" and args.layout == "strided" and args.dropout == 0
                        else None),
            "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "avg_launch_us": round(fwd_avg_ms * 1e3, 2),
            "launches": fwd_n,
            "launch_timing": ("HIP events attached to the GEMM dispatches of one timed step in %d"
                              % args.time_every),
            "dx_gemm_tflops": round(bwd_achieved, 2) if bwd_achieved else None,
            "gemm_launches": gemm_launches,
        },
        "cpu_baseline": cpu,
        "extras": extras,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
