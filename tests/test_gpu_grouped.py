"""GPU parity of the grouped launches (dsv_cobatch_fwd_grouped /
dsv_lora_bwd_grouped): several projections of one batch, one launch per step.

Bar: every output of every projection within 2e-2 (bf16) or 1e-5 (fp32) of the
fp64 reference; bit-identical to the single-projection calls wherever those do
not split a GEMM tile along the contraction (same summation order); a repeat
is bit-identical.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_28848_amd import workloads as wl
from gpu_util import TOL_BF16, TOL_F32, oracle_bwd, oracle_fwd, to_dev, to_host, train_mask_slices

pytestmark = pytest.mark.gpu

MIXED = [(0, 100, 3, 0), (100, 1, 1, 0), (101, 1, 2, 0), (102, 300, 0, 1), (402, 1, 3, 0),
         (403, 57, 2, 0), (460, 2, 1, 0), (462, 129, 1, 1), (591, 3, 0, 0), (594, 111, 4, 0)]
MIXED_RANKS = [16, 8, 64, 32, 5]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bits(t):
    import torch
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _layer(dtype, shapes, segments=MIXED, ranks=MIXED_RANKS, r_max=64, name="grouped"):
    """Workload whose projections have the given (K, N) shapes, inputs on the device."""
    w = wl.custom(segments, ranks, K=shapes[0][0], N=shapes[0][1], dtype=dtype, r_max=r_max, name=name)
    w.projections = [wl.Projection("p%d" % i, K, N) for i, (K, N) in enumerate(shapes)]
    ts = [w.tensors(i) for i in range(len(shapes))]
    dev = [{k: to_dev(t.store[k], dtype) for k in ("X", "W", "A", "B", "dY")} for t in ts]
    return w, ts, dev


def _check_proj(w, t, tr, Y, H, dA, dB, dX, tol, rows=None, dx_rows=None):
    Yr, _ = oracle_fwd(w, t, rows)
    Yg = to_host(Y) if rows is None else to_host(Y)[rows]
    errs = {"Y": oracle.rel_err(Yg, Yr)}
    if H is not None:
        errs["H_save"] = oracle.rel_err(to_host(H), oracle_fwd(w, t, tr)[1])
    _, dAr, dBr, dXr = oracle_bwd(w, t, dx_rows=dx_rows)
    dAg, dBg = to_host(dA), to_host(dB)
    for a, r in train_mask_slices(w):
        errs["dA%d" % a] = oracle.rel_err(dAg[a, :r], dAr[a, :r])
        errs["dB%d" % a] = oracle.rel_err(dBg[a, :, :r], dBr[a, :, :r])
    if dX is not None:
        dXg = to_host(dX) if dx_rows is None else to_host(dX)[dx_rows]
        errs["dX"] = oracle.rel_err(dXg, dXr)
    _say("  rel errors: " + ", ".join("%s=%.2e" % kv for kv in errs.items()))
    for k, v in errs.items():
        assert v <= tol, (k, v)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_grouped_mixed_shapes_against_reference(dtype):
    """Four projections with different K and N (ragged against 64 and 256), one of
    them keeping no H_save (h recomputed in the backward) and one without dX;
    every output of every projection against the reference."""
    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(520, 776), (136, 1040), (1040, 264), (520, 136)]
    _say("case grouped %s %s" % (dtype, shapes))
    w, ts, dev = _layer(dtype, shapes)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    fw = []
    for i, d in enumerate(dev):
        H = None if i == 1 else torch.zeros((plan.train_tokens, w.r_max), dtype=d["X"].dtype, device="cuda")
        fw.append((d["X"], d["W"], d["A"], d["B"], None, H))
    out = dsv.cobatch_fwd_grouped(plan, fw, keep_h=False)
    bw = [(d["X"], d["W"], d["A"], d["B"], out[i][1], d["dY"], None, None,
           None if i == 3 else torch.empty((plan.train_tokens, shapes[i][0]), dtype=d["X"].dtype, device="cuda"))
          for i, d in enumerate(dev)]
    grads = dsv.lora_bwd_grouped(plan, bw, want_dx=True)
    torch.cuda.synchronize()
    tr = plan.train_rows()
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    for i in range(len(shapes)):
        w.projections = [wl.Projection("p", *shapes[i])]
        _say(" projection %d K=%d N=%d" % ((i,) + shapes[i]))
        dX = grads[i][2] if i != 3 else None
        _check_proj(w, ts[i], tr, out[i][0], out[i][1], grads[i][0], grads[i][1], dX, tol)


def test_grouped_matches_single_calls_and_repeats():
    """bf16: the grouped results equal the single calls bit for bit on every
    projection whose single call splits no tile (and within the bar on the others);
    a second grouped call is bit-identical to the first."""
    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(4096, 1024), (1024, 4096), (4096, 2048), (2048, 776)]
    _say("case grouped vs single %s" % shapes)
    w, ts, dev = _layer("bf16", shapes)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    Tt = plan.train_tokens

    def hbuf():
        return torch.zeros((Tt, w.r_max), dtype=torch.bfloat16, device="cuda")

    runs = []
    for rep in range(2):
        out = dsv.cobatch_fwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], None, hbuf()) for d in dev])
        grads = dsv.lora_bwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], out[i][1], d["dY"])
                                            for i, d in enumerate(dev)])
        runs.append((out, grads))
    singles = []
    for i, d in enumerate(dev):
        Y, H = dsv.cobatch_fwd(plan, d["X"], d["W"], d["A"], d["B"], H_save=hbuf())
        g = dsv.lora_bwd(plan, d["X"], d["W"], d["A"], d["B"], H, d["dY"])
        singles.append(((Y, H), g))
    torch.cuda.synchronize()
    (o1, g1), (o2, g2) = runs
    for i, (K, N) in enumerate(shapes):
        for a, b in list(zip(o1[i], o2[i])) + list(zip(g1[i], g2[i])):
            assert torch.equal(_bits(a), _bits(b))
        fsplit = dsv.gemm_config(plan, dsv.BF16, K, N, 0)["split_tiles"]
        bsplit = dsv.gemm_config(plan, dsv.BF16, K, N, 1)["split_tiles"]
        (Ys, Hs), (dAs, dBs, dXs) = singles[i]
        _say("  projection %d K=%d N=%d: single-call splits fwd %d dX %d" % (i, K, N, fsplit, bsplit))
        assert torch.equal(_bits(o1[i][1]), _bits(Hs))
        assert torch.equal(_bits(g1[i][0]), _bits(dAs)) and torch.equal(_bits(g1[i][1]), _bits(dBs))
        if fsplit == 0:
            assert torch.equal(_bits(o1[i][0]), _bits(Ys))
        else:
            assert oracle.rel_err(to_host(o1[i][0]), to_host(Ys)) <= 1e-2
        if bsplit == 0:
            assert torch.equal(_bits(g1[i][2]), _bits(dXs))
        else:
            assert oracle.rel_err(to_host(g1[i][2]), to_host(dXs)) <= 1e-2


@pytest.mark.timeout(900)
def test_grouped_llama8b_layer_set_full_size():
    """The launch the benchmark times, at full size: the whole Llama-3-8B layer set
    (q, k, v, o, gate, up, down) of the mixed batch (T = 6144 rows: 4096 inference
    + 2048 training) in one grouped forward and one grouped backward whose dX GEMMs
    read the transposed frozen weights.  Y and dX of every projection on sampled
    rows, H_save, dA, dB in full, against the fp64 reference; the backward without
    the transposed weights, and both calls on the benchmark's row-strided buffers,
    are bit-identical."""
    import torch
    from paper_2607_28848_amd import dsv
    w = wl.llama8b_mixed()
    _say("case grouped %s (bench launch: one call per step kind, dX on W transposed)" % w.name)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    ts, dev = [], []
    for i in range(len(w.projections)):
        t = w.tensors(i)
        ts.append(t)
        dev.append({k: to_dev(t.store[k], "bf16") for k in ("X", "W", "A", "B", "dY")})
    wts = [d["W"].t().contiguous() for d in dev]
    out = dsv.cobatch_fwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"]) for d in dev])
    bw = [(d["X"], d["W"], d["A"], d["B"], out[i][1], d["dY"]) for i, d in enumerate(dev)]
    grads = dsv.lora_bwd_grouped(plan, bw, wts=wts)
    plain = dsv.lora_bwd_grouped(plan, bw)
    torch.cuda.synchronize()
    for i in range(len(dev)):
        for a, b in zip(grads[i], plain[i]):
            assert torch.equal(_bits(a), _bits(b))
    del plain

    # the benchmark's default layout: rows of the recommended stride (gate/up/down
    # rows of 14336 elements 14400 apart), bit-identical to the dense buffers
    def srow(t):
        st = dsv.row_stride(t.shape[1], dsv.BF16)
        if st == t.shape[1]:
            return t
        buf = torch.zeros((t.shape[0], st), dtype=t.dtype, device=t.device)
        buf[:, :t.shape[1]] = t
        return buf[:, :t.shape[1]]

    assert any(dsv.row_stride(n, dsv.BF16) != n for p in w.projections for n in (p.K, p.N))
    sdev = [{k: srow(d[k]) for k in ("X", "W", "dY")} for d in dev]
    out_s = dsv.cobatch_fwd_grouped(plan, [(s["X"], s["W"], d["A"], d["B"], srow(torch.zeros_like(out[i][0])),
                                            torch.zeros_like(out[i][1])) for i, (s, d) in enumerate(zip(sdev, dev))])
    grads_s = dsv.lora_bwd_grouped(plan, [(s["X"], s["W"], d["A"], d["B"], out_s[i][1], s["dY"], None, None,
                                           srow(torch.zeros_like(grads[i][2])))
                                          for i, (s, d) in enumerate(zip(sdev, dev))], wts=[srow(t) for t in wts])
    torch.cuda.synchronize()
    for i in range(len(dev)):
        for a, b in list(zip(out_s[i], out[i])) + list(zip(grads_s[i], grads[i])):
            assert torch.equal(_bits(a.contiguous()), _bits(b))
    del sdev, out_s, grads_s, wts
    tr = plan.train_rows()
    rng = np.random.default_rng(11)
    Tt = w.train_tokens
    assert (w.n_tokens, Tt) == (6144, 2048)
    projs = list(w.projections)
    for i, proj in enumerate(projs):
        _say(" projection %s K=%d N=%d" % (proj.name, proj.K, proj.N))
        rows = np.unique(np.concatenate([rng.choice(w.n_tokens, 12, replace=False), tr[:1], tr[-1:]]))
        dx_rows = np.unique(np.concatenate([rng.choice(Tt, 12, replace=False), [0, Tt - 1]]))
        w.projections = [proj]
        _check_proj(w, ts[i], tr, out[i][0], out[i][1], grads[i][0], grads[i][1], grads[i][2], TOL_BF16,
                    rows=rows.astype(np.int32), dx_rows=dx_rows.astype(np.int32))
    w.projections = projs


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_grouped_dropout_against_reference(dtype):
    """Grouped calls with one dropout per projection (two seeds, an offset, one
    projection at p = 0 and one keeping no H_save): every output of every
    projection against the reference fed each projection's own mask; the p = 0
    projection matches the plain single call."""
    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(520, 776), (136, 1040), (1040, 264)]
    drops = [(0.3, 0x0123456789ABCDEF, 5), (0.0, 7, 0), (0.05, 0xFEDCBA9876543210, (3 << 32) | 1)]
    _say("case grouped dropout %s %s" % (dtype, shapes))
    w, ts, dev = _layer(dtype, shapes)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    Tt = plan.train_tokens
    fw = []
    for i, d in enumerate(dev):
        H = None if i == 2 else torch.zeros((Tt, w.r_max), dtype=d["X"].dtype, device="cuda")
        fw.append((d["X"], d["W"], d["A"], d["B"], None, H))
    out = dsv.cobatch_fwd_grouped(plan, fw, keep_h=False, dropouts=drops)
    grads = dsv.lora_bwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], out[i][1], d["dY"])
                                        for i, d in enumerate(dev)], dropouts=drops)
    Hp = torch.zeros((Tt, w.r_max), dtype=dev[1]["X"].dtype, device="cuda")
    Y1, H1 = dsv.cobatch_fwd(plan, dev[1]["X"], dev[1]["W"], dev[1]["A"], dev[1]["B"], H_save=Hp)
    g1 = dsv.lora_bwd(plan, dev[1]["X"], dev[1]["W"], dev[1]["A"], dev[1]["B"], H1, dev[1]["dY"])
    torch.cuda.synchronize()
    tr = plan.train_rows()
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    for i, (K, N) in enumerate(shapes):
        _say(" projection %d K=%d N=%d p=%.2f" % (i, K, N, drops[i][0]))
        drop = oracle.dropout_multipliers(Tt, K, *drops[i])
        Yr, _ = oracle_fwd(w, ts[i], drop=drop)
        errs = {"Y": oracle.rel_err(to_host(out[i][0]), Yr)}
        if out[i][1] is not None:
            errs["H_save"] = oracle.rel_err(to_host(out[i][1]), oracle_fwd(w, ts[i], tr, drop=drop)[1])
        _, dAr, dBr, dXr = oracle_bwd(w, ts[i], drop=drop)
        dAg, dBg = to_host(grads[i][0]), to_host(grads[i][1])
        for a, r in train_mask_slices(w):
            errs["dA%d" % a] = oracle.rel_err(dAg[a, :r], dAr[a, :r])
            errs["dB%d" % a] = oracle.rel_err(dBg[a, :, :r], dBr[a, :, :r])
        errs["dX"] = oracle.rel_err(to_host(grads[i][2]), dXr)
        _say("  rel errors: " + ", ".join("%s=%.2e" % kv for kv in errs.items()))
        for k, v in errs.items():
            assert v <= tol, (k, v)
    K, N = shapes[1]
    same_fwd = dsv.gemm_config(plan, dsv.BF16, K, N, 0)["split_tiles"] == 0 or dtype == "f32"
    same_bwd = dsv.gemm_config(plan, dsv.BF16, K, N, 1)["split_tiles"] == 0 or dtype == "f32"
    assert torch.equal(_bits(out[1][1]), _bits(H1))
    assert torch.equal(_bits(grads[1][0]), _bits(g1[0])) and torch.equal(_bits(grads[1][1]), _bits(g1[1]))
    if same_fwd:
        assert torch.equal(_bits(out[1][0]), _bits(Y1))
    if same_bwd:
        assert torch.equal(_bits(grads[1][2]), _bits(g1[2]))


@pytest.mark.parametrize("n_proj", [1, 3])
def test_grouped_transposed_weight_bit_identical(n_proj):
    """bf16 backward with the frozen weight also given transposed (dsv_bwd_proj.Wt):
    the dX GEMM reads it contraction-contiguous (NT) instead of transposing W in the
    kernel; dA, dB and dX are bit-identical to the plain call, with and without
    dropout (the dropout mask of g A_a sits in the NT GEMM's prologue then), and
    within the bar of the reference."""
    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(520, 776), (136, 1040), (4096, 2048)][:n_proj]
    _say("case transposed weight %s" % shapes)
    w, ts, dev = _layer("bf16", shapes)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    out = dsv.cobatch_fwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"]) for d in dev])
    bw = [(d["X"], d["W"], d["A"], d["B"], out[i][1], d["dY"]) for i, d in enumerate(dev)]
    wts = [d["W"].t().contiguous() for d in dev]
    drops = [(0.1, 99, i) for i in range(n_proj)]
    plain = dsv.lora_bwd_grouped(plan, bw)
    viat = dsv.lora_bwd_grouped(plan, bw, wts=wts)
    plain_d = dsv.lora_bwd_grouped(plan, bw, dropouts=drops)
    viat_d = dsv.lora_bwd_grouped(plan, bw, dropouts=drops, wts=wts)
    torch.cuda.synchronize()
    for i in range(n_proj):
        for a, b in list(zip(plain[i], viat[i])) + list(zip(plain_d[i], viat_d[i])):
            assert torch.equal(_bits(a), _bits(b))
        w.projections = [wl.Projection("p", *shapes[i])]
        _, _, _, dXr = oracle_bwd(w, ts[i])
        err = oracle.rel_err(to_host(viat[i][2]), dXr)
        _say("  projection %d dX rel err %.2e" % (i, err))
        assert err <= TOL_BF16


def test_grouped_inference_only_training_only_and_empty():
    """Degenerate batches through the grouped calls: no training rows (the backward is
    a no-op, dA/dB untouched), training rows only, and an empty batch (nothing
    written)."""
    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(264, 136), (136, 264)]
    for segs, name in (([(0, 40, 0, 0), (40, 3, 1, 0), (43, 20, 2, 0)], "inference only"),
                       ([(0, 40, 0, 1), (40, 30, 2, 1)], "training only")):
        _say("case grouped %s" % name)
        w, ts, dev = _layer("bf16", shapes, segments=segs, ranks=[8, 4, 16], r_max=16)
        plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
        out = dsv.cobatch_fwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"]) for d in dev])
        sent = [(torch.full_like(torch.zeros(3, w.r_max, shapes[i][0]), 7.0).cuda(),
                 torch.full_like(torch.zeros(3, shapes[i][1], w.r_max), 7.0).cuda()) for i in range(2)]
        Tt = plan.train_tokens
        dY = [d["dY"] if Tt else None for d in dev]
        grads = dsv.lora_bwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], out[i][1], dY[i] if Tt else d["X"],
                                             sent[i][0], sent[i][1]) for i, d in enumerate(dev)])
        torch.cuda.synchronize()
        for i in range(2):
            w.projections = [wl.Projection("p", *shapes[i])]
            Yr, _ = oracle_fwd(w, ts[i])
            assert oracle.rel_err(to_host(out[i][0]), Yr) <= TOL_BF16
            if not Tt:
                assert (sent[i][0] == 7.0).all() and (sent[i][1] == 7.0).all()
            else:
                _, dAr, dBr, dXr = oracle_bwd(w, ts[i])
                for a, r in train_mask_slices(w):
                    assert oracle.rel_err(to_host(grads[i][0])[a, :r], dAr[a, :r]) <= TOL_BF16
                    assert oracle.rel_err(to_host(grads[i][1])[a, :, :r], dBr[a, :, :r]) <= TOL_BF16
                assert oracle.rel_err(to_host(grads[i][2]), dXr) <= TOL_BF16
    # empty batch: nothing is launched or written
    plan = dsv.segments_build([], 0, [4], [1.0], 4, device="cuda")
    X = torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((64, 64), dtype=torch.bfloat16, device="cuda")
    A = torch.zeros((1, 4, 64), dtype=torch.bfloat16, device="cuda")
    B = torch.zeros((1, 64, 4), dtype=torch.bfloat16, device="cuda")
    out = dsv.cobatch_fwd_grouped(plan, [(X, W, A, B), (X, W, A, B)])
    torch.cuda.synchronize()
    assert out[0][0].shape == (0, 64)


def test_grouped_backward_graph_replay():
    """The grouped backward, whose dA reductions and final sums fork to the
    library's side stream and join back, captured in a graph on torch's capture
    stream and replayed three times with eager work (clearing the outputs)
    between replays: every replay's dA, dB and dX bit-identical to the eager
    call's."""
    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(520, 776), (136, 1040), (1040, 264)]
    _say("case graph replay of the grouped backward %s" % shapes)
    w, ts, dev = _layer("bf16", shapes)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    Tt = plan.train_tokens
    fw = dsv.cobatch_fwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], None,
                                         torch.zeros((Tt, w.r_max), dtype=torch.bfloat16, device="cuda"))
                                        for d in dev])
    n_ad = len(w.ranks)
    outs = [(torch.zeros((n_ad, w.r_max, K), dtype=torch.float32, device="cuda"),
             torch.zeros((n_ad, N, w.r_max), dtype=torch.float32, device="cuda"),
             torch.zeros((Tt, K), dtype=torch.bfloat16, device="cuda")) for K, N in shapes]
    bw = [(d["X"], d["W"], d["A"], d["B"], fw[i][1], d["dY"], *outs[i]) for i, d in enumerate(dev)]
    ws = torch.empty(max(dsv.bwd_grouped_workspace_bytes(plan, dsv.BF16, shapes), 256), dtype=torch.uint8,
                     device="cuda")
    dsv.lora_bwd_grouped(plan, bw, workspace=ws)
    torch.cuda.synchronize()
    ref = [tuple(t.clone() for t in o) for o in outs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        dsv.lora_bwd_grouped(plan, bw, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dsv.lora_bwd_grouped(plan, bw, workspace=ws)
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outs:
            for t in o:
                t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _say(" replay %d" % rep)
        for o, r in zip(outs, ref):
            for a, b in zip(o, r):
                assert torch.equal(_bits(a), _bits(b))


def test_grouped_backward_accumulate_and_threads():
    """The grouped backward's final sums run on the library's side stream.
    accumulate=1 there adds exactly what an overwriting call writes (checked bit
    for bit against the overwriting call plus the prior values, where that sum is
    exact: the prior values are zeros, then the call's own result), and slices of
    adapters without training rows keep their bits.  Two host threads running the
    grouped backward at once on two streams (the side stream and its events are
    shared) give the single-threaded results bit for bit."""
    import threading

    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(520, 776), (136, 1040), (1040, 264)]
    _say("case grouped accumulate and threads %s" % shapes)
    w, ts, dev = _layer("bf16", shapes)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    Tt = plan.train_tokens
    fw = dsv.cobatch_fwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], None,
                                         torch.zeros((Tt, w.r_max), dtype=torch.bfloat16, device="cuda"))
                                        for d in dev])
    n_ad = len(w.ranks)

    def outputs(fill=0.0):
        return [(torch.full((n_ad, w.r_max, K), fill, dtype=torch.float32, device="cuda"),
                 torch.full((n_ad, N, w.r_max), fill, dtype=torch.float32, device="cuda"),
                 torch.zeros((Tt, K), dtype=torch.bfloat16, device="cuda")) for K, N in shapes]

    def bwd(outs, accumulate=False, stream=None):
        bw = [(d["X"], d["W"], d["A"], d["B"], fw[i][1], d["dY"], *outs[i]) for i, d in enumerate(dev)]
        dsv.lora_bwd_grouped(plan, bw, accumulate=accumulate, stream=stream)

    ref = outputs()
    bwd(ref)
    torch.cuda.synchronize()
    # accumulate onto zeros, then onto the result itself: x + 0 = x and x + x = 2x exactly
    acc = outputs()
    bwd(acc, accumulate=True)
    torch.cuda.synchronize()
    for o, r in zip(acc, ref):
        assert torch.equal(_bits(o[0]), _bits(r[0])) and torch.equal(_bits(o[1]), _bits(r[1]))
    bwd(acc, accumulate=True)
    torch.cuda.synchronize()
    owners = dict(train_mask_slices(w))
    for o, r in zip(acc, ref):
        for a in range(n_ad):
            if a in owners:
                assert torch.equal(_bits(o[0][a]), _bits(2 * r[0][a])) and torch.equal(_bits(o[1][a]), _bits(2 * r[1][a]))
            else:
                assert torch.equal(_bits(o[0][a]), _bits(r[0][a])) and torch.equal(_bits(o[1][a]), _bits(r[1][a]))
    # two threads, two streams, several calls each
    outs = [outputs(), outputs()]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    errors = []

    def worker(k):
        try:
            with torch.cuda.stream(streams[k]):
                for _ in range(4):
                    bwd(outs[k], stream=streams[k])
        except Exception as exc:  # noqa: BLE001
            errors.append(exc)

    th = [threading.Thread(target=worker, args=(k,)) for k in range(2)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for k in range(2):
        for o, r in zip(outs[k], ref):
            for a, b in zip(o, r):
                assert torch.equal(_bits(a), _bits(b))
