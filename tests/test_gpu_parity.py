"""GPU parity: the HIP path (through the C ABI) against the fp64 reference.

Bar: max|gpu - ref| / max|ref| per output tensor <= 2e-2 for bf16 inputs and
<= 1e-5 for fp32 inputs; indexing (H_save placement, untouched slices and
padding) bit-exact; permuting the segment table and repeating a call give
bit-identical results.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_28848_amd import workloads as wl
from gpu_util import (TOL_BF16, TOL_F32, Run, oracle_bwd, oracle_fwd, to_host,
                      train_mask_slices)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _check_all(w, run, Y, H, dA, dB, dX, tol, rows=None, dx_rows=None):
    t = run.t
    Yr, Hr = oracle_fwd(w, t, rows)
    Yg = to_host(Y) if rows is None else to_host(Y)[rows]
    errs = {"Y": oracle.rel_err(Yg, Yr)}
    tr = run.plan.train_rows()
    if len(tr):
        Hg = to_host(H)
        # H_save row i is the h of token row tr[i]
        Hfull, _ = None, None
        Hr_t = oracle_fwd(w, t, tr)[1]
        errs["H_save"] = oracle.rel_err(Hg, Hr_t)
        G, dAr, dBr, dXr = oracle_bwd(w, t, dx_rows=dx_rows)
        dAg, dBg = to_host(dA), to_host(dB)
        for a, r in train_mask_slices(w):
            errs["dA%d" % a] = oracle.rel_err(dAg[a, :r], dAr[a, :r])
            errs["dB%d" % a] = oracle.rel_err(dBg[a, :, :r], dBr[a, :, :r])
        dXg = to_host(dX) if dx_rows is None else to_host(dX)[dx_rows]
        errs["dX"] = oracle.rel_err(dXg, dXr)
    _say("  rel errors: " + ", ".join("%s=%.2e" % kv for kv in errs.items()))
    for k, v in errs.items():
        assert v <= tol, (k, v)
    return errs


def _full(w, pad=np.nan, tol=TOL_BF16):
    _say("case %s T=%d Tt=%d K=%d N=%d" % (w.name, w.n_tokens, w.train_tokens,
                                          w.projections[0].K, w.projections[0].N))
    run = Run(w, pad=pad)
    Y, H = run.fwd()
    dA, dB, dX = run.bwd(H)
    import torch
    torch.cuda.synchronize()
    return run, _check_all(w, run, Y, H, dA, dB, dX, tol)


def test_tiny_f32():
    """Tiny fp32 layer: K = N = 512, 2 adapters of rank 8, 3 segments."""
    _full(wl.tiny(), tol=TOL_F32)


MIXED = [(0, 100, 3, 0), (100, 1, 1, 0), (101, 1, 2, 0), (102, 300, 0, 1), (402, 1, 3, 0),
         (403, 57, 2, 0), (460, 2, 1, 0), (462, 129, 1, 1), (591, 3, 0, 0), (594, 111, 4, 0)]
MIXED_RANKS = [16, 8, 64, 32, 5]


def test_mixed_bf16_ragged():
    """Several row tiles with a ragged tail, K not a multiple of 64, N not of 256, mixed
    ranks (one of them not a multiple of 8), decode singles among prefill and two
    training segments on two adapters; rank padding is NaN."""
    w = wl.custom(MIXED, MIXED_RANKS, K=520, N=776, r_max=64, name="mixed_ragged")
    _full(w)


WIDE = [(0, 70, 1, 0), (70, 300, 2, 1), (370, 3, 0, 0), (373, 45, 2, 1), (418, 290, 0, 1), (708, 1, 1, 0)]


@pytest.mark.parametrize("train_rank", [32, 64])
def test_wide_training_ranks(train_rank):
    """A training adapter of rank 32 or 64 (the token reductions then run two or
    four 16-rank tiles) beside one of rank 16, with training segments of 300, 45
    and 290 tokens (several 256-token chunks, ragged against the 32-token steps)
    and inference rows between them: Y, H_save, dA, dB and dX against the oracle."""
    w = wl.custom(WIDE, [16, 8, train_rank], K=520, N=776, r_max=64, name="wide_rank%d" % train_rank)
    _full(w)


SPLIT = ([(0, 180, 1, 0)] + [(180 + i, 1, 2 + i % 3, 0) for i in range(20)] +
         [(200, 300, 0, 1), (500, 200, 3, 0)])
SPLIT_RANKS = [16, 8, 32, 64, 5]


def test_split_tiles_ragged():
    """256 x 256 tiles whose last partial wave is split along the contraction, in both
    GEMMs: ragged rows (T = 700, T_t = 300), columns (N = 2000) and contraction (the dX
    GEMM's 2000 = 31 * 64 + 16), decode singles on the gathered path inside split tiles.
    Y and dX on sampled rows, H_save, dA and dB in full; a repeat is bit-identical."""
    import torch
    from paper_2607_28848_amd import dsv
    w = wl.custom(SPLIT, SPLIT_RANKS, K=4096, N=2000, r_max=64, name="split_ragged")
    run = Run(w, pad=np.nan)
    fc = dsv.gemm_config(run.plan, dsv.BF16, 4096, 2000, 0)
    bc = dsv.gemm_config(run.plan, dsv.BF16, 4096, 2000, 1)
    _say("  gemm configs: fwd %s dX %s" % (fc, bc))
    if fc["split_tiles"] == 0 or bc["split_tiles"] == 0:
        pytest.skip("this device's compute-unit count gives no split for these shapes")
    assert run.plan.counts()["gathered_rows"] >= 20
    Y, H = run.fwd()
    dA, dB, dX = run.bwd(H)
    Y2, _ = run.fwd()
    _, _, dX2 = run.bwd(H)
    torch.cuda.synchronize()
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))
    assert torch.equal(dX.view(torch.int16), dX2.view(torch.int16))
    rows = np.unique(np.concatenate([np.arange(0, 700, 7), [179, 180, 199, 200, 499, 500, 699]]))
    dx_rows = np.unique(np.concatenate([np.arange(0, 300, 5), [255, 256, 299]]))
    _check_all(w, run, Y, H, dA, dB, dX, TOL_BF16, rows=rows.astype(np.int32),
               dx_rows=dx_rows.astype(np.int32))


@pytest.mark.parametrize("dtype,K,N,r_max", [("bf16", 520, 776, 64), ("f32", 520, 776, 64), ("bf16", 4096, 4096, 64),
                                             ("bf16", 4104, 2056, 64), ("bf16", 4104, 2056, 16),
                                             ("bf16", 520, 776, 16), ("bf16", 520, 776, 12)])
def test_residual_only_retention_recomputes_h_bit_exact(dtype, K, N, r_max):
    """A forward that keeps no H_save (the caller keeps X) and a backward that
    recomputes h from X and A give bit-identical Y, dA, dB and dX to keeping H_save
    (the recompute is the forward's own shrink over the training rows; at K = 4096 both
    split the contraction into chunks).  r_max = 16 runs the rank-16 shrink, whose
    chunks load three buffers deep.  r_max = 12 gives the kept H_save rows of 24
    bytes: the dB reduction then reads h element by element (the two-buffer token
    reduction), while the recomputed h (rows of 16 entries) goes through the
    pipelined one that stages h in LDS; both sum in the same order."""
    import torch
    ranks = MIXED_RANKS if r_max == 64 else [min(x, r_max) for x in (16, 8, 16, 12, 5)]
    w = wl.custom(MIXED, ranks, K=K, N=N, dtype=dtype, r_max=r_max, name="recompute")
    run = Run(w)
    Y1, H = run.fwd()
    dA1, dB1, dX1 = run.bwd(H)
    Y2, H2 = run.dsv.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, keep_h=False)
    assert H2 is None
    dA2, dB2, dX2 = run.bwd(None)
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)  # noqa: E731
    for a, b in ((Y1, Y2), (dA1, dA2), (dB1, dB2), (dX1, dX2)):
        assert torch.equal(bits(a), bits(b))


@pytest.mark.parametrize("K,N", [(4096, 4096), (4104, 2056)])
def test_split_contraction_rank_kernels(K, N):
    """Contractions of 8+ chunks of 256 columns: the shrink (over K) and g (over N)
    split them into pieces (K = 4096: 2 of 8 chunks; K = 4104: 3 pieces of 6, 6 and 5
    chunks, the last one 8 columns wide; N = 2056: 5 + 4 chunks) whose fp32 sums a
    second kernel adds in order; Y and dX on sampled rows, H_save, dA and dB in full."""
    ranks = [16, 8, 16, 12, 5]
    w = wl.custom(MIXED, ranks, K=K, N=N, r_max=16, name="split_rank")
    run = Run(w, pad=np.nan)
    Y, H = run.fwd()
    dA, dB, dX = run.bwd(H)
    import torch
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, w.n_tokens, 9), [99, 100, 101, 102, 401, 402, 704]]))
    dx_rows = np.unique(np.concatenate([np.arange(0, run.plan.train_tokens, 7), [299, 300, 428]]))
    _check_all(w, run, Y, H, dA, dB, dX, TOL_BF16, rows=rows.astype(np.int32), dx_rows=dx_rows.astype(np.int32))


def test_mixed_f32_ragged():
    w = wl.custom(MIXED, MIXED_RANKS, K=136, N=200, dtype="f32", r_max=64, name="mixed_f32")
    _full(w, tol=TOL_F32)


def test_decode_heavy_small():
    rng = np.random.default_rng(5)
    pieces = [(1, int(a), 0) for a in rng.integers(0, 16, size=300)] + [(200, 1, 1)]
    order = rng.permutation(len(pieces))
    segs, s = [], 0
    for i in order:
        l, a, t = pieces[i]
        segs.append((s, l, a, t))
        s += l
    ranks = [(8, 16, 32, 64)[a % 4] for a in range(16)]
    w = wl.custom(segs, ranks, K=256, N=512, r_max=64, name="decode_small")
    run, _ = _full(w)
    assert run.plan.counts()["gathered_rows"] >= 290


def test_inference_only_and_training_only():
    w = wl.custom([(0, 300, 0, 0), (300, 33, 1, 0)], [8, 16], K=128, N=264, r_max=16, name="inf_only")
    run = Run(w)
    Y, H = run.fwd()
    assert H is None and run.plan.train_tokens == 0
    dA, dB, dX = run.bwd(None)                   # no training rows: a no-op
    Yr, _ = oracle_fwd(w, run.t)
    assert oracle.rel_err(to_host(Y), Yr) <= TOL_BF16
    assert (to_host(dA) == 0).all() and (to_host(dB) == 0).all() and dX is None
    w2 = wl.custom([(0, 70, 1, 1), (70, 200, 0, 1)], [8, 16], K=128, N=264, r_max=16, name="train_only")
    _full(w2)


def test_empty_batch():
    import torch
    from paper_2607_28848_amd import dsv
    plan = dsv.segments_build([], 0, [4], [2.0], 4, device="cuda")
    X = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((32, 64), dtype=torch.bfloat16, device="cuda")
    A = torch.zeros((1, 4, 64), dtype=torch.bfloat16, device="cuda")
    B = torch.zeros((1, 32, 4), dtype=torch.bfloat16, device="cuda")
    Y, H = dsv.cobatch_fwd(plan, X, W, A, B)
    assert Y.shape == (0, 32) and H is None


def test_zero_B_is_exactly_base():
    """B = 0: the low-rank term enters the fp32 accumulator as an exact zero, so Y is
    bit-identical however the rows are grouped (tile groups or gathered path)."""
    import torch
    w1 = wl.custom(MIXED, MIXED_RANKS, K=520, N=776, r_max=64, name="zeroB")
    run1 = Run(w1)
    run1.B.zero_()
    Y1, _ = run1.fwd()
    # same tokens, every row its own single-token segment on a rotating adapter
    segs = [(t, 1, t % 5, 0) for t in range(w1.n_tokens)]
    w2 = wl.custom(segs, MIXED_RANKS, K=520, N=776, r_max=64, name="zeroB_singles")
    run2 = Run(w2, tensors=run1.t)
    run2.B.zero_()
    Y2, _ = run2.fwd()
    torch.cuda.synchronize()
    assert run2.plan.counts()["gathered_rows"] == w2.n_tokens
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    t = run1.t
    assert oracle.rel_err(to_host(Y1), t.X @ t.W.T) <= TOL_BF16


def test_table_permutation_bit_exact_and_deterministic():
    import torch
    w = wl.custom(MIXED, MIXED_RANKS, K=520, N=776, r_max=64, name="perm")
    run = Run(w)
    Tt = run.plan.train_tokens
    nan_h = lambda: torch.full((Tt, 64), float("nan"), dtype=torch.bfloat16, device="cuda")  # noqa: E731
    Y, H = run.fwd(H_save=nan_h())   # rank padding of H_save is never written: same sentinel
    dA, dB, dX = run.bwd(H)
    rng = np.random.default_rng(3)
    perm = [MIXED[i] for i in rng.permutation(len(MIXED))]
    w2 = wl.custom(perm, MIXED_RANKS, K=520, N=776, r_max=64, name="perm2")
    run2 = Run(w2, tensors=run.t)
    for _ in range(2):  # permuted table, then a repeat of it
        Y2, H2 = run2.fwd(H_save=nan_h())
        dA2, dB2, dX2 = run2.bwd(H2)
        torch.cuda.synchronize()
        for name, u, v in (("Y", Y, Y2), ("H_save", H, H2), ("dX", dX, dX2)):
            assert torch.equal(u.view(torch.int16), v.view(torch.int16)), name
        for name, u, v in (("dA", dA, dA2), ("dB", dB, dB2)):
            assert torch.equal(u.view(torch.int32), v.view(torch.int32)), name


def test_accumulate_and_untouched_slices():
    """accumulate=1 adds to the training adapters' slices; other adapters' slices and
    the rank padding of every slice keep their sentinel bits; H_save padding columns
    are never written."""
    import torch
    w = wl.custom(MIXED, MIXED_RANKS, K=520, N=776, r_max=64, name="accum")
    run = Run(w)
    Tt = run.plan.train_tokens
    H = torch.full((Tt, 64), float("nan"), dtype=torch.bfloat16, device="cuda")
    Y, H = run.fwd(H_save=H)
    dA0 = torch.randn((5, 64, 520), device="cuda")
    dB0 = torch.randn((5, 776, 64), device="cuda")
    dA, dB = dA0.clone(), dB0.clone()
    run.bwd(H, dA=dA, dB=dB, accumulate=True)
    torch.cuda.synchronize()
    Hh = to_host(H)
    ra = np.array([w.ranks[a] for a in oracle.rows(w.segments, w.n_tokens, 5)[0][run.plan.train_rows()]])
    for i, r in enumerate(ra):
        assert np.isnan(Hh[i, r:]).all() and np.isfinite(Hh[i, :r]).all()
    G, dAr, dBr, _ = oracle_bwd(w, run.t)
    dA_h, dB_h, dA0_h, dB0_h = (x.cpu().numpy().astype(np.float64) for x in (dA, dB, dA0, dB0))
    owners = dict(train_mask_slices(w))
    for a in range(5):
        r = int(w.ranks[a])
        if a in owners:
            assert oracle.rel_err(dA_h[a, :r] - dA0_h[a, :r], dAr[a, :r]) <= TOL_BF16
            assert oracle.rel_err(dB_h[a, :, :r] - dB0_h[a, :, :r], dBr[a, :, :r]) <= TOL_BF16
            assert (dA_h[a, r:] == dA0_h[a, r:]).all() and (dB_h[a, :, r:] == dB0_h[a, :, r:]).all()
        else:
            assert (dA_h[a] == dA0_h[a]).all() and (dB_h[a] == dB0_h[a]).all()


def _sampled(w, p, n_rows=24, seed=0):
    """Full-size projection: every output of the HIP path against the reference on
    sampled rows (Y, dX) and in full (H_save, dA, dB); a one-projection workload also
    through the grouped call the bench times (dX on the transposed weight), bit for bit."""
    import torch
    K, N = w.projections[p].K, w.projections[p].N
    _say("case %s/%s T=%d Tt=%d K=%d N=%d" % (w.name, w.projections[p].name, w.n_tokens,
                                             w.train_tokens, K, N))
    run = Run(w, p=p, pad=np.nan)
    Y, H = run.fwd()
    dA, dB, dX = run.bwd(H)
    torch.cuda.synchronize()
    rng = np.random.default_rng(seed + p)
    # segment boundaries and random rows
    firsts = [s for (s, l, _, _) in w.segments if l] + [s + l - 1 for (s, l, _, _) in w.segments if l]
    rows = np.unique(np.concatenate([rng.choice(w.n_tokens, n_rows, replace=False),
                                     rng.choice(firsts, min(n_rows, len(firsts)), replace=False)]))
    Tt = w.train_tokens
    if len(w.projections) == 1 and Tt:
        # the bench's launch of a one-projection workload: a group of one whose dX
        # GEMM reads the transposed weight; same sums, so bit-identical results
        Wt = run.W.t().contiguous()
        (Yg, Hg), = run.dsv.cobatch_fwd_grouped(run.plan, [(run.X, run.W, run.A, run.B)])
        (dAg, dBg, dXg), = run.dsv.lora_bwd_grouped(run.plan, [(run.X, run.W, run.A, run.B, Hg, run.dY)],
                                                    wts=[Wt])
        torch.cuda.synchronize()
        bits = lambda t: t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)  # noqa: E731
        for a, b in ((Y, Yg), (dX, dXg), (dA, dAg), (dB, dBg)):
            assert torch.equal(bits(a), bits(b))
        r_t = min(r for _, r in train_mask_slices(w))  # columns every H_save row holds
        assert torch.equal(bits(H[:, :r_t]), bits(Hg[:, :r_t]))
        del Wt, Yg, Hg, dAg, dBg, dXg
    dx_rows = np.unique(np.concatenate([rng.choice(Tt, n_rows, replace=False), [0, Tt - 1]])) if Tt else None
    return _check_all(w, run, Y, H, dA, dB, dX, TOL_BF16, rows=rows.astype(np.int32),
                      dx_rows=None if dx_rows is None else dx_rows.astype(np.int32))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("p", range(7))
def test_llama8b_layer_set_full_size(p):
    """Llama-3-8B layer set (q, k, v, o, gate, up, down) at full size, bf16."""
    _sampled(wl.llama8b_mixed(), p)


@pytest.mark.timeout(600)
def test_decode_heavy_full_size():
    """256 single-token decode segments over 64 adapters of ranks 8..64 + 2048 training
    tokens on the 4096 x 14336 gate projection."""
    w = wl.decode_heavy()
    _sampled(w, 0)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("p", range(2))
def test_llama70b_full_size(p):
    _sampled(wl.llama70b(), p, n_rows=12)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("frac", [0.0, 0.25, 0.5, 0.75, 1.0])
def test_load_sweep_full_size(frac):
    """Load sweep on the 4096 x 14336 layer: 16384 tokens, training fraction 0 .. 1."""
    _sampled(wl.load_sweep(frac), 0, n_rows=12)


def test_gemm_launch_timing():
    """dsv_timing_*: the events ride the GEMM launches' dispatches, one pair per launch
    (forward, dX: a split-tile launch is timed from its tile kernel to its fixup), with
    positive durations; a backward without training rows launches no GEMM and adds no pair."""
    import torch
    from paper_2607_28848_amd import dsv
    w = wl.custom(MIXED, [16, 8, 16, 12, 5], K=4096, N=4104, r_max=16, name="timing")
    run = Run(w, pad=np.nan)
    fc = dsv.gemm_config(run.plan, dsv.BF16, 4096, 4104, 0)
    bc = dsv.gemm_config(run.plan, dsv.BF16, 4096, 4104, 1)
    _say("  gemm configs: fwd %s dX %s" % (fc, bc))
    torch.cuda.synchronize()
    dsv.timing_read()  # discard anything recorded before
    dsv.timing_enable(True)
    try:
        Y, H = run.fwd()
        dA, dB, dX = run.bwd(H)
        inf = dsv.segments_build([(s, l, a, 0) for (s, l, a, _) in w.segments], w.n_tokens, w.ranks, w.scales,
                                 w.r_max, device="cuda")
        dsv.lora_bwd(inf, run.X, run.W, run.A, run.B, None, run.dY[:1])
        torch.cuda.synchronize()
    finally:
        dsv.timing_enable(False)
    fwd_ms, fwd_n, bwd_ms, bwd_n = dsv.timing_read()
    assert (fwd_n, bwd_n) == (1, 1)
    assert 0.0 < fwd_ms < 1e3 and 0.0 < bwd_ms < 1e3
    assert dsv.timing_read()[1] == 0  # a read resets the pairs
