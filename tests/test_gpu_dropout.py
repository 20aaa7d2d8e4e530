"""GPU parity of LoRA dropout on the training rows (Sec. 4.1 fine-tunes with
dropout 0.05): dsv_cobatch_fwd_dropout / dsv_lora_bwd_dropout against the fp64
reference fed the same Philox4x32-10 mask (the reference draws it from the
generator's published definition; the HIP path regenerates it on the device).

Bar: the mask itself bit-exact; Y, H_save, dA, dB and dX within 2e-2 (bf16) or
1e-5 (fp32) of the reference; p = 0 and residual-only retention bit-identical to
the plain path and to kept H_save.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_28848_amd import workloads as wl
from gpu_util import (TOL_BF16, TOL_F32, Run, oracle_bwd, oracle_fwd, to_dev, to_host,
                      train_mask_slices)

pytestmark = pytest.mark.gpu

MIXED = [(0, 100, 3, 0), (100, 1, 1, 0), (101, 1, 2, 0), (102, 300, 0, 1), (402, 1, 3, 0),
         (403, 57, 2, 0), (460, 2, 1, 0), (462, 129, 1, 1), (591, 3, 0, 0), (594, 111, 4, 0)]
MIXED_RANKS = [16, 8, 64, 32, 5]
SEED = 0x0123456789ABCDEF
OFFSET = (7 << 32) | 3


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bits(t):
    import torch
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _check(w, run, drop, Y, H, dA, dB, dX, tol, rows=None, dx_rows=None):
    t = run.t
    Yr, _ = oracle_fwd(w, t, rows, drop=drop)
    Yg = to_host(Y) if rows is None else to_host(Y)[rows]
    errs = {"Y": oracle.rel_err(Yg, Yr)}
    tr = run.plan.train_rows()
    errs["H_save"] = oracle.rel_err(to_host(H), oracle_fwd(w, t, tr, drop=drop)[1])
    _, dAr, dBr, dXr = oracle_bwd(w, t, dx_rows=dx_rows, drop=drop)
    dAg, dBg = to_host(dA), to_host(dB)
    for a, r in train_mask_slices(w):
        errs["dA%d" % a] = oracle.rel_err(dAg[a, :r], dAr[a, :r])
        errs["dB%d" % a] = oracle.rel_err(dBg[a, :, :r], dBr[a, :, :r])
    dXg = to_host(dX) if dx_rows is None else to_host(dX)[dx_rows]
    errs["dX"] = oracle.rel_err(dXg, dXr)
    _say("  rel errors: " + ", ".join("%s=%.2e" % kv for kv in errs.items()))
    for k, v in errs.items():
        assert v <= tol, (k, v)


@pytest.mark.parametrize("dtype,p", [("bf16", 0.05), ("bf16", 0.3), ("f32", 0.05), ("f32", 0.3)])
def test_dropout_parity_mixed_ragged(dtype, p):
    """Mixed batch (K = 520: the mask's last word is partial; N = 776; ranks 16, 8,
    64, 32, 5; two training segments on two adapters), every output against the
    reference under the same mask."""
    import torch
    _say("case dropout %s p=%.2f" % (dtype, p))
    w = wl.custom(MIXED, MIXED_RANKS, K=520, N=776, dtype=dtype, r_max=64, name="dropout")
    run = Run(w)
    d = (p, SEED, OFFSET)
    Y, H = run.dsv.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, dropout=d)
    dA, dB, dX = run.dsv.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H, run.dY, dropout=d)
    torch.cuda.synchronize()
    drop = oracle.dropout_multipliers(w.train_tokens, 520, p, SEED, OFFSET)
    _check(w, run, drop, Y, H, dA, dB, dX, TOL_BF16 if dtype == "bf16" else TOL_F32)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_dropout_mask_bit_exact(dtype):
    """With W = 0 and A, B, dY positive, dX = mask * (g A) / (1 - p) is zero exactly
    where an element is dropped: its zero pattern is the device's mask, compared bit
    for bit with the generator's; a different offset draws a different mask."""
    import torch
    _say("case dropout mask %s" % dtype)
    K, N, p = 520, 136, 0.3
    w = wl.custom(MIXED, MIXED_RANKS, K=K, N=N, dtype=dtype, r_max=64, name="dropout_mask")
    t = w.tensors(0)
    run = Run(w, tensors=t)
    run.W = torch.zeros_like(run.W)
    run.A = to_dev(np.abs(t.A), dtype)
    run.B = to_dev(np.abs(t.B), dtype)
    run.dY = to_dev(np.abs(t.dY), dtype)
    Tt = w.train_tokens
    for off in (OFFSET, OFFSET + 1):
        _, _, dX = run.dsv.lora_bwd(run.plan, run.X, run.W, run.A, run.B, None, run.dY,
                                    dropout=(p, SEED, off))
        torch.cuda.synchronize()
        got = to_host(dX) != 0.0
        ref = oracle.dropout_keep(Tt, K, p, SEED, off)
        assert got.shape == ref.shape
        assert np.array_equal(got, ref), int((got != ref).sum())
        frac = 1.0 - ref.mean()
        _say("  offset %d: dropped fraction %.4f" % (off, frac))
        assert abs(frac - p) < 0.02


@pytest.mark.parametrize("dtype,K,N", [("bf16", 520, 776), ("f32", 520, 776), ("bf16", 4096, 4096)])
def test_dropout_p0_retention_and_repeat_bit_exact(dtype, K, N):
    """p = 0 gives the plain entry points' results bit for bit; under p = 0.05 a
    forward that keeps no H_save and a backward that recomputes h through the
    regenerated mask match keeping H_save bit for bit, and a repeat is identical."""
    import torch
    _say("case dropout bit-exact %s K=%d N=%d" % (dtype, K, N))
    w = wl.custom(MIXED, MIXED_RANKS, K=K, N=N, dtype=dtype, r_max=64, name="dropout_bits")
    run = Run(w)
    ds = run.dsv

    def hbuf():  # H_save with its rank padding cleared (the path never writes it)
        return torch.zeros((run.plan.train_tokens, w.r_max), dtype=run.X.dtype, device=run.X.device)

    Y0, H0 = ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, H_save=hbuf())
    g0 = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H0, run.dY)
    Yz, Hz = ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, H_save=hbuf(), dropout=(0.0, SEED, OFFSET))
    gz = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, Hz, run.dY, dropout=(0.0, SEED, OFFSET))
    d = (0.05, SEED, OFFSET)
    Y1, H1 = ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, H_save=hbuf(), dropout=d)
    g1 = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H1, run.dY, dropout=d)
    Y2, H2 = ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, keep_h=False, dropout=d)
    assert H2 is None
    g2 = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, None, run.dY, dropout=d)
    Y3, H3 = ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, H_save=hbuf(), dropout=d)
    g3 = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H3, run.dY, dropout=d)
    torch.cuda.synchronize()
    for a, b in [(Y0, Yz), (H0, Hz)] + list(zip(g0, gz)):
        assert torch.equal(_bits(a), _bits(b))
    for a, b in [(Y1, Y2), (Y1, Y3), (H1, H3)] + list(zip(g1, g2)) + list(zip(g1, g3)):
        assert torch.equal(_bits(a), _bits(b))
    assert not torch.equal(_bits(Y0), _bits(Y1))  # the mask does change the training rows


SPLIT = ([(0, 180, 1, 0)] + [(180 + i, 1, 2 + i % 3, 0) for i in range(20)] +
         [(200, 300, 0, 1), (500, 200, 3, 0)])
SPLIT_RANKS = [16, 8, 32, 64, 5]


def test_dropout_split_tiles_ragged():
    """Dropout through 256 x 256 tiles split along the contraction (the dX GEMM adds
    the masked low-rank term in the kernel that sums the pieces): T = 700, T_t = 300,
    K = 4096, N = 2000; Y and dX on sampled rows, H_save, dA and dB in full."""
    import torch
    _say("case dropout split tiles")
    w = wl.custom(SPLIT, SPLIT_RANKS, K=4096, N=2000, r_max=64, name="dropout_split")
    run = Run(w)
    bc = run.dsv.gemm_config(run.plan, run.dsv.BF16, 4096, 2000, 1)
    _say("  dX gemm config %s" % bc)
    d = (0.05, SEED, OFFSET)
    Y, H = run.dsv.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, dropout=d)
    dA, dB, dX = run.dsv.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H, run.dY, dropout=d)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, 700, 7), [179, 180, 199, 200, 499, 500, 699]]))
    dx_rows = np.unique(np.concatenate([np.arange(0, 300, 5), [255, 256, 299]]))
    drop = oracle.dropout_multipliers(w.train_tokens, 4096, 0.05, SEED, OFFSET)
    _check(w, run, drop, Y, H, dA, dB, dX, TOL_BF16, rows=rows.astype(np.int32),
           dx_rows=dx_rows.astype(np.int32))


@pytest.mark.timeout(600)
def test_dropout_llama8b_full_size():
    """The Llama-3-8B q projection (K = N = 4096) of the mixed batch (6144 rows: 4096
    inference + 2048 training) with dropout 0.05 on its training rows: Y and dX on
    sampled rows, H_save, dA, dB in full."""
    import torch
    w = wl.llama8b_mixed()
    K = w.projections[0].K
    _say("case dropout %s/%s" % (w.name, w.projections[0].name))
    run = Run(w, p=0)
    d = (0.05, SEED, OFFSET)
    Y, H = run.dsv.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, dropout=d)
    dA, dB, dX = run.dsv.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H, run.dY, dropout=d)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    tr = run.plan.train_rows()
    rows = np.unique(np.concatenate([rng.choice(w.n_tokens, 16, replace=False), tr[:2], tr[-2:]]))
    Tt = w.train_tokens
    dx_rows = np.unique(np.concatenate([rng.choice(Tt, 16, replace=False), [0, Tt - 1]]))
    drop = oracle.dropout_multipliers(Tt, K, 0.05, SEED, OFFSET)
    _check(w, run, drop, Y, H, dA, dB, dX, TOL_BF16, rows=rows.astype(np.int32),
           dx_rows=dx_rows.astype(np.int32))


def _unpack(buf, Tt, K):
    """[Tt * ceil(K/32)] mask words -> [Tt][K] keep flags (bit b of word w: column 32 w + b)."""
    wds = buf.cpu().numpy().view(np.uint32).reshape(Tt, (K + 31) // 32)
    bits = (wds[:, :, None] >> np.arange(32, dtype=np.uint32)[None, None, :]) & 1
    return bits.reshape(Tt, -1)[:, :K].astype(bool)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_dropout_mask_buffer_single(dtype):
    """dsv_dropout.mask: the forward draws the generator's mask into the caller's
    buffer (bit-exact against the reference generator) and its results do not
    change; a backward given the buffer matches the one that redraws bit for bit;
    a backward given a buffer drawn at another offset computes that offset's
    gradients (it reads the buffer, it does not redraw)."""
    import torch
    _say("case dropout mask buffer %s" % dtype)
    K, N, p = 520, 776, 0.05
    w = wl.custom(MIXED, MIXED_RANKS, K=K, N=N, dtype=dtype, r_max=64, name="dropout_buf")
    run = Run(w)
    ds = run.dsv
    Tt = w.train_tokens
    nw = ds.dropout_mask_words(run.plan, K)
    buf = torch.zeros(nw, dtype=torch.int32, device="cuda")
    other = torch.zeros(nw, dtype=torch.int32, device="cuda")
    d = (p, SEED, OFFSET)

    def hbuf():  # H_save with its rank padding cleared (the path never writes it)
        return torch.zeros((Tt, w.r_max), dtype=run.X.dtype, device=run.X.device)

    Y0, H0 = ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, H_save=hbuf(), dropout=d)
    Y1, H1 = ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, H_save=hbuf(), dropout=d + (buf,))
    ds.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, H_save=hbuf(), dropout=(p, SEED, OFFSET + 1, other))
    g0 = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H0, run.dY, dropout=d)
    g1 = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, H0, run.dY, dropout=d + (buf,))
    g2 = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, None, run.dY, dropout=d + (buf,))
    g0b = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, None, run.dY, dropout=d)
    # the offset's mask through the buffer, against the redrawn one of that offset
    g_o = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, None, run.dY, dropout=(p, SEED, OFFSET, other))
    g_r = ds.lora_bwd(run.plan, run.X, run.W, run.A, run.B, None, run.dY, dropout=(p, SEED, OFFSET + 1))
    torch.cuda.synchronize()
    assert np.array_equal(_unpack(buf, Tt, K), oracle.dropout_keep(Tt, K, p, SEED, OFFSET))
    assert np.array_equal(_unpack(other, Tt, K), oracle.dropout_keep(Tt, K, p, SEED, OFFSET + 1))
    for a, b in [(Y0, Y1), (H0, H1)] + list(zip(g0, g1)) + list(zip(g0b, g2)) + list(zip(g_o, g_r)):
        assert torch.equal(_bits(a), _bits(b))
    assert not torch.equal(_bits(g_o[2]), _bits(g0b[2]))


def test_dropout_mask_buffer_grouped():
    """The grouped calls with per-projection mask buffers (one projection given a
    buffer in the backward, the other redrawn): every output bit-identical to the
    grouped calls without buffers, and each buffer the generator's mask."""
    import torch
    from paper_2607_28848_amd import dsv
    _say("case dropout mask buffer grouped")
    shapes = [(520, 776), (136, 264)]
    runs = [Run(wl.custom(MIXED, MIXED_RANKS, K=K, N=N, dtype="bf16", r_max=64, name="dbg%d" % i))
            for i, (K, N) in enumerate(shapes)]
    plan = runs[0].plan
    Tt = runs[0].w.train_tokens
    bufs = [torch.zeros(dsv.dropout_mask_words(plan, K), dtype=torch.int32, device="cuda") for K, _ in shapes]
    drops = [(0.05, SEED + i, OFFSET) for i in range(2)]
    def outs():  # Y and H_save, H_save's rank padding cleared (the path never writes it)
        return [(r.X, r.W, r.A, r.B, torch.empty((r.w.n_tokens, N), dtype=r.X.dtype, device="cuda"),
                 torch.zeros((Tt, r.w.r_max), dtype=r.X.dtype, device="cuda")) for r, (_, N) in zip(runs, shapes)]

    out0 = dsv.cobatch_fwd_grouped(plan, outs(), dropouts=drops)
    out1 = dsv.cobatch_fwd_grouped(plan, outs(), dropouts=[d + (b,) for d, b in zip(drops, bufs)])
    bwd_in = [(r.X, r.W, r.A, r.B, o[1], r.dY) for r, o in zip(runs, out0)]
    gb0 = dsv.lora_bwd_grouped(plan, bwd_in, dropouts=drops)
    gb1 = dsv.lora_bwd_grouped(plan, bwd_in, dropouts=[drops[0] + (bufs[0],), drops[1]])
    torch.cuda.synchronize()
    for (K, _), b, d in zip(shapes, bufs, drops):
        assert np.array_equal(_unpack(b, Tt, K), oracle.dropout_keep(Tt, K, 0.05, d[1], OFFSET))
    for o0, o1 in zip(out0, out1):
        for a, b in zip(o0, o1):
            assert torch.equal(_bits(a), _bits(b))
    for x0, x1 in zip(gb0, gb1):
        for a, b in zip(x0, x1):
            assert torch.equal(_bits(a), _bits(b))


@pytest.mark.parametrize("K,N", [(520, 776), (4096, 2000)])
def test_dropout_dx_transposed_weight_bit_exact(K, N):
    """Under dropout the dX GEMM on the transposed weight (NT) and on W itself (NN)
    give bit-identical dX, dA and dB (single and grouped calls)."""
    import torch
    from paper_2607_28848_amd import dsv
    _say("case dropout Wt K=%d N=%d" % (K, N))
    w = wl.custom(SPLIT if K == 4096 else MIXED, SPLIT_RANKS if K == 4096 else MIXED_RANKS, K=K, N=N,
                  r_max=64, name="dropout_wt")
    run = Run(w)
    d = (0.05, SEED, OFFSET)
    Y, H = run.dsv.cobatch_fwd(run.plan, run.X, run.W, run.A, run.B, dropout=d)
    Wt = run.W.t().contiguous()
    args = [(run.X, run.W, run.A, run.B, H, run.dY)]
    g_nn = dsv.lora_bwd_grouped(run.plan, args + args, dropouts=[d, d])
    g_nt = dsv.lora_bwd_grouped(run.plan, args + args, dropouts=[d, d], wts=[Wt, Wt])
    torch.cuda.synchronize()
    for a, b in zip(g_nn, g_nt):
        for x, y in zip(a, b):
            assert torch.equal(_bits(x), _bits(y))
