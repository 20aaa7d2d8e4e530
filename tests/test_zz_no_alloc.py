"""GPU test of the allocation-free forward (dsv_cobatch_fwd_noalloc): its output
against dsv_cobatch_fwd's on the same inputs, through the C ABI, on two calls in a
row (the second with a smaller batch, so it runs over what the first left in the
scratch), then an fp32 call, and a batch whose intermediates exceed the scratch
(rejected before any launch, nothing written).

Bar: H_save bit-identical; Y bit-identical where dsv_cobatch_fwd splits no GEMM
tile along the contraction, else within 2e-2 of it (max abs difference over max
abs value)."""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_28848_amd import workloads as wl
from gpu_util import TOL_BF16, to_dev, to_host

pytestmark = pytest.mark.gpu

MIXED = [(0, 100, 3, 0), (100, 1, 1, 0), (101, 1, 2, 0), (102, 300, 0, 1), (402, 1, 3, 0),
         (403, 57, 2, 0), (460, 2, 1, 0), (462, 129, 1, 1), (591, 3, 0, 0), (594, 111, 4, 0)]
SMALL = [(0, 40, 1, 0), (40, 1, 0, 0), (41, 1, 2, 0), (42, 90, 0, 1), (132, 3, 2, 0), (135, 70, 2, 1)]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bits(t):
    import torch
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _case(segs, ranks, K, N, r_max, dtype, name):
    """Both forwards of one batch; returns nothing, asserts the bar."""
    import torch
    from paper_2607_28848_amd import dsv
    _say("case %s: %s K=%d N=%d r_max=%d" % (name, dtype, K, N, r_max))
    w = wl.custom(segs, ranks, K=K, N=N, dtype=dtype, r_max=r_max, name=name)
    t = w.tensors(0, pad=np.nan)
    X, W, A, B = (to_dev(t.store[k], dtype) for k in ("X", "W", "A", "B"))
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    Tt = plan.train_tokens
    Y0, H0 = dsv.cobatch_fwd(plan, X, W, A, B)
    Y1 = torch.full_like(Y0, float("nan"))
    H1 = torch.full_like(H0, float("nan")) if H0 is not None else None
    dsv.cobatch_fwd_noalloc(plan, X, W, A, B, Y1, H1)
    torch.cuda.synchronize()
    if Tt:
        r_t = min(int(w.ranks[a]) for (_, l, a, tr) in w.segments if tr and l)
        assert torch.equal(_bits(H0[:, :r_t]), _bits(H1[:, :r_t]))
    split = dsv.gemm_config(plan, dsv.BF16, K, N, 0)["split_tiles"] if dtype == "bf16" else 0
    if split == 0:
        assert torch.equal(_bits(Y0), _bits(Y1))
        _say("  Y and H_save bit-identical")
    else:
        err = oracle.rel_err(to_host(Y1), to_host(Y0))
        _say("  dsv_cobatch_fwd splits %d tiles; Y rel diff %.2e" % (split, err))
        assert err <= TOL_BF16


def test_noalloc_forward_matches_cobatch_fwd_two_calls():
    """A mixed batch (prefill, decode rows on the gathered path, training rows, ranks
    5..64), then a smaller batch over the scratch the first one left, then fp32."""
    _case(MIXED, [16, 8, 64, 32, 5], K=2056, N=1544, r_max=64, dtype="bf16", name="mixed")
    _case(SMALL, [16, 8, 32], K=264, N=328, r_max=32, dtype="bf16", name="smaller")
    _case(SMALL, [16, 8, 32], K=136, N=200, r_max=32, dtype="f32", name="fp32")


def test_noalloc_forward_large_gemm_split_case():
    """A 6144 x 4096 x 14336 forward (the Llama-3-8B gate projection of the mixed
    batch), where dsv_cobatch_fwd may split the last partial wave of tiles: the
    allocation-free form takes whole tiles instead."""
    w = wl.llama8b_mixed()
    _case(w.segments, list(w.ranks), K=4096, N=14336, r_max=w.r_max, dtype="bf16", name="llama8b gate")


def test_noalloc_forward_rejects_oversized_batch():
    """h of 600000 rows at rank stride 64 (76.8 MB) does not fit the 64 MiB scratch:
    DSV_ERR_SIZE before any launch, the output untouched."""
    import torch
    from paper_2607_28848_amd import dsv
    T, K, N, r = 600000, 8, 8, 64
    plan = dsv.segments_build([(0, T, 0, 0)], T, [r], [1.0], r, device="cuda")
    X = torch.zeros((T, K), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((N, K), dtype=torch.bfloat16, device="cuda")
    A = torch.zeros((1, r, K), dtype=torch.bfloat16, device="cuda")
    B = torch.zeros((1, N, r), dtype=torch.bfloat16, device="cuda")
    Y = torch.full((T, N), 3.0, dtype=torch.bfloat16, device="cuda")
    assert dsv.fwd_workspace_bytes(plan, dsv.BF16, K, N) > dsv.NOALLOC_SCRATCH_BYTES
    with pytest.raises(dsv.DsvError) as ei:
        dsv.cobatch_fwd_noalloc(plan, X, W, A, B, Y)
    assert ei.value.status == dsv.ERR_SIZE
    torch.cuda.synchronize()
    assert bool((Y == 3.0).all())
