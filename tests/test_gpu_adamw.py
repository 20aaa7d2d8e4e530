"""GPU parity of the fused AdamW step of the training adapters (dsv_adamw_step)
against the fp64 reference: fp32 masters and moments within 1e-5 (max abs error /
max abs reference, per tensor), the parameter copy exactly the rounded master, and
every other adapter and every rank-padding entry untouched (bit-exact)."""
import numpy as np
import pytest

import oracle
from gpu_util import TOL_F32, Run
from paper_2607_28848_amd import workloads as wl

pytestmark = pytest.mark.gpu

MIXED = [(0, 100, 3, 0), (100, 1, 1, 0), (101, 1, 2, 0), (102, 300, 0, 1), (402, 1, 3, 0),
         (403, 57, 2, 0), (460, 2, 1, 0), (462, 129, 1, 1), (591, 3, 0, 0), (594, 111, 4, 0)]
MIXED_RANKS = [16, 8, 64, 32, 5]
HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_adamw_three_steps(dtype):
    import torch
    from paper_2607_28848_amd import dsv
    w = wl.custom(MIXED, MIXED_RANKS, K=520, N=776, dtype=dtype, r_max=64, name="adamw")
    run = Run(w, pad=np.nan)
    A, B = run.A, run.B                      # parameter stacks (NaN rank padding)
    A0, B0 = A.clone(), B.clone()
    Am, Bm = A.float().clone(), B.float().clone()   # fp32 masters start at the parameters
    mA, vA, mB, vB = (torch.zeros_like(x) for x in (Am, Am, Bm, Bm))
    train = sorted({a for (_, l, a, t) in MIXED if t and l})
    ranks = MIXED_RANKS
    # reference state (fp64), trained slices only
    ref = {}
    for a in train:
        r = ranks[a]
        ref[a] = [Am[a, :r].double().cpu().numpy(), np.zeros((r, 520)), np.zeros((r, 520)),
                  Bm[a, :, :r].double().cpu().numpy(), np.zeros((776, r)), np.zeros((776, r))]
    rng = np.random.default_rng(21)
    for step in (1, 2, 3):
        gA = torch.tensor(rng.normal(size=Am.shape) * 1e-2, dtype=torch.float32, device="cuda")
        gB = torch.tensor(rng.normal(size=Bm.shape) * 1e-2, dtype=torch.float32, device="cuda")
        dsv.adamw_step(run.plan, step, gA, gB, Am, Bm, mA, vA, mB, vB, A=A, B=B, **HP)
        for a in train:
            r = ranks[a]
            s = ref[a]
            s[0], s[1], s[2] = oracle.adamw(s[0], gA[a, :r].double().cpu().numpy(), s[1], s[2], step, **HP)
            s[3], s[4], s[5] = oracle.adamw(s[3], gB[a, :, :r].double().cpu().numpy(), s[4], s[5], step, **HP)
    torch.cuda.synchronize()
    for a in train:
        r = ranks[a]
        s = ref[a]
        got = [Am[a, :r], mA[a, :r], vA[a, :r], Bm[a, :, :r], mB[a, :, :r], vB[a, :, :r]]
        for name, gt, rf in zip(["A", "mA", "vA", "B", "mB", "vB"], got, s):
            e = oracle.rel_err(gt.double().cpu().numpy(), rf)
            assert e <= TOL_F32, (a, name, e)
        # the parameter copy is the master rounded once
        assert torch.equal(A[a, :r].cpu(), Am[a, :r].cpu().to(A.dtype))
        assert torch.equal(B[a, :, :r].cpu(), Bm[a, :, :r].cpu().to(B.dtype))
    # untouched: other adapters, rank padding of the trained ones (NaN stays NaN)
    same = lambda x, y: torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),  # noqa: E731
                                    y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))
    for a in range(len(ranks)):
        r = ranks[a] if a in train else 0
        assert same(A[a, r:], A0[a, r:]) and same(B[a, :, r:], B0[a, :, r:])
        if a not in train:
            assert not mA[a].any() and not vB[a].any()
