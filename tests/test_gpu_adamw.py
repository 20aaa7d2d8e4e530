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


# Training adapters 0 (rank 16) and 1 (rank 8): B in float4 units.  Training
# adapter 4 (rank 5) as well: B one entry at a time.
GROUP_CASES = {
    "ranks_mult4": MIXED,
    "rank5_scalar_b": MIXED[:-1] + [(594, 111, 4, 1)],
}


@pytest.mark.parametrize("case", sorted(GROUP_CASES))
def test_adamw_grouped_three_projections(case):
    """dsv_adamw_step_grouped over three projections of different K x N: two steps
    against the fp64 reference (1e-5 per tensor), bit-identical to the single calls
    on copies of the same state, the parameter copy the rounded master, and every
    other adapter and rank-padding entry untouched."""
    import torch
    from paper_2607_28848_amd import dsv
    segs = GROUP_CASES[case]
    shapes = [(520, 776), (136, 64), (264, 1032)]
    runs = [Run(wl.custom(segs, MIXED_RANKS, K=K, N=N, dtype="bf16", r_max=64, name="adamw_g%d" % i), pad=np.nan)
            for i, (K, N) in enumerate(shapes)]
    plan = runs[0].plan
    train = sorted({a for (_, l, a, t) in segs if t and l})
    rng = np.random.default_rng(33)
    state, single, ref, orig = [], [], [], []
    for run in runs:
        Am, Bm = run.A.float().clone(), run.B.float().clone()
        st = [Am, Bm] + [torch.zeros_like(x) for x in (Am, Am, Bm, Bm)] + [run.A, run.B]
        state.append(st)
        single.append([x.clone() for x in st])
        orig.append((run.A.clone(), run.B.clone()))
        ref.append({a: [Am[a, :MIXED_RANKS[a]].double().cpu().numpy(), 0.0, 0.0,
                        Bm[a, :, :MIXED_RANKS[a]].double().cpu().numpy(), 0.0, 0.0] for a in train})
    for step in (1, 2):
        grads = [(torch.tensor(rng.normal(size=st[0].shape) * 1e-2, dtype=torch.float32, device="cuda"),
                  torch.tensor(rng.normal(size=st[1].shape) * 1e-2, dtype=torch.float32, device="cuda"))
                 for st in state]
        dsv.adamw_step_grouped(plan, step, [(g[0], g[1], *st) for g, st in zip(grads, state)], **HP)
        for g, st in zip(grads, single):
            dsv.adamw_step(plan, step, g[0], g[1], *st[:6], A=st[6], B=st[7], **HP)
        for g, rf in zip(grads, ref):
            for a in train:
                r = MIXED_RANKS[a]
                s = rf[a]
                gA = g[0][a, :r].double().cpu().numpy()
                gB = g[1][a, :, :r].double().cpu().numpy()
                mA0 = s[1] if step > 1 else np.zeros_like(gA)
                vA0 = s[2] if step > 1 else np.zeros_like(gA)
                mB0 = s[4] if step > 1 else np.zeros_like(gB)
                vB0 = s[5] if step > 1 else np.zeros_like(gB)
                s[0], s[1], s[2] = oracle.adamw(s[0], gA, mA0, vA0, step, **HP)
                s[3], s[4], s[5] = oracle.adamw(s[3], gB, mB0, vB0, step, **HP)
    torch.cuda.synchronize()
    bits = lambda x: x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32)  # noqa: E731
    for p, (st, sg, rf, (A0, B0)) in enumerate(zip(state, single, ref, orig)):
        for x, y in zip(st, sg):
            assert torch.equal(bits(x), bits(y)), p
        Am, Bm, mA, vA, mB, vB, A, B = st
        for a in train:
            r = MIXED_RANKS[a]
            got = [Am[a, :r], mA[a, :r], vA[a, :r], Bm[a, :, :r], mB[a, :, :r], vB[a, :, :r]]
            for name, gt, want in zip(["A", "mA", "vA", "B", "mB", "vB"], got, rf[a]):
                e = oracle.rel_err(gt.double().cpu().numpy(), want)
                assert e <= TOL_F32, (p, a, name, e)
            assert torch.equal(A[a, :r].cpu(), Am[a, :r].cpu().to(A.dtype))
            assert torch.equal(B[a, :, :r].cpu(), Bm[a, :, :r].cpu().to(B.dtype))
        for a in range(len(MIXED_RANKS)):
            r = MIXED_RANKS[a] if a in train else 0
            assert torch.equal(bits(A[a, r:]), bits(A0[a, r:])) and torch.equal(bits(B[a, :, r:]), bits(B0[a, :, r:]))
            if a not in train:
                assert not mA[a].any() and not vB[a].any()
