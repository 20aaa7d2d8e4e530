"""GPU: row-strided operands of the grouped calls (the ldx, ldw, ldy / ldx,
ldw, lddy, lddx, ldwt fields of dsv_fwd_proj and dsv_bwd_proj).

Bar: the results on strided buffers are bit-identical to those on dense
buffers holding the same values (a stride changes no arithmetic), the elements
between rows are never written, and the strided results are within the bf16 /
fp32 bar of the fp64 reference.
"""
import sys

import pytest

from gpu_util import TOL_BF16, TOL_F32
from test_gpu_grouped import _bits, _check_proj, _layer

pytestmark = pytest.mark.gpu

# per-operand padding (elements past the row) of the strided run, per projection
PADS = [dict(X=8, W=64, Y=24, dY=136, dX=8, Wt=64),
        dict(X=64, W=0, Y=0, dY=8, dX=64, Wt=0),
        dict(X=0, W=8, Y=64, dY=0, dX=0, Wt=8)]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _sentinel(dtype):
    import torch
    # a NaN bit pattern no kernel writes: bf16 0x7FC1, fp32 0x7FC00001
    return torch.tensor([0x7FC1 if dtype == torch.bfloat16 else 0x7FC00001],
                        dtype=torch.int16 if dtype == torch.bfloat16 else torch.int32)


def _padded(t, pad):
    """(buffer, view): a [R][C + pad] buffer whose padding holds the sentinel and
    whose first C columns hold t; the view is its [R][C] part."""
    import torch
    R, C = t.shape
    buf = torch.empty((R, C + pad), dtype=t.dtype, device=t.device)
    _bits(buf).fill_(int(_sentinel(t.dtype)[0]))
    buf[:, :C] = t
    return buf, buf[:, :C]


def _pad_untouched(buf, C):
    import torch
    if buf.shape[1] == C:
        return True
    s = int(_sentinel(buf.dtype)[0])
    return bool(torch.all(_bits(buf[:, C:]) == s).item())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_proj", [1, 3])
def test_strided_grouped_matches_dense(dtype, n_proj):
    """Grouped forward and backward (with the transposed weight for bf16) on
    row-strided X, W, Y, dY, dX and Wt against the same calls on dense buffers:
    every output bit-identical, row padding of Y and dX unwritten, and every
    output within the bar of the reference.  Shapes ragged against 64 and 256."""
    import torch
    from paper_2607_28848_amd import dsv
    shapes = [(520, 776), (136, 1040), (1040, 264)][:n_proj]
    _say("case strided %s n_proj=%d %s" % (dtype, n_proj, shapes))
    w, ts, dev = _layer(dtype, shapes)
    plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max, device="cuda")
    Tt = plan.train_tokens
    bf = dtype == "bf16"

    def hbuf(d):
        return torch.zeros((Tt, w.r_max), dtype=d["X"].dtype, device="cuda")

    # dense
    Hd = [hbuf(d) for d in dev]
    out_d = dsv.cobatch_fwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], None, Hd[i])
                                           for i, d in enumerate(dev)])
    wts_d = [d["W"].t().contiguous() for d in dev] if bf else None
    g_d = dsv.lora_bwd_grouped(plan, [(d["X"], d["W"], d["A"], d["B"], out_d[i][1], d["dY"])
                                      for i, d in enumerate(dev)], wts=wts_d)
    # strided
    fw, bw, bufs, wts_s = [], [], [], []
    for i, d in enumerate(dev):
        p = PADS[i]
        K, N = shapes[i]
        _, Xs = _padded(d["X"], p["X"])
        _, Ws = _padded(d["W"], p["W"])
        _, dYs = _padded(d["dY"], p["dY"])
        Yb, Ys = _padded(torch.zeros((w.n_tokens, N), dtype=d["X"].dtype, device="cuda"), p["Y"])
        dXb, dXs = _padded(torch.zeros((Tt, K), dtype=d["X"].dtype, device="cuda"), p["dX"])
        if bf:
            wts_s.append(_padded(wts_d[i], p["Wt"])[1])
        bufs.append((Yb, dXb))
        fw.append((Xs, Ws, d["A"], d["B"], Ys, hbuf(d)))
        bw.append([Xs, Ws, d["A"], d["B"], None, dYs, None, None, dXs])
    out_s = dsv.cobatch_fwd_grouped(plan, fw)
    for i in range(n_proj):
        bw[i][4] = out_s[i][1]
    g_s = dsv.lora_bwd_grouped(plan, [tuple(b) for b in bw], wts=wts_s if bf else None)
    torch.cuda.synchronize()
    tr = plan.train_rows()
    tol = TOL_BF16 if bf else TOL_F32
    projs = list(w.projections)
    for i, (K, N) in enumerate(shapes):
        _say(" projection %d K=%d N=%d pads %s" % (i, K, N, PADS[i]))
        for a, b in list(zip(out_s[i], out_d[i])) + list(zip(g_s[i], g_d[i])):
            assert torch.equal(_bits(a.contiguous()), _bits(b.contiguous()))
        assert _pad_untouched(bufs[i][0], N) and _pad_untouched(bufs[i][1], K)
        w.projections = [projs[i]]
        _check_proj(w, ts[i], tr, out_s[i][0], out_s[i][1], g_s[i][0], g_s[i][1], g_s[i][2], tol)
    w.projections = projs
