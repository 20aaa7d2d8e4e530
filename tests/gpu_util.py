"""Helpers of the GPU tests: move a workload's inputs to the device, run the HIP
path through the C ABI binding, bring results back as float64, and run the
fp64 reference on the same inputs."""
from __future__ import annotations

import numpy as np

import oracle
from paper_2607_28848_amd import workloads as wl

TOL_BF16 = 2e-2
TOL_F32 = 1e-5


def to_dev(arr, dtype: str):
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    return t.to("cuda")


def to_host(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return wl.bf16_bits_to_f64(bits)
    return t.detach().cpu().numpy().astype(np.float64)


class Run:
    """One projection of a workload through the GPU path."""

    def __init__(self, w: wl.Workload, p: int = 0, pad=np.nan, tensors=None):
        from paper_2607_28848_amd import dsv
        self.w = w
        self.t = tensors if tensors is not None else w.tensors(p, pad=pad)
        self.plan = dsv.segments_build(w.segments, w.n_tokens, w.ranks, w.scales, w.r_max,
                                       device="cuda")
        st = self.t.store
        self.X, self.W = to_dev(st["X"], w.dtype), to_dev(st["W"], w.dtype)
        self.A, self.B = to_dev(st["A"], w.dtype), to_dev(st["B"], w.dtype)
        self.dY = to_dev(st["dY"], w.dtype)
        self.dsv = dsv

    def fwd(self, H_save=None):
        Y, H = self.dsv.cobatch_fwd(self.plan, self.X, self.W, self.A, self.B, H_save=H_save)
        return Y, H

    def bwd(self, H_save, dA=None, dB=None, accumulate=False, want_dx=True):
        return self.dsv.lora_bwd(self.plan, self.X, self.W, self.A, self.B, H_save, self.dY,
                                 dA=dA, dB=dB, want_dx=want_dx, accumulate=accumulate)


def oracle_fwd(w, t, rows=None, drop=None):
    return oracle.forward(w.segments, w.ranks, w.scales, w.r_max, t.X, t.W, t.A, t.B, rows, drop=drop)


def oracle_bwd(w, t, dx_rows=None, dA=None, dB=None, drop=None):
    return oracle.backward(w.segments, w.ranks, w.scales, w.r_max, t.X, t.W, t.A, t.B, t.dY,
                           dA=dA, dB=dB, dx_rows=dx_rows, drop=drop)


def train_mask_slices(w):
    """[(adapter, rank)] of adapters that own training rows."""
    ads = sorted({a for (_, l, a, tr) in w.segments if tr and l > 0})
    return [(a, int(w.ranks[a])) for a in ads]
