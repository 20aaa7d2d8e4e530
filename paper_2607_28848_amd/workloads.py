"""Seeded synthetic inputs for the co-batched multi-LoRA layer.

This module only draws numbers and segment tables; it holds none of the
layer's arithmetic, so both the HIP path and the fp64 reference consume it.

Distributions (the paper's workload, Sec. 4.1, is Llama 3-8B with rank-16,
alpha-32 adapters fine-tuned on Alpaca; neither the weights nor the corpus are
used: these synthetic draws of the same shapes stand in for them):
    X, dY ~ N(0, 1);  W ~ N(0, variance 1/K);  A ~ U[-1/sqrt(K), 1/sqrt(K)];
    B ~ N(0, std 0.02);  every adapter scale s_a = 2.0 (= alpha / r of the
    paper's adapter).
Values are drawn in float64 and rounded to nearest-even into the workload's
dtype (bf16 or fp32); consumers get both the rounded values (float64) and the
raw storage bits.

Draw order: the segment structure comes from ``default_rng(seed)``
(lengths, adapters, then the order shuffle); projection p draws X, W, A, B, dY
in that order from ``default_rng([seed, p + 1])``.

Storage is the paper's orientation (Sec. 2.2), row-major:
    X [T][K], W [N][K], A [n_ad][r_max][K], B [n_ad][N][r_max], dY [T_t][N].
Rank padding (j >= r_a) is filled with ``pad`` (NaN in tests, 0 in the bench).
"""
from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

import numpy as np

Segment = Tuple[int, int, int, int]  # (start, len, adapter, is_train)


def round_bf16(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Round float64 values to bfloat16, nearest-even, directly from float64.

    Returns (values as float64, storage bits as uint16).  NaN stays NaN.
    Finite inputs must lie in the normal bf16 range (true for every draw here).
    The rounding works on the float64 bit pattern: the 45 low mantissa bits
    are dropped with round-half-to-even (a carry ripples into the exponent).
    """
    x = np.ascontiguousarray(x, np.float64)
    u = x.view(np.uint64)
    r = u >> np.uint64(45)
    r &= np.uint64(1)
    r += np.uint64((1 << 44) - 1)
    r += u
    r &= np.uint64(~((1 << 45) - 1) & 0xFFFFFFFFFFFFFFFF)
    v = r.view(np.float64)
    nan = np.isnan(x)
    if nan.any():
        v[nan] = np.nan
    bits = v.astype(np.float32).view(np.uint32)
    bits >>= np.uint32(16)
    return v, bits.astype(np.uint16)


def round_f32(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    v32 = np.asarray(x, np.float64).astype(np.float32)
    return v32.astype(np.float64), v32


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    f32 = (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)
    with np.errstate(invalid="ignore"):
        return f32.astype(np.float64)


@dataclasses.dataclass
class Projection:
    name: str
    K: int   # in features
    N: int   # out features


@dataclasses.dataclass
class Tensors:
    """One projection's inputs: float64 values (dtype-rounded) and storage arrays."""
    X: np.ndarray
    W: np.ndarray
    A: np.ndarray
    B: np.ndarray
    dY: np.ndarray
    store: dict   # name -> uint16 bf16 bits or float32 values, same shapes


@dataclasses.dataclass
class Workload:
    name: str
    dtype: str                       # "bf16" or "f32"
    segments: List[Segment]
    n_tokens: int
    ranks: np.ndarray                # int32 [n_ad]
    scales: np.ndarray               # float32 [n_ad]
    r_max: int
    projections: List[Projection]
    seed: int = 0

    @property
    def n_adapters(self) -> int:
        return int(self.ranks.shape[0])

    @property
    def train_tokens(self) -> int:
        return int(sum(l for (_, l, _, t) in self.segments if t))

    def tensors(self, p: int, pad: float = np.nan, with_dy: bool = True) -> Tensors:
        """Draw projection p's inputs."""
        proj = self.projections[p]
        K, N, r_max = proj.K, proj.N, self.r_max
        n_ad, T, Tt = self.n_adapters, self.n_tokens, self.train_tokens
        rng = np.random.default_rng([self.seed, p + 1])
        X = rng.standard_normal((T, K))
        W = rng.standard_normal((N, K)) * (1.0 / np.sqrt(K))
        lim = 1.0 / np.sqrt(K)
        A = rng.uniform(-lim, lim, size=(n_ad, r_max, K))
        B = rng.standard_normal((n_ad, N, r_max)) * 0.02
        dY = rng.standard_normal((Tt, N)) if with_dy else np.zeros((Tt, N))
        for a in range(n_ad):
            r = int(self.ranks[a])
            A[a, r:, :] = pad
            B[a, :, r:] = pad
        rnd = round_bf16 if self.dtype == "bf16" else round_f32
        vals, store = {}, {}
        for nm, arr in (("X", X), ("W", W), ("A", A), ("B", B), ("dY", dY)):
            v, s = rnd(arr)
            vals[nm] = v
            store[nm] = s
        return Tensors(vals["X"], vals["W"], vals["A"], vals["B"], vals["dY"], store)


def _lay_out(rng: np.random.Generator, pieces: Sequence[Tuple[int, int, int]]) -> List[Segment]:
    """Shuffle (len, adapter, is_train) pieces and assign consecutive starts."""
    order = rng.permutation(len(pieces))
    segs, start = [], 0
    for i in order:
        l, a, t = pieces[int(i)]
        segs.append((start, int(l), int(a), int(t)))
        start += int(l)
    return segs


LLAMA3_8B = [Projection("q", 4096, 4096), Projection("k", 4096, 1024),
             Projection("v", 4096, 1024), Projection("o", 4096, 4096),
             Projection("gate", 4096, 14336), Projection("up", 4096, 14336),
             Projection("down", 14336, 4096)]


def tiny(seed: int = 0) -> Workload:
    """K = N = 512 fp32; 2 adapters of rank 8; 128 + 64 inference rows, 64 training rows."""
    segs = [(0, 128, 0, 0), (128, 64, 1, 0), (192, 64, 0, 1)]
    return Workload("tiny_512_f32", "f32", segs, 256, np.array([8, 8], np.int32),
                    np.full(2, 2.0, np.float32), 8, [Projection("tiny", 512, 512)], seed)


def llama8b_mixed(seed: int = 0) -> Workload:
    """Llama-3-8B layer set, bf16: 8 x 512 prefill on adapters U{0..31}, 2 x 1024 training
    on adapter 0, 32 adapters of rank 16."""
    rng = np.random.default_rng(seed)
    ads = rng.integers(0, 32, size=8)
    pieces = [(512, int(a), 0) for a in ads] + [(1024, 0, 1), (1024, 0, 1)]
    segs = _lay_out(rng, pieces)
    return Workload("llama3_8b_layer_set_mixed", "bf16", segs, 6144,
                    np.full(32, 16, np.int32), np.full(32, 2.0, np.float32), 16,
                    list(LLAMA3_8B), seed)


def decode_heavy(seed: int = 0) -> Workload:
    """4096 x 14336 gate, bf16: 256 one-token decode segments over 64 adapters with ranks
    (8,16,32,64)[a mod 4], plus one 2048-token training sequence on adapter 1."""
    rng = np.random.default_rng(seed)
    ads = rng.integers(0, 64, size=256)
    pieces = [(1, int(a), 0) for a in ads] + [(2048, 1, 1)]
    segs = _lay_out(rng, pieces)
    ranks = np.array([(8, 16, 32, 64)[a % 4] for a in range(64)], np.int32)
    return Workload("decode_heavy_gate_4096x14336", "bf16", segs, 2304, ranks,
                    np.full(64, 2.0, np.float32), 64, [Projection("gate", 4096, 14336)], seed)


def llama70b(seed: int = 0) -> Workload:
    """Llama-3-70B up/down on one GPU, bf16: 16 prefill segments with lognormal(6, 0.7)
    lengths clipped to [32, 4096] plus 4 x 2048 training on adapter 0; 16 adapters of rank 64."""
    rng = np.random.default_rng(seed)
    lens = np.clip(np.rint(rng.lognormal(6.0, 0.7, size=16)), 32, 4096).astype(int)
    ads = rng.integers(0, 16, size=16)
    pieces = [(int(l), int(a), 0) for l, a in zip(lens, ads)] + [(2048, 0, 1)] * 4
    segs = _lay_out(rng, pieces)
    T = sum(p[0] for p in pieces)
    return Workload("llama3_70b_up_down", "bf16", segs, T, np.full(16, 64, np.int32),
                    np.full(16, 2.0, np.float32), 64,
                    [Projection("up", 8192, 28672), Projection("down", 28672, 8192)], seed)


def load_sweep(frac: float, seed: int = 0) -> Workload:
    """4096 x 14336, bf16, 64 adapters of rank 16, 16384 tokens; a fraction `frac` of them
    in 1024-token training sequences on adapter 0, the rest in inference segments with
    lognormal(5.5, 1.0) lengths."""
    rng = np.random.default_rng(seed)
    total = 16384
    n_train = int(round(16 * frac))
    inf_tokens = total - 1024 * n_train
    pieces = []
    left = inf_tokens
    while left > 0:
        l = int(np.clip(np.rint(rng.lognormal(5.5, 1.0)), 1, left))
        pieces.append((l, int(rng.integers(0, 64)), 0))
        left -= l
    pieces += [(1024, 0, 1)] * n_train
    segs = _lay_out(rng, pieces)
    return Workload("load_sweep_4096x14336_f%.2f" % frac, "bf16", segs, total,
                    np.full(64, 16, np.int32), np.full(64, 2.0, np.float32), 16,
                    [Projection("gate", 4096, 14336)], seed)


def custom(segments: Sequence[Segment], ranks: Sequence[int], K: int, N: int,
           dtype: str = "bf16", r_max: int | None = None, scales=None, seed: int = 0,
           name: str = "custom") -> Workload:
    """A small workload with an explicit segment table (used by the tests)."""
    ranks = np.asarray(ranks, np.int32)
    T = sum(int(s[1]) for s in segments)
    if r_max is None:
        r_max = int(ranks.max())
    sc = np.full(ranks.shape[0], 2.0, np.float32) if scales is None else np.asarray(scales, np.float32)
    return Workload(name, dtype, [tuple(int(v) for v in s) for s in segments], T, ranks, sc,
                    int(r_max), [Projection(name, K, N)], seed)


CONFIGS = {
    "tiny": tiny,
    "llama8b": llama8b_mixed,
    "decode": decode_heavy,
    "llama70b": llama70b,
}
