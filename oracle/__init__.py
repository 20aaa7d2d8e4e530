"""fp64 reference ("oracle") of the co-batched multi-LoRA linear layer.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the bench's
CPU-baseline leg are the only callers.  The product path (the HIP library
under ``paper_2607_28848_amd``) never imports this package, and this package
imports nothing from it.

The arithmetic lives in ``dsvo.c`` (plain fp64 loops, see ``dsvo.h`` for the
definitions and the paper passages they follow).  This module builds that file
with gcc and marshals numpy arrays through ctypes.

Layouts (row-major, the paper's orientation of Sec. 2.2, i.e. the
torch.nn.Linear / PEFT parameter layout):
    X [T][K]   W [N][K]   A [n_ad][r_max][K]   B [n_ad][N][r_max]
    dY, dX, H_save, G: compact training rows, ascending token row.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dsvo.c")
_LIB = os.path.join(_HERE, "libdsvo.so")
_ASAN_LIB = os.path.join(_HERE, "_build", "libdsvo_asan.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile dsvo.c into libdsvo.so next to it (gcc, -O2, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c99", "-Wall",
             "-o", tmp, _SRC, "-lm"], cwd=_HERE)
        os.replace(tmp, _LIB)
    return _LIB


def build_asan() -> str:
    """Compile dsvo.c with AddressSanitizer + UBSan into _build/libdsvo_asan.so,
    for host-sanitizer runs of the oracle's tests (DSVO_LIBRARY names it)."""
    os.makedirs(os.path.dirname(_ASAN_LIB), exist_ok=True)
    tmp = _ASAN_LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(
        ["gcc", "-O1", "-g", "-fopenmp", "-shared", "-fPIC", "-std=c99", "-Wall",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
         "-o", tmp, _SRC, "-lm"], cwd=_HERE)
    os.replace(tmp, _ASAN_LIB)
    return _ASAN_LIB


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("DSVO_LIBRARY")
        if not path:
            path = _LIB
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
        lib = ctypes.CDLL(path)
        i32p = ctypes.POINTER(ctypes.c_int32)
        f64p = ctypes.POINTER(ctypes.c_double)
        ci = ctypes.c_int
        lib.dsvo_rows.argtypes = [ci, ci, i32p, ci, i32p, i32p]
        lib.dsvo_rows.restype = ci
        lib.dsvo_forward.argtypes = [ci, ci, ci, ci, i32p, ci, i32p, f64p, ci,
                                     f64p, f64p, f64p, f64p, f64p, ci, i32p, f64p, f64p]
        lib.dsvo_forward.restype = ci
        lib.dsvo_backward.argtypes = [ci, ci, ci, ci, i32p, ci, i32p, f64p, ci,
                                      f64p, f64p, f64p, f64p, f64p, f64p, f64p, f64p, f64p,
                                      ci, i32p, f64p]
        lib.dsvo_backward.restype = ci
        lib.dsvo_threads.argtypes = []
        lib.dsvo_threads.restype = ci
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the reference's loops run with."""
    return int(_load().dsvo_threads())


def _i32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f64(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _seg_table(segments):
    t = np.asarray(segments, dtype=np.int32).reshape(-1, 4)
    return np.ascontiguousarray(t)


def rows(segments, n_tokens: int, n_adapters: int):
    """(row_adapter[T], train_rows[T_t]) of a segment table; raises on a bad table."""
    seg, segp = _i32(_seg_table(segments))
    ra, rap = _i32(np.zeros(max(n_tokens, 1), np.int32))
    tr, trp = _i32(np.zeros(max(n_tokens, 1), np.int32))
    tt = _load().dsvo_rows(n_tokens, seg.shape[0], segp, n_adapters, rap, trp)
    if tt < 0:
        raise ValueError("segment table does not tile [0, n_tokens) or names a bad adapter")
    return ra[:n_tokens].copy(), tr[:tt].copy()


def _drop_ptr(drop):
    if drop is None:
        return None, ctypes.POINTER(ctypes.c_double)()
    return _f64(drop)


def forward(segments, ranks, scales, r_max, X, W, A, B, rows_sel=None, drop=None):
    """fp64 forward.  Returns (Y[rows][N], H[rows][r_max]); rows default to all.

    H entries at j >= r_a are NaN (never written by the definition).  drop: the
    LoRA-dropout multipliers of the training rows, [T_t][K] (dropout_multipliers),
    or None."""
    X, Xp = _f64(X)
    W, Wp = _f64(W)
    A, Ap = _f64(A)
    B, Bp = _f64(B)
    T, K = X.shape
    N = W.shape[0]
    n_ad = A.shape[0]
    assert W.shape == (N, K) and A.shape == (n_ad, r_max, K) and B.shape == (n_ad, N, r_max)
    seg, segp = _i32(_seg_table(segments))
    rk, rkp = _i32(ranks)
    sc, scp = _f64(scales)
    if rows_sel is None:
        rows_sel = np.arange(T, dtype=np.int32)
    rs, rsp = _i32(rows_sel)
    dr_, drp_ = _drop_ptr(drop)
    Y = np.empty((rs.shape[0], N), np.float64)
    H = np.full((rs.shape[0], r_max), np.nan, np.float64)
    rc = _load().dsvo_forward(T, K, N, seg.shape[0], segp, n_ad, rkp, scp, r_max,
                              Xp, Wp, Ap, Bp, drp_, rs.shape[0], rsp,
                              Y.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                              H.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError("oracle forward rejected its arguments")
    return Y, H


def backward(segments, ranks, scales, r_max, X, W, A, B, dY, dA=None, dB=None, dx_rows=None,
             drop=None):
    """fp64 backward.  Returns (G, dA, dB, dX).  drop as in forward.

    dA/dB are copies of the given arrays (NaN-filled when None) with the slices
    of adapters that own training rows overwritten.  dX covers the compact
    training rows in dx_rows (default: all)."""
    X, Xp = _f64(X)
    W, Wp = _f64(W)
    A, Ap = _f64(A)
    B, Bp = _f64(B)
    dY, dYp = _f64(dY)
    T, K = X.shape
    N = W.shape[0]
    n_ad = A.shape[0]
    seg, segp = _i32(_seg_table(segments))
    rk, rkp = _i32(ranks)
    sc, scp = _f64(scales)
    tt = dY.shape[0]
    dA = np.full((n_ad, r_max, K), np.nan) if dA is None else np.array(dA, np.float64, copy=True)
    dB = np.full((n_ad, N, r_max), np.nan) if dB is None else np.array(dB, np.float64, copy=True)
    G = np.full((max(tt, 1), r_max), np.nan)
    if dx_rows is None:
        dx_rows = np.arange(tt, dtype=np.int32)
    dr, drp = _i32(dx_rows)
    dq_, dqp_ = _drop_ptr(drop)
    dX = np.empty((dr.shape[0], K), np.float64)
    f64p = ctypes.POINTER(ctypes.c_double)
    rc = _load().dsvo_backward(T, K, N, seg.shape[0], segp, n_ad, rkp, scp, r_max,
                               Xp, Wp, Ap, Bp, dqp_, dYp, G.ctypes.data_as(f64p),
                               dA.ctypes.data_as(f64p), dB.ctypes.data_as(f64p),
                               dr.shape[0], drp, dX.ctypes.data_as(f64p))
    if rc != 0:
        raise ValueError("oracle backward rejected its arguments")
    return G[:tt], dA, dB, dX


def rel_err(got, ref) -> float:
    """max|got - ref| / max|ref| over the finite reference entries, in fp64."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    m = np.isfinite(ref)
    den = np.max(np.abs(ref[m])) if m.any() else 0.0
    num = np.max(np.abs(got[m] - ref[m])) if m.any() else 0.0
    if den == 0.0:
        return float(num)
    return float(num / den)


def adamw(p, g, m, v, step, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01):
    """One AdamW step in fp64 (Sec. 4.1 training configuration: AdamW, learning
    rate 1e-3, weight decay 0.01; Sec. 3.2: the update is applied to the adapter
    weights after the backward).  Decoupled weight decay as in Loshchilov & Hutter
    (ICLR 2019) with the schedule multiplier equal to the learning rate:

        m_t = beta1 m + (1 - beta1) g           v_t = beta2 v + (1 - beta2) g^2
        m^  = m_t / (1 - beta1^t)                v^  = v_t / (1 - beta2^t)
        p_t = p - lr (m^ / (sqrt(v^) + eps) + weight_decay p)

    Returns (p_t, m_t, v_t) as new fp64 arrays; the inputs are not modified."""
    p, g, m, v = (np.asarray(x, np.float64) for x in (p, g, m, v))
    m_t = beta1 * m + (1.0 - beta1) * g
    v_t = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m_t / (1.0 - beta1 ** step)
    v_hat = v_t / (1.0 - beta2 ** step)
    p_t = p - lr * (m_hat / (np.sqrt(v_hat) + eps) + weight_decay * p)
    return p_t, m_t, v_t


# ---------------------------------------------------------------------------
# LoRA dropout (Sec. 4.1: dropout 0.05 on the adapter input of the training
# rows) with a counter-based generator: Philox4x32-10 (Salmon, Moraes, Dror and
# Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011), written from
# its published definition.
# ---------------------------------------------------------------------------
_PHILOX_M = (0xD2511F53, 0xCD9E8D57)   # round multipliers
_PHILOX_W = (0x9E3779B9, 0xBB67AE85)   # key increments (Weyl sequence)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Philox4x32 with 10 rounds, elementwise over equally shaped uint32 arrays
    (counter words c0..c3, key words k0, k1).  Returns the four output words."""
    c = [np.asarray(x, np.uint64) & 0xFFFFFFFF for x in (c0, c1, c2, c3)]
    k = [np.asarray(x, np.uint64) & 0xFFFFFFFF for x in (k0, k1)]
    for rnd in range(10):
        if rnd:
            k = [(k[0] + _PHILOX_W[0]) & 0xFFFFFFFF, (k[1] + _PHILOX_W[1]) & 0xFFFFFFFF]
        p0 = c[0] * np.uint64(_PHILOX_M[0])     # 32 x 32 -> 64 bit products
        p1 = c[2] * np.uint64(_PHILOX_M[1])
        c = [((p1 >> 32) ^ c[1] ^ k[0]) & 0xFFFFFFFF, p1 & 0xFFFFFFFF,
             ((p0 >> 32) ^ c[3] ^ k[1]) & 0xFFFFFFFF, p0 & 0xFFFFFFFF]
    return [x.astype(np.uint32) for x in c]


def dropout_keep(n_rows: int, K: int, p: float, seed: int, offset: int = 0):
    """Kept-element mask [n_rows][K] of the training rows (compact order i):
    element (i, k) takes word k % 4 of Philox4x32-10 at counter
    (k // 4, i, offset low, offset high) and key (seed low, seed high), and is
    dropped when that word is below floor(p * 2^32)."""
    thr = min(int(p * 4294967296.0), 0xFFFFFFFF)
    q = np.arange((K + 3) // 4, dtype=np.uint64)
    i = np.arange(n_rows, dtype=np.uint64)
    Q, I = np.meshgrid(q, i)
    words = philox4x32_10(Q, I, np.full_like(Q, offset & 0xFFFFFFFF), np.full_like(Q, offset >> 32),
                          np.full_like(Q, seed & 0xFFFFFFFF), np.full_like(Q, seed >> 32))
    u = np.stack(words, axis=-1).reshape(n_rows, -1)[:, :K]
    return u >= thr


def dropout_multipliers(n_rows: int, K: int, p: float, seed: int, offset: int = 0):
    """[n_rows][K] fp64: kept mask / (1 - p) (inverted dropout), for forward / backward."""
    return dropout_keep(n_rows, K, p, seed, offset).astype(np.float64) / (1.0 - p)
