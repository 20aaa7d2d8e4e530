"""ctypes binding of libdsv.so (include/dsv.h): argument marshalling only.

Every step of the layer runs in the HIP library; torch supplies device memory
and the current HIP stream.  Importing this module fails loudly when the
library has not been built (``python -m paper_2607_28848_amd.build``).

Layouts (the paper's orientation, = torch.nn.Linear / PEFT parameters):
    X [T][K], W [N][K], A [n_ad][r_max][K], B [n_ad][N][r_max],
    Y [T][N], H_save / dY / dX over the compact training rows,
    dA [n_ad][r_max][K] fp32, dB [n_ad][N][r_max] fp32.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# DSV_LIBRARY may name another build of the same library (the host-sanitized
# variant of build.py); it must exist, there is no fallback either way.
LIB_PATH = os.environ.get("DSV_LIBRARY") or os.path.join(_HERE, "libdsv.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("%s is not built: run `python -m paper_2607_28848_amd.build` "
                      "(there is no fallback implementation)" % LIB_PATH)

# torch ships its own HIP runtime (same SONAME as /opt/rocm's).  Load it first so
# that libdsv.so binds to that one runtime: device pointers and streams handed
# over from torch are only valid in the runtime that created them.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

OK, ERR_ARG, ERR_RANGE, ERR_LAYOUT, ERR_SIZE, ERR_DEVICE = 0, -1, -2, -3, -4, -5
BF16, F32 = 0, 1
MAX_RANK = 64

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_sz = ctypes.c_size_t
_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)

_lib.dsv_segments_build.argtypes = [_i32p, _i32, _i32, _i32p, _f32p, _i32, _i32, _vp,
                                    ctypes.POINTER(_sz), _vp, ctypes.POINTER(_vp)]
_lib.dsv_segments_build.restype = ctypes.c_int
_lib.dsv_plan_train_rows.argtypes = [_vp]
_lib.dsv_plan_train_rows.restype = _i32
_lib.dsv_plan_train_row_index.argtypes = [_vp, _i32p]
_lib.dsv_plan_train_row_index.restype = _i32
_lib.dsv_plan_gathered_rows.argtypes = [_vp, _i32p]
_lib.dsv_plan_gathered_rows.restype = _i32
_lib.dsv_plan_meta_copy.argtypes = [_vp, _vp, _sz]
_lib.dsv_plan_meta_copy.restype = ctypes.c_int
_lib.dsv_plan_counts.argtypes = [_vp, _i32p]
_lib.dsv_plan_counts.restype = ctypes.c_int
_lib.dsv_plan_free.argtypes = [_vp]
_lib.dsv_plan_free.restype = None
_lib.dsv_cobatch_fwd_workspace.argtypes = [_vp, ctypes.c_int, _i32, _i32, ctypes.POINTER(_sz)]
_lib.dsv_cobatch_fwd_workspace.restype = ctypes.c_int
_lib.dsv_cobatch_fwd.argtypes = [_vp, ctypes.c_int, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                 _vp, _sz, _vp]
_lib.dsv_cobatch_fwd.restype = ctypes.c_int
_lib.dsv_cobatch_fwd_noalloc.argtypes = [_vp, ctypes.c_int, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
_lib.dsv_cobatch_fwd_noalloc.restype = ctypes.c_int
NOALLOC_SCRATCH_BYTES = 64 << 20  # DSV_NOALLOC_SCRATCH_BYTES of include/dsv.h
_lib.dsv_lora_bwd_workspace.argtypes = [_vp, ctypes.c_int, _i32, _i32, ctypes.POINTER(_sz)]
_lib.dsv_lora_bwd_workspace.restype = ctypes.c_int
_lib.dsv_lora_bwd.argtypes = [_vp, ctypes.c_int, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                              _vp, _vp, _i32, _vp, _sz, _vp]
_lib.dsv_lora_bwd.restype = ctypes.c_int
class Dropout(ctypes.Structure):
    _fields_ = [("p", ctypes.c_double), ("seed", ctypes.c_uint64), ("offset", ctypes.c_uint64), ("mask", _vp)]


_lib.dsv_cobatch_fwd_dropout.argtypes = [_vp, ctypes.c_int, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                         ctypes.POINTER(Dropout), _vp, _sz, _vp]
_lib.dsv_cobatch_fwd_dropout.restype = ctypes.c_int
_lib.dsv_lora_bwd_dropout_workspace.argtypes = [_vp, ctypes.c_int, _i32, _i32, ctypes.POINTER(_sz)]
_lib.dsv_lora_bwd_dropout_workspace.restype = ctypes.c_int
_lib.dsv_lora_bwd_dropout.argtypes = [_vp, ctypes.c_int, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                      _vp, _vp, _i32, ctypes.POINTER(Dropout), _vp, _sz, _vp]
_lib.dsv_lora_bwd_dropout.restype = ctypes.c_int
class FwdProj(ctypes.Structure):
    _fields_ = [("K", _i32), ("N", _i32), ("X", _vp), ("W", _vp), ("A", _vp), ("B", _vp), ("Y", _vp),
                ("H_save", _vp), ("ldx", _i32), ("ldw", _i32), ("ldy", _i32)]


class BwdProj(ctypes.Structure):
    _fields_ = [("K", _i32), ("N", _i32), ("X", _vp), ("W", _vp), ("A", _vp), ("B", _vp), ("H_save", _vp),
                ("dY", _vp), ("dA", _vp), ("dB", _vp), ("dX", _vp), ("Wt", _vp), ("ldx", _i32), ("ldw", _i32),
                ("lddy", _i32), ("lddx", _i32), ("ldwt", _i32)]


_lib.dsv_row_stride.argtypes = [_i32, ctypes.c_int]
_lib.dsv_row_stride.restype = _i32


MAX_GROUP = 8
_lib.dsv_cobatch_fwd_grouped_workspace.argtypes = [_vp, ctypes.c_int, _i32, ctypes.POINTER(FwdProj),
                                                   ctypes.POINTER(_sz)]
_lib.dsv_cobatch_fwd_grouped_workspace.restype = ctypes.c_int
_lib.dsv_cobatch_fwd_grouped.argtypes = [_vp, ctypes.c_int, _i32, ctypes.POINTER(FwdProj), _vp, _sz, _vp]
_lib.dsv_cobatch_fwd_grouped.restype = ctypes.c_int
_lib.dsv_lora_bwd_grouped_workspace.argtypes = [_vp, ctypes.c_int, _i32, ctypes.POINTER(BwdProj),
                                                ctypes.POINTER(_sz)]
_lib.dsv_lora_bwd_grouped_workspace.restype = ctypes.c_int
_lib.dsv_lora_bwd_grouped.argtypes = [_vp, ctypes.c_int, _i32, ctypes.POINTER(BwdProj), _i32, _vp, _sz, _vp]
_lib.dsv_lora_bwd_grouped.restype = ctypes.c_int
_lib.dsv_cobatch_fwd_grouped_dropout.argtypes = [_vp, ctypes.c_int, _i32, ctypes.POINTER(FwdProj),
                                                 ctypes.POINTER(Dropout), _vp, _sz, _vp]
_lib.dsv_cobatch_fwd_grouped_dropout.restype = ctypes.c_int
_lib.dsv_lora_bwd_grouped_dropout.argtypes = [_vp, ctypes.c_int, _i32, ctypes.POINTER(BwdProj), _i32,
                                              ctypes.POINTER(Dropout), _vp, _sz, _vp]
_lib.dsv_lora_bwd_grouped_dropout.restype = ctypes.c_int
_lib.dsv_timing_enable.argtypes = [_i32]
_lib.dsv_timing_enable.restype = ctypes.c_int
_lib.dsv_timing_read.argtypes = [ctypes.POINTER(ctypes.c_double), _i32p,
                                 ctypes.POINTER(ctypes.c_double), _i32p]
_lib.dsv_timing_read.restype = ctypes.c_int
class AdamWHparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double)]


_lib.dsv_adamw_step.argtypes = [_vp, ctypes.c_int, _i32, _i32, _i32, ctypes.POINTER(AdamWHparams)] + [_vp] * 11
_lib.dsv_adamw_step.restype = ctypes.c_int


class AdamWProj(ctypes.Structure):
    _fields_ = [("K", _i32), ("N", _i32)] + [(n, _vp) for n in (
        "dA", "dB", "A_master", "B_master", "A_m", "A_v", "B_m", "B_v", "A", "B")]


_lib.dsv_adamw_step_grouped.argtypes = [_vp, ctypes.c_int, _i32, ctypes.POINTER(AdamWProj), _i32,
                                        ctypes.POINTER(AdamWHparams), _vp]
_lib.dsv_adamw_step_grouped.restype = ctypes.c_int
_lib.dsv_gemm_config.argtypes = [_vp, ctypes.c_int, _i32, _i32, _i32, _i32p]
_lib.dsv_gemm_config.restype = ctypes.c_int
_lib.dsv_status_string.argtypes = [ctypes.c_int]
_lib.dsv_status_string.restype = ctypes.c_char_p

COUNT_NAMES = ("fwd_tiles", "shrink_items", "gathered_rows", "gather_items", "bwd_tiles",
               "chunks", "train_adapters", "train_items", "fwd_tiles128", "bwd_tiles128")


class DsvError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s: %s" % (what, _lib.dsv_status_string(status).decode()))


def _check(rc: int, what: str):
    if rc != OK:
        raise DsvError(rc, what)


def lib_handle() -> ctypes.CDLL:
    return _lib


def _stream_handle(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(int(stream.cuda_stream))


def _ptr(t) -> ctypes.c_void_p:
    return ctypes.c_void_p(0 if t is None else int(t.data_ptr()))


def row_stride(n: int, dtype_code: int = 0) -> int:
    """dsv_row_stride: the row stride (elements) recommended for buffers with rows of n elements."""
    return int(_lib.dsv_row_stride(int(n), int(dtype_code)))


def _ld(t, row_len: int) -> int:
    """The row stride a grouped call passes for tensor t: 0 when t is dense, else t.stride(0).
    The elements of a row must be contiguous."""
    if t is None or t.is_contiguous():
        return 0
    if t.dim() != 2 or t.shape[1] != row_len or t.stride(1) != 1:
        raise ValueError("a strided operand must be 2-D with contiguous rows of %d elements" % row_len)
    return int(t.stride(0))


def _dense(*ts):
    """The single-projection calls take dense buffers only (the grouped calls take row strides)."""
    for t in ts:
        if t is not None and not t.is_contiguous():
            raise ValueError("non-contiguous operand: the single-projection calls take dense buffers; "
                             "pass row-strided operands to the grouped calls")


class Plan:
    """A packed segment table.  device=None builds a host-only plan (inspection only)."""

    def __init__(self, segments: Sequence[Sequence[int]], n_tokens: int, ranks, scales, r_max: int,
                 device=None, stream=None):
        seg = np.ascontiguousarray(np.asarray(segments, np.int32).reshape(-1, 4))
        self.segments = seg
        self.n_tokens = int(n_tokens)
        self.ranks = np.ascontiguousarray(np.asarray(ranks, np.int32))
        self.scales = np.ascontiguousarray(np.asarray(scales, np.float32))
        self.r_max = int(r_max)
        self._h = ctypes.c_void_p()
        self.meta = None
        nbytes = _sz(0)
        args = (seg.ctypes.data_as(_i32p), seg.shape[0], self.n_tokens,
                self.ranks.ctypes.data_as(_i32p), self.scales.ctypes.data_as(_f32p),
                self.ranks.shape[0], self.r_max)
        if device is None:
            _check(_lib.dsv_segments_build(*args, None, ctypes.byref(nbytes), None,
                                           ctypes.byref(self._h)), "dsv_segments_build")
        else:
            import torch
            _check(_lib.dsv_segments_build(*args, None, ctypes.byref(nbytes), None, None),
                   "dsv_segments_build (size query)")
            self.meta = torch.empty(max(int(nbytes.value), 256), dtype=torch.uint8, device=device)
            _check(_lib.dsv_segments_build(*args, _ptr(self.meta), ctypes.byref(nbytes),
                                           _stream_handle(stream), ctypes.byref(self._h)),
                   "dsv_segments_build")
        self.meta_bytes = int(nbytes.value)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:  # _lib is None at interpreter exit
            _lib.dsv_plan_free(h)
            self._h = ctypes.c_void_p()

    @property
    def handle(self):
        return self._h

    @property
    def train_tokens(self) -> int:
        return int(_lib.dsv_plan_train_rows(self._h))

    def train_rows(self) -> np.ndarray:
        out = np.zeros(max(self.train_tokens, 1), np.int32)
        n = _lib.dsv_plan_train_row_index(self._h, out.ctypes.data_as(_i32p))
        if n < 0:
            raise DsvError(n, "dsv_plan_train_row_index")
        return out[:n]

    def gathered_rows(self) -> np.ndarray:
        out = np.zeros(max(self.n_tokens, 1), np.int32)
        n = _lib.dsv_plan_gathered_rows(self._h, out.ctypes.data_as(_i32p))
        if n < 0:
            raise DsvError(n, "dsv_plan_gathered_rows")
        return out[:n]

    def meta_words(self) -> np.ndarray:
        out = np.zeros(self.meta_bytes // 4, np.int32)
        _check(_lib.dsv_plan_meta_copy(self._h, out.ctypes.data, self.meta_bytes), "dsv_plan_meta_copy")
        return out

    def counts(self) -> dict:
        out = np.zeros(len(COUNT_NAMES), np.int32)
        _check(_lib.dsv_plan_counts(self._h, out.ctypes.data_as(_i32p)), "dsv_plan_counts")
        return dict(zip(COUNT_NAMES, (int(v) for v in out)))


def segments_build(segments, n_tokens, ranks, scales, r_max, device=None, stream=None) -> Plan:
    return Plan(segments, n_tokens, ranks, scales, r_max, device=device, stream=stream)


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError("dsv supports bfloat16 and float32 tensors, got %s" % t.dtype)


def fwd_workspace_bytes(plan: Plan, dtype_code: int, K: int, N: int) -> int:
    n = _sz(0)
    _check(_lib.dsv_cobatch_fwd_workspace(plan.handle, dtype_code, K, N, ctypes.byref(n)),
           "dsv_cobatch_fwd_workspace")
    return int(n.value)


def bwd_workspace_bytes(plan: Plan, dtype_code: int, K: int, N: int, dropout: bool = False) -> int:
    n = _sz(0)
    if dropout:
        _check(_lib.dsv_lora_bwd_dropout_workspace(plan.handle, dtype_code, K, N, ctypes.byref(n)),
               "dsv_lora_bwd_dropout_workspace")
    else:
        _check(_lib.dsv_lora_bwd_workspace(plan.handle, dtype_code, K, N, ctypes.byref(n)),
               "dsv_lora_bwd_workspace")
    return int(n.value)


def _dropout(dropout):
    """(p, seed, offset) or (p, seed, offset, mask) -> the C struct (None stays None).
    mask: a device int32 tensor of T_t * ceil(K / 32) words the forward fills and the
    backward reads (dsv_dropout.mask), or None."""
    if dropout is None:
        return None
    p, seed, offset = dropout[:3]
    mask = dropout[3] if len(dropout) > 3 else None
    return Dropout(float(p), int(seed), int(offset), None if mask is None else ctypes.c_void_p(mask.data_ptr()))


def dropout_mask_words(plan: "Plan", K: int) -> int:
    """32-bit words of a projection's dropout mask buffer (T_t * ceil(K / 32))."""
    return plan.train_tokens * ((K + 31) // 32)


def _workspace(nbytes, device, given):
    import torch
    if given is not None:
        return given
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def cobatch_fwd(plan: Plan, X, W, A, B, Y=None, H_save=None, workspace=None, stream=None,
                keep_h: bool = True, dropout=None):
    """Y = X W^T + s_a (X A_a^T) B_a^T per row; H_save = X A_a^T of the training rows
    (keep_h=False keeps none: lora_bwd with H_save=None recomputes it from X).
    dropout=(p, seed, offset): LoRA dropout on the training rows' adapter input
    (dsv_cobatch_fwd_dropout)."""
    import torch
    _dense(X, W, A, B, Y, H_save)
    dt = _dtype_code(X)
    T, K = X.shape
    N = W.shape[0]
    if Y is None:
        Y = torch.empty((T, N), dtype=X.dtype, device=X.device)
    if H_save is None and plan.train_tokens > 0 and keep_h:
        H_save = torch.empty((plan.train_tokens, plan.r_max), dtype=X.dtype, device=X.device)
    ws = _workspace(fwd_workspace_bytes(plan, dt, K, N), X.device, workspace)
    d = _dropout(dropout)
    if d is None:
        _check(_lib.dsv_cobatch_fwd(plan.handle, dt, K, N, _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(Y),
                                    _ptr(H_save), _ptr(ws), ws.numel() * ws.element_size(),
                                    _stream_handle(stream)), "dsv_cobatch_fwd")
    else:
        _check(_lib.dsv_cobatch_fwd_dropout(plan.handle, dt, K, N, _ptr(X), _ptr(W), _ptr(A), _ptr(B),
                                            _ptr(Y), _ptr(H_save), ctypes.byref(d), _ptr(ws),
                                            ws.numel() * ws.element_size(), _stream_handle(stream)),
               "dsv_cobatch_fwd_dropout")
    return Y, H_save


def cobatch_fwd_noalloc(plan: Plan, X, W, A, B, Y, H_save=None, stream=None):
    """dsv_cobatch_fwd_noalloc: the forward with the library's device scratch as
    workspace (no device allocation in the call).  The caller passes the outputs:
    Y [T][N] and, when the batch has training rows, H_save [T_t][r_max] (or None
    to keep nothing).  Returns (Y, H_save)."""
    _dense(X, W, A, B, Y, H_save)
    dt = _dtype_code(X)
    K = X.shape[1]
    N = W.shape[0]
    _check(_lib.dsv_cobatch_fwd_noalloc(plan.handle, dt, K, N, _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(Y),
                                        _ptr(H_save), _stream_handle(stream)), "dsv_cobatch_fwd_noalloc")
    return Y, H_save


def lora_bwd(plan: Plan, X, W, A, B, H_save, dY, dA=None, dB=None, dX=None, want_dx=True,
             accumulate: bool = False, workspace=None, stream=None, dropout=None):
    """LoRA gradients of the training rows: dA, dB (fp32) and dX.  dropout=(p, seed,
    offset) must repeat the forward's (dsv_lora_bwd_dropout)."""
    import torch
    _dense(X, W, A, B, H_save, dY, dA, dB, dX)
    dt = _dtype_code(X)
    T, K = X.shape
    N = W.shape[0]
    n_ad = A.shape[0]
    if dA is None:
        dA = torch.zeros((n_ad, plan.r_max, K), dtype=torch.float32, device=X.device)
    if dB is None:
        dB = torch.zeros((n_ad, N, plan.r_max), dtype=torch.float32, device=X.device)
    if dX is None and want_dx and plan.train_tokens > 0:
        dX = torch.empty((plan.train_tokens, K), dtype=X.dtype, device=X.device)
    d = _dropout(dropout)
    ws = _workspace(bwd_workspace_bytes(plan, dt, K, N, d is not None), X.device, workspace)
    if d is None:
        _check(_lib.dsv_lora_bwd(plan.handle, dt, K, N, _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(H_save),
                                 _ptr(dY), _ptr(dA), _ptr(dB), _ptr(dX if want_dx else None),
                                 1 if accumulate else 0, _ptr(ws), ws.numel() * ws.element_size(),
                                 _stream_handle(stream)), "dsv_lora_bwd")
    else:
        _check(_lib.dsv_lora_bwd_dropout(plan.handle, dt, K, N, _ptr(X), _ptr(W), _ptr(A), _ptr(B),
                                         _ptr(H_save), _ptr(dY), _ptr(dA), _ptr(dB),
                                         _ptr(dX if want_dx else None), 1 if accumulate else 0,
                                         ctypes.byref(d), _ptr(ws), ws.numel() * ws.element_size(),
                                         _stream_handle(stream)), "dsv_lora_bwd_dropout")
    return dA, dB, dX


def _fwd_projs(items):
    arr = (FwdProj * len(items))()
    for i, (X, W, A, B, Y, H) in enumerate(items):
        K, N = X.shape[1], W.shape[0]
        _dense(A, B, H)
        arr[i] = FwdProj(K, N, _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(Y), _ptr(H), _ld(X, K), _ld(W, K),
                         _ld(Y, N))
    return arr


def fwd_grouped_workspace_bytes(plan: Plan, dtype_code: int, shapes) -> int:
    """shapes: [(K, N)] of the projections."""
    arr = (FwdProj * len(shapes))()
    for i, (K, N) in enumerate(shapes):
        arr[i].K, arr[i].N = K, N
    n = _sz(0)
    _check(_lib.dsv_cobatch_fwd_grouped_workspace(plan.handle, dtype_code, len(shapes), arr, ctypes.byref(n)),
           "dsv_cobatch_fwd_grouped_workspace")
    return int(n.value)


def bwd_grouped_workspace_bytes(plan: Plan, dtype_code: int, shapes) -> int:
    arr = (BwdProj * len(shapes))()
    for i, (K, N) in enumerate(shapes):
        arr[i].K, arr[i].N = K, N
    n = _sz(0)
    _check(_lib.dsv_lora_bwd_grouped_workspace(plan.handle, dtype_code, len(shapes), arr, ctypes.byref(n)),
           "dsv_lora_bwd_grouped_workspace")
    return int(n.value)


def _dropouts(dropouts, n):
    """[(p, seed, offset)] * n -> C array (None stays None)."""
    if dropouts is None:
        return None
    if len(dropouts) != n:
        raise ValueError("one dropout per projection")
    arr = (Dropout * n)()
    for i, d in enumerate(dropouts):
        arr[i] = _dropout(d)
    return arr


def cobatch_fwd_grouped(plan: Plan, projs, workspace=None, stream=None, keep_h: bool = True, dropouts=None):
    """dsv_cobatch_fwd_grouped.  projs: [(X, W, A, B)] or [(X, W, A, B, Y, H_save)];
    returns [(Y, H_save)] in the same order.  dropouts: one (p, seed, offset) per
    projection (dsv_cobatch_fwd_grouped_dropout)."""
    import torch
    items = []
    for pr in projs:
        X, W, A, B = pr[:4]
        Y = pr[4] if len(pr) > 4 and pr[4] is not None else torch.empty((X.shape[0], W.shape[0]), dtype=X.dtype,
                                                                          device=X.device)
        H = pr[5] if len(pr) > 5 else None
        if H is None and keep_h and plan.train_tokens > 0:
            H = torch.empty((plan.train_tokens, plan.r_max), dtype=X.dtype, device=X.device)
        items.append((X, W, A, B, Y, H))
    dt = _dtype_code(items[0][0])
    ws = _workspace(fwd_grouped_workspace_bytes(plan, dt, [(it[0].shape[1], it[1].shape[0]) for it in items]),
                    items[0][0].device, workspace)
    arr = _fwd_projs(items)
    dr = _dropouts(dropouts, len(items))
    if dr is None:
        _check(_lib.dsv_cobatch_fwd_grouped(plan.handle, dt, len(items), arr, _ptr(ws),
                                            ws.numel() * ws.element_size(), _stream_handle(stream)),
               "dsv_cobatch_fwd_grouped")
    else:
        _check(_lib.dsv_cobatch_fwd_grouped_dropout(plan.handle, dt, len(items), arr, dr, _ptr(ws),
                                                    ws.numel() * ws.element_size(), _stream_handle(stream)),
               "dsv_cobatch_fwd_grouped_dropout")
    return [(it[4], it[5]) for it in items]


def lora_bwd_grouped(plan: Plan, projs, accumulate: bool = False, want_dx: bool = True, workspace=None,
                     stream=None, dropouts=None, wts=None):
    """dsv_lora_bwd_grouped.  projs: [(X, W, A, B, H_save, dY)] or with (dA, dB, dX) appended;
    returns [(dA, dB, dX)].  wts: optional transposed weights [K][N] per projection (or None
    entries)."""
    import torch
    items = []
    for pr in projs:
        X, W, A, B, H, dY = pr[:6]
        K, N, n_ad = X.shape[1], W.shape[0], A.shape[0]
        dA = pr[6] if len(pr) > 6 and pr[6] is not None else torch.zeros((n_ad, plan.r_max, K), dtype=torch.float32,
                                                                          device=X.device)
        dB = pr[7] if len(pr) > 7 and pr[7] is not None else torch.zeros((n_ad, N, plan.r_max), dtype=torch.float32,
                                                                          device=X.device)
        dX = pr[8] if len(pr) > 8 else None
        if dX is None and want_dx and plan.train_tokens > 0:
            dX = torch.empty((plan.train_tokens, K), dtype=X.dtype, device=X.device)
        items.append((X, W, A, B, H, dY, dA, dB, dX if want_dx else None))
    dt = _dtype_code(items[0][0])
    ws = _workspace(bwd_grouped_workspace_bytes(plan, dt, [(it[0].shape[1], it[1].shape[0]) for it in items]),
                    items[0][0].device, workspace)
    arr = (BwdProj * len(items))()
    for i, (X, W, A, B, H, dY, dA, dB, dX) in enumerate(items):
        Wt = wts[i] if wts is not None else None
        K, N = X.shape[1], W.shape[0]
        _dense(A, B, H, dA, dB)
        arr[i] = BwdProj(K, N, _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(H), _ptr(dY), _ptr(dA), _ptr(dB), _ptr(dX),
                         _ptr(Wt), _ld(X, K), _ld(W, K), _ld(dY, N), _ld(dX, K), _ld(Wt, N))
    dr = _dropouts(dropouts, len(items))
    if dr is None:
        _check(_lib.dsv_lora_bwd_grouped(plan.handle, dt, len(items), arr, 1 if accumulate else 0, _ptr(ws),
                                         ws.numel() * ws.element_size(), _stream_handle(stream)),
               "dsv_lora_bwd_grouped")
    else:
        _check(_lib.dsv_lora_bwd_grouped_dropout(plan.handle, dt, len(items), arr, 1 if accumulate else 0, dr,
                                                 _ptr(ws), ws.numel() * ws.element_size(), _stream_handle(stream)),
               "dsv_lora_bwd_grouped_dropout")
    return [(it[6], it[7], it[8]) for it in items]


def adamw_step(plan: Plan, step: int, dA, dB, A_master, B_master, A_m, A_v, B_m, B_v, A=None, B=None,
               lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, stream=None):
    """One fused AdamW step of the plan's training adapters (dsv_adamw_step); updates
    the fp32 masters and moments in place and writes the rounded copy into A / B."""
    import torch
    K = A_master.shape[2]
    N = B_master.shape[1]
    ref = A if A is not None else A_master
    code = BF16 if ref.dtype == torch.bfloat16 else F32
    hp = AdamWHparams(lr, beta1, beta2, eps, weight_decay)
    ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())  # noqa: E731
    _check(_lib.dsv_adamw_step(plan.handle, code, K, N, step, ctypes.byref(hp), ptr(dA), ptr(dB),
                               ptr(A_master), ptr(B_master), ptr(A_m), ptr(A_v), ptr(B_m), ptr(B_v),
                               ptr(A), ptr(B), _stream_handle(stream)),
           "dsv_adamw_step")


def adamw_step_grouped(plan: Plan, step: int, items, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                       weight_decay=0.01, stream=None):
    """The AdamW step of several projections in one launch (dsv_adamw_step_grouped).
    items: [(dA, dB, A_master, B_master, A_m, A_v, B_m, B_v, A, B)], A / B may be None."""
    adamw_grouped_prepared(plan, items, lr, beta1, beta2, eps, weight_decay, stream)(step)


def adamw_grouped_prepared(plan: Plan, items, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                           weight_decay=0.01, stream=None):
    """Marshal the arguments of dsv_adamw_step_grouped once; returns step(t), which
    only makes the call (for loops that repeat it over the same buffers)."""
    import torch
    arr = (AdamWProj * len(items))()
    code = None
    ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())  # noqa: E731
    for i, it in enumerate(items):
        dA, dB, Am, Bm, mA, vA, mB, vB, A, B = it
        ref = A if A is not None else Am
        c = BF16 if ref.dtype == torch.bfloat16 else F32
        if code is None:
            code = c
        elif c != code:
            raise ValueError("adamw_step_grouped: parameter copies of one dtype")
        arr[i] = AdamWProj(Am.shape[2], Bm.shape[1], *[ptr(t) for t in (dA, dB, Am, Bm, mA, vA, mB, vB, A, B)])
    hp = AdamWHparams(lr, beta1, beta2, eps, weight_decay)
    args = (plan.handle, code if code is not None else BF16, len(items), arr)
    tail = (ctypes.byref(hp), _stream_handle(stream))

    def step(t: int) -> None:
        _check(_lib.dsv_adamw_step_grouped(*args, t, *tail), "dsv_adamw_step_grouped")
    return step


GEMM_CONFIG_NAMES = ("tile_m", "tile_n", "row_tiles", "col_tiles", "split_tiles", "split_ways")


def gemm_config(plan: Plan, dtype_code: int, K: int, N: int, pass_: int) -> dict:
    """Tile shape and contraction split of the forward (pass_ 0) or dX (pass_ 1) GEMM."""
    out = (ctypes.c_int32 * 6)()
    _check(_lib.dsv_gemm_config(plan.handle, dtype_code, K, N, pass_, out), "dsv_gemm_config")
    return dict(zip(GEMM_CONFIG_NAMES, list(out)))


def timing_enable(on: bool = True):
    _check(_lib.dsv_timing_enable(1 if on else 0), "dsv_timing_enable")


def timing_read():
    """(fwd GEMM ms, fwd launches, dX GEMM ms, dX launches) since the last read."""
    fm, bm = ctypes.c_double(0), ctypes.c_double(0)
    fn, bn = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(_lib.dsv_timing_read(ctypes.byref(fm), ctypes.byref(fn), ctypes.byref(bm),
                                ctypes.byref(bn)), "dsv_timing_read")
    return fm.value, fn.value, bm.value, bn.value
