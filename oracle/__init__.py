"""CPU oracle for the EmbeddingBag training step (ctypes over liboracle.so).

TEST INFRASTRUCTURE ONLY: the test suite, the package smoke check and the
benchmark's CPU-baseline leg are its only callers.  It shares no code with
the GPU library and never touches a GPU.  See oracle.cpp for the definitions
it follows (Section II's L = A^T W, Algorithms 1-4 of Section III-A, the
Split-SGD-BF16 storage of Section VII).

All arrays are numpy, host-resident, C-contiguous:
  tables[t]  float32 [M_t, E]       (split: hi/lo uint16 [M_t, E])
  indices    int32   [NS]           table-local rows
  offsets    int32   [T*B + 1]      bag k = t*B + b is indices[O[k]:O[k+1]]
  pooled     float32 [T, B, E]
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# EMBBAG_ORACLE_LIB points the tests' mutation check at a deliberately broken
# build of oracle.cpp; normally unset.
_LIB_PATH = os.environ.get("EMBBAG_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_WORKSPACE = -2
ERR_INDEX_RANGE = -3
ERR_OFFSETS = -4

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = C.CDLL(_LIB_PATH)
        p, i32, i64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_float
        L.oracle_validate.argtypes = [i32, i32, i32, p, p, p, i64]
        L.oracle_forward.argtypes = [i32, i32, i32, p, p, p, p, i64, p]
        L.oracle_forward_literal.argtypes = [i32, i32, i32, p, p, p, p, i64, p]
        L.oracle_forward_split.argtypes = [i32, i32, i32, p, p, p, p, i64, p]
        L.oracle_dedup.argtypes = [i32, i32, p, p, p, i64, p, p, p, p, p]
        L.oracle_backward_sgd.argtypes = [p, i32, i32, i32, p, p, p, p, i64, f32]
        L.oracle_backward_sgd_literal.argtypes = [p, i32, i32, i32, p, p, p, p, i64, f32]
        L.oracle_backward_sgd_split.argtypes = [p, i32, i32, i32, p, p, p, p, p, i64, f32]
        L.oracle_forward_weighted.argtypes = [i32, i32, i32, p, p, p, p, i64, p, i32, p]
        L.oracle_backward_sgd_weighted.argtypes = [p, i32, i32, i32, p, p, p, p, i64, p, i32, f32]
        L.oracle_bf16_round.argtypes = [p, p, i64]
        L.oracle_bf16_widen.argtypes = [p, p, i64]
        L.oracle_forward_split_bf16_act.argtypes = [i32, i32, i32, p, p, p, p, i64, p]
        L.oracle_backward_sgd_split_bf16_act.argtypes = [p, i32, i32, i32, p, p, p, p, p, i64, f32]
        L.oracle_split.argtypes = [p, p, p, i64]
        L.oracle_combine.argtypes = [p, p, p, i64]
        L.oracle_split_roundtrip_mismatches.argtypes = [C.c_uint64, C.c_uint64]
        L.oracle_split_roundtrip_mismatches.restype = i64
        for name in ("oracle_validate", "oracle_forward", "oracle_forward_literal",
                     "oracle_forward_split", "oracle_dedup", "oracle_backward_sgd",
                     "oracle_backward_sgd_literal", "oracle_backward_sgd_split",
                     "oracle_forward_weighted", "oracle_backward_sgd_weighted",
                     "oracle_forward_split_bf16_act", "oracle_backward_sgd_split_bf16_act"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    a = np.asarray(a)
    if a.dtype != dtype or not a.flags.c_contiguous:
        raise TypeError(f"expected C-contiguous {np.dtype(dtype).name}, got {a.dtype}")
    return a


def _rows(tables):
    return np.array([t.shape[0] for t in tables], dtype=np.int64)


def _ptr_array(tables):
    arr = (C.c_void_p * max(1, len(tables)))()
    for i, t in enumerate(tables):
        arr[i] = t.ctypes.data
    return arr


def validate(rows, dim: int, batch: int, indices, offsets, num_tables: int | None = None,
             num_indices: int | None = None) -> int:
    rows = np.asarray(rows, dtype=np.int64)
    T = len(rows) if num_tables is None else num_tables
    I = None if indices is None else _c(indices, np.int32)
    O = None if offsets is None else _c(offsets, np.int32)
    NS = (0 if I is None else I.size) if num_indices is None else num_indices
    return lib().oracle_validate(T, batch, dim, _ptr(rows), _ptr(I), _ptr(O), NS)


def forward(tables, batch: int, indices, offsets, literal: bool = False):
    """Sum-pooled forward.  Returns (status, pooled[T, B, E]) (pooled zeros on error)."""
    tables = [_c(t, np.float32) for t in tables]
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    T, E = len(tables), tables[0].shape[1]
    rows = _rows(tables)
    Y = np.zeros((T, batch, E), dtype=np.float32)
    fn = lib().oracle_forward_literal if literal else lib().oracle_forward
    rc = fn(T, batch, E, _ptr(rows), _ptr_array(tables), _ptr(I), _ptr(O), I.size, _ptr(Y))
    return rc, Y


def forward_split(hi_tables, batch: int, indices, offsets):
    hi_tables = [_c(t, np.uint16) for t in hi_tables]
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    T, E = len(hi_tables), hi_tables[0].shape[1]
    rows = _rows(hi_tables)
    Y = np.zeros((T, batch, E), dtype=np.float32)
    rc = lib().oracle_forward_split(T, batch, E, _ptr(rows), _ptr_array(hi_tables), _ptr(I),
                                    _ptr(O), I.size, _ptr(Y))
    return rc, Y


def dedup(rows, batch: int, indices, offsets):
    """Integer work of the backward: stable sort of (key, bag) by key, unique keys.

    Returns (status, dict) with sorted_keys, sorted_bags (uint32 [NS]),
    unique_keys (uint32 [U]), seg_off (int32 [U+1]) and num_unique.
    """
    rows = np.asarray(rows, dtype=np.int64)
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    NS = I.size
    sk = np.zeros(NS, np.uint32)
    sb = np.zeros(NS, np.uint32)
    uk = np.zeros(NS, np.uint32)
    so = np.zeros(NS + 1, np.int32)
    nu = np.zeros(1, np.int64)
    rc = lib().oracle_dedup(len(rows), batch, _ptr(rows), _ptr(I), _ptr(O), NS, _ptr(sk),
                            _ptr(sb), _ptr(uk), _ptr(so), _ptr(nu))
    U = int(nu[0])
    return rc, dict(sorted_keys=sk, sorted_bags=sb, unique_keys=uk[:U], seg_off=so[:U + 1],
                    num_unique=U)


def backward_sgd(grad, batch: int, indices, offsets, lr: float, tables, literal: bool = False) -> int:
    """Fused backward + sparse SGD; updates ``tables`` in place.  Returns status."""
    tables = [_c(t, np.float32) for t in tables]
    G = _c(grad, np.float32)
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    T, E = len(tables), tables[0].shape[1]
    rows = _rows(tables)
    fn = lib().oracle_backward_sgd_literal if literal else lib().oracle_backward_sgd
    return fn(_ptr(G), T, batch, E, _ptr(rows), _ptr_array(tables), _ptr(I), _ptr(O), I.size, lr)


def backward_sgd_split(grad, batch: int, indices, offsets, lr: float, hi_tables, lo_tables) -> int:
    hi_tables = [_c(t, np.uint16) for t in hi_tables]
    lo_tables = [_c(t, np.uint16) for t in lo_tables]
    G = _c(grad, np.float32)
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    T, E = len(hi_tables), hi_tables[0].shape[1]
    rows = _rows(hi_tables)
    return lib().oracle_backward_sgd_split(_ptr(G), T, batch, E, _ptr(rows), _ptr_array(hi_tables),
                                           _ptr_array(lo_tables), _ptr(I), _ptr(O), I.size, lr)


POOL_SUM = 0
POOL_MEAN = 1


def forward_weighted(tables, batch: int, indices, offsets, weights=None, mode: int = POOL_SUM):
    """Weighted-sum (per-look-up weights) or mean pooling.  Returns (status, pooled)."""
    tables = [_c(t, np.float32) for t in tables]
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    a = None if weights is None else _c(weights, np.float32)
    T, E = len(tables), tables[0].shape[1]
    rows = _rows(tables)
    Y = np.zeros((T, batch, E), dtype=np.float32)
    rc = lib().oracle_forward_weighted(T, batch, E, _ptr(rows), _ptr_array(tables), _ptr(I),
                                       _ptr(O), I.size, _ptr(a), mode, _ptr(Y))
    return rc, Y


def backward_sgd_weighted(grad, batch: int, indices, offsets, lr: float, tables, weights=None,
                          mode: int = POOL_SUM) -> int:
    tables = [_c(t, np.float32) for t in tables]
    G = _c(grad, np.float32)
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    a = None if weights is None else _c(weights, np.float32)
    T, E = len(tables), tables[0].shape[1]
    rows = _rows(tables)
    return lib().oracle_backward_sgd_weighted(_ptr(G), T, batch, E, _ptr(rows), _ptr_array(tables),
                                              _ptr(I), _ptr(O), I.size, _ptr(a), mode, lr)


def bf16_round(x):
    """FP32 -> BF16 bit patterns (uint16), round to nearest, ties to even."""
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().oracle_bf16_round(_ptr(x), _ptr(out), x.size)
    return out


def bf16_widen(h):
    """BF16 bit patterns (uint16) -> FP32, exact."""
    h = _c(h, np.uint16)
    out = np.empty(h.shape, np.float32)
    lib().oracle_bf16_widen(_ptr(h), _ptr(out), h.size)
    return out


def forward_split_bf16_act(hi_tables, batch: int, indices, offsets):
    """Split forward with BF16 pooled outputs.  Returns (status, pooled uint16 [T, B, E])."""
    hi_tables = [_c(t, np.uint16) for t in hi_tables]
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    T, E = len(hi_tables), hi_tables[0].shape[1]
    rows = _rows(hi_tables)
    Y = np.zeros((T, batch, E), dtype=np.uint16)
    rc = lib().oracle_forward_split_bf16_act(T, batch, E, _ptr(rows), _ptr_array(hi_tables),
                                             _ptr(I), _ptr(O), I.size, _ptr(Y))
    return rc, Y


def backward_sgd_split_bf16_act(grad_bf16, batch: int, indices, offsets, lr: float, hi_tables,
                                lo_tables) -> int:
    """Split update driven by a BF16 gradient (uint16 bit patterns [T, B, E])."""
    hi_tables = [_c(t, np.uint16) for t in hi_tables]
    lo_tables = [_c(t, np.uint16) for t in lo_tables]
    G = _c(grad_bf16, np.uint16)
    I, O = _c(indices, np.int32), _c(offsets, np.int32)
    T, E = len(hi_tables), hi_tables[0].shape[1]
    rows = _rows(hi_tables)
    return lib().oracle_backward_sgd_split_bf16_act(_ptr(G), T, batch, E, _ptr(rows),
                                                    _ptr_array(hi_tables), _ptr_array(lo_tables),
                                                    _ptr(I), _ptr(O), I.size, lr)


def split(w):
    w = _c(w, np.float32)
    hi = np.empty(w.shape, np.uint16)
    lo = np.empty(w.shape, np.uint16)
    lib().oracle_split(_ptr(w), _ptr(hi), _ptr(lo), w.size)
    return hi, lo


def combine(hi, lo):
    hi, lo = _c(hi, np.uint16), _c(lo, np.uint16)
    w = np.empty(hi.shape, np.float32)
    lib().oracle_combine(_ptr(hi), _ptr(lo), _ptr(w), hi.size)
    return w


def split_roundtrip_mismatches(start: int, count: int) -> int:
    return int(lib().oracle_split_roundtrip_mismatches(start, count))
