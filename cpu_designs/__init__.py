"""The paper's multi-core CPU designs (Algorithm 1; Algorithms 2-4 fused with
row ownership), run on the host for context beside the GPU library.

Thin ctypes wrappers over ``libcpudesigns.so`` (``build.py``).  Tables are
C-contiguous float32 arrays of shape [M_t, E]; indices and offsets int32;
gradients float32 of shape [T, B, E].
"""
import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcpudesigns.so")
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built (python cpu_designs/build.py)")
        L = C.CDLL(LIB_PATH)
        p, i32, f32 = C.c_void_p, C.c_int32, C.c_float
        L.cpu_designs_threads.restype = C.c_int
        L.cpu_designs_forward.argtypes = [i32, i32, i32, p, p, p, p, i32]
        L.cpu_designs_backward_sgd.argtypes = [i32, i32, i32, p, p, p, p, p, f32, i32]
        _lib = L
    return _lib


def _tables(tables):
    for w in tables:
        if w.dtype != np.float32 or w.ndim != 2 or not w.flags.c_contiguous:
            raise ValueError("tables must be C-contiguous float32 [M, E] arrays")
    arr = (C.c_void_p * len(tables))(*[w.ctypes.data for w in tables])
    return arr


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data


def threads() -> int:
    return int(lib().cpu_designs_threads())


def forward(tables, batch: int, indices, offsets, nthreads: int):
    """Pooled sums [T, B, E] (float32); returns (status, Y)."""
    T, E = len(tables), int(tables[0].shape[1])
    Wp = _tables(tables)
    I, Ip = _i32(indices)
    O, Op = _i32(offsets)
    Y = np.empty((T, batch, E), dtype=np.float32)
    rc = lib().cpu_designs_forward(T, batch, E, Wp, Ip, Op, Y.ctypes.data, int(nthreads))
    return rc, Y


def backward_sgd(grad, batch: int, indices, offsets, lr: float, tables, nthreads: int) -> int:
    """Applies W <- W - lr * dW in place, the rows shared out by ownership."""
    T, E = len(tables), int(tables[0].shape[1])
    Wp = _tables(tables)
    I, Ip = _i32(indices)
    O, Op = _i32(offsets)
    rows = np.array([w.shape[0] for w in tables], dtype=np.int64)
    G = np.ascontiguousarray(grad, dtype=np.float32)
    if G.shape != (T, batch, E):
        raise ValueError("grad must be [T, B, E]")
    return int(lib().cpu_designs_backward_sgd(T, batch, E, rows.ctypes.data, Wp, Ip, Op,
                                              G.ctypes.data, C.c_float(lr), int(nthreads)))
