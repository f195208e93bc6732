"""MI355X (gfx950) EmbeddingBag training step — thin Python binding.

Argument marshalling only: every function takes torch tensors that live on
the GPU, passes their device pointers and the current HIP stream to the C ABI
of ``libembbag.so`` (declared in ``include/embbag.h``) and returns its status
code.  All computation happens in the library's HIP kernels; there is no CPU
path, and loading fails loudly when the library has not been built.  The
buffer sizes the C ABI takes on trust (table widths, offsets, activations,
outputs) are checked here against the call's sizes first (ValueError).
``Tables`` (FP32) and ``SplitTables`` (hi, lo) check a list of tables and
build its C descriptor once; every entry point accepts them where it takes a
list, which keeps a repeated call's host cost to the call itself.

Operators (arXiv 2005.04680): Algorithm 1 (sum-pooled forward), Algorithms
2-3 fused into one backward + sparse SGD update of the touched rows, and the
Split-SGD-BF16 storage of Section VII.
"""
from __future__ import annotations

import ctypes as C
import functools
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libembbag.so")

EMBBAG_OK = 0
EMBBAG_ERR_INVALID_ARG = -1
EMBBAG_ERR_WORKSPACE = -2
EMBBAG_ERR_INDEX_RANGE = -3
EMBBAG_ERR_OFFSETS = -4
EMBBAG_ERR_HIP = -5
EMBBAG_POOL_SUM = 0
EMBBAG_POOL_MEAN = 1
EMBBAG_NOALLOC_SCRATCH_BYTES = 64 << 20  # the no-allocation entry point's fixed workspace


class EmbbagError(RuntimeError):
    def __init__(self, code: int, where: str = ""):
        super().__init__(f"{where}: {embbag_status_string(code)} ({code})")
        self.code = code


class _Tables(C.Structure):
    _fields_ = [("num_tables", C.c_int32), ("dim", C.c_int32),
                ("rows", C.POINTER(C.c_int64)), ("weights", C.POINTER(C.c_void_p))]


class _SplitTables(C.Structure):
    _fields_ = [("num_tables", C.c_int32), ("dim", C.c_int32),
                ("rows", C.POINTER(C.c_int64)), ("hi", C.POINTER(C.c_void_p)),
                ("lo", C.POINTER(C.c_void_p))]


_lib = None


def lib():
    """The loaded libembbag.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2005_04680_amd.build` (hipcc, gfx950)")
        L = C.CDLL(LIB_PATH)
        p, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
        L.embbag_status_string.argtypes = [C.c_int]
        L.embbag_status_string.restype = C.c_char_p
        L.embbag_forward.argtypes = [p, i32, p, p, i64, p, p, p]
        L.embbag_forward_split_bf16.argtypes = [p, i32, p, p, i64, p, p, p]
        L.embbag_backward_workspace_bytes.argtypes = [i32, i32, i64, i32]
        L.embbag_backward_workspace_bytes.restype = sz
        L.embbag_backward_sgd.argtypes = [p, i32, p, p, i64, C.c_float, p, p, sz, p, p]
        L.embbag_backward_sgd_split_bf16.argtypes = [p, i32, p, p, i64, C.c_float, p, p, sz, p, p]
        L.embbag_forward_pooled.argtypes = [p, i32, p, p, i64, p, i32, p, p, p]
        L.embbag_backward_sgd_pooled.argtypes = [p, i32, p, p, i64, p, i32, C.c_float, p, p, sz,
                                                 p, p]
        L.embbag_backward_prepare.argtypes = [i32, p, i32, i32, p, p, i64, p, sz, p, p]
        L.embbag_backward_prepare_pooled.argtypes = [i32, p, i32, i32, p, p, i64, p, i32, p, sz,
                                                     p, p]
        L.embbag_backward_apply_sgd_pooled.argtypes = [p, i32, p, i64, p, i32, C.c_float, p, p,
                                                       sz, p]
        L.embbag_backward_apply_sgd.argtypes = [p, i32, i64, C.c_float, p, p, sz, p]
        L.embbag_backward_apply_sgd_split_bf16.argtypes = [p, i32, i64, C.c_float, p, p, sz, p]
        L.embbag_forward_split_bf16_act.argtypes = [p, i32, p, p, i64, p, p, p]
        L.embbag_backward_sgd_split_bf16_act.argtypes = [p, i32, p, p, i64, C.c_float, p, p, sz,
                                                         p, p]
        L.embbag_backward_apply_sgd_split_bf16_act.argtypes = [p, i32, i64, C.c_float, p, p, sz, p]
        L.embbag_split_fp32.argtypes = [p, p, p, i64, p]
        L.embbag_combine_fp32.argtypes = [p, p, p, i64, p]
        L.embbag_dedup_workspace_bytes.argtypes = [i32, i32, i64]
        L.embbag_dedup_workspace_bytes.restype = sz
        L.embbag_dedup.argtypes = [i32, p, i32, p, p, i64, p, p, p, p, p, p, sz, p, p]
        L.embbag_baseline_materialize.argtypes = [p, i32, i32, i32, p, i64, p, p, p]
        L.embbag_baseline_update_atomic.argtypes = [p, i32, p, p, i64, C.c_float, p, p, p]
        L.embbag_baseline_backward_sgd_atomic.argtypes = [p, i32, p, p, i64, C.c_float, p, p, p]
        L.embbag_baseline_update_owner.argtypes = [p, i32, p, p, i64, C.c_float, p, i32, p]
        L.embbag_baseline_touch_rows.argtypes = [i32, i64, p, p, sz, p]
        L.embbag_baseline_touch_rows_split.argtypes = [i32, i64, p, p, sz, p]
        L.embbag_status_read.argtypes = [p, p]
        L.embbag_backward_sgd_noalloc.argtypes = [p, i32, p, p, i64, C.c_float, p, p, p]
        for n in ("embbag_forward", "embbag_forward_split_bf16", "embbag_backward_sgd",
                  "embbag_backward_sgd_split_bf16", "embbag_backward_prepare",
                  "embbag_forward_pooled", "embbag_backward_sgd_pooled",
                  "embbag_backward_prepare_pooled", "embbag_backward_apply_sgd_pooled",
                  "embbag_backward_apply_sgd", "embbag_backward_apply_sgd_split_bf16",
                  "embbag_forward_split_bf16_act", "embbag_backward_sgd_split_bf16_act",
                  "embbag_backward_apply_sgd_split_bf16_act",
                  "embbag_split_fp32", "embbag_combine_fp32", "embbag_dedup",
                  "embbag_baseline_materialize", "embbag_baseline_update_atomic",
                  "embbag_baseline_backward_sgd_atomic", "embbag_baseline_update_owner",
                  "embbag_baseline_touch_rows", "embbag_baseline_touch_rows_split",
                  "embbag_status_read",
                  "embbag_backward_sgd_noalloc"):
            getattr(L, n).restype = C.c_int
        _lib = L
    return _lib


def embbag_status_string(code: int) -> str:
    return lib().embbag_status_string(int(code)).decode()


def check(code: int, where: str = "embbag") -> None:
    if code != EMBBAG_OK:
        raise EmbbagError(code, where)


# ---- marshalling helpers ---------------------------------------------------
def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _ptr(t, dtypes=None, name="tensor"):
    """Device pointer of a contiguous GPU tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    return t.data_ptr()


@functools.lru_cache(maxsize=None)
def _dt(*names):
    import torch
    return tuple(getattr(torch, n) for n in names if hasattr(torch, n))


# Buffer shapes the C ABI assumes but cannot check (it takes raw pointers): a
# table narrower than `dim`, or an offsets, activation or output buffer shorter
# than its sizes imply, would let a kernel read or write past its end.  These
# checks raise ValueError before any library call.  Sizes the library itself
# rejects (a negative batch, no tables) are left to its status codes.
def _need(ok, msg):
    if not ok:
        raise ValueError(msg)


def _check_bags(T, batch, offsets):
    if offsets is not None and T >= 1 and batch >= 0:
        _need(offsets.numel() == T * batch + 1,
              f"offsets: {offsets.numel()} entries, expected num_tables * batch + 1 = "
              f"{T * batch + 1}")


def _check_numel(t, n, name, exact=True):
    if t is not None and n >= 0:
        ok = t.numel() == n if exact else t.numel() >= n
        _need(ok, f"{name}: {t.numel()} elements, expected {'' if exact else 'at least '}{n}")


def _check_act(t, T, batch, dim, name):
    if T >= 1 and batch >= 0:
        _check_numel(t, T * batch * dim, f"{name} (num_tables x batch x dim)")


def _check_tables(tables, what="table"):
    if isinstance(tables, (Tables, SplitTables)):
        return tables.dim
    if len(tables) == 0:
        return 0
    dim = int(tables[0].shape[1]) if len(tables[0].shape) == 2 else -1
    for i, t in enumerate(tables):
        _need(len(t.shape) == 2 and int(t.shape[1]) == dim,
              f"{what} {i}: shape {tuple(t.shape)}, expected 2-D with {dim} columns like {what} 0")
    return dim


_FP32_TABLES = object()  # _tables_struct's default: an FP32 entry point


def _tables_struct(tables, split_lo=_FP32_TABLES):
    """The C table descriptor (and the objects it points into) of FP32
    tables, or of split tables when `split_lo` is given (None when `tables`
    is a SplitTables)."""
    fp32 = split_lo is _FP32_TABLES
    if isinstance(tables, Tables):
        if not fp32:
            raise TypeError("FP32 Tables given where split tables (hi, lo) are expected")
        return tables.struct, tables
    if isinstance(tables, SplitTables):
        if fp32:
            raise TypeError("SplitTables given where FP32 tables are expected")
        return tables.struct, tables
    if fp32:
        split_lo = None
    else:
        _need(split_lo is not None, "split tables need their lo halves")
    import torch
    T = len(tables)
    _check_tables(tables, "table" if split_lo is None else "hi table")
    if split_lo is not None:
        _need(len(split_lo) == T, f"{len(split_lo)} lo tables for {T} hi tables")
        for i, (h, l) in enumerate(zip(tables, split_lo)):
            _need(tuple(l.shape) == tuple(h.shape),
                  f"lo table {i}: shape {tuple(l.shape)} differs from its hi half {tuple(h.shape)}")
    rows = (C.c_int64 * max(T, 1))(*[int(t.shape[0]) for t in tables])
    dim = int(tables[0].shape[1]) if T else 0
    ptrs = (C.c_void_p * max(T, 1))(*[_ptr(t, None, "table") for t in tables])
    keep = [rows, ptrs]
    if split_lo is None:
        for t in tables:
            if t.dtype != torch.float32:
                raise TypeError("FP32 tables expected")
        s = _Tables(T, dim, C.cast(rows, C.POINTER(C.c_int64)), C.cast(ptrs, C.POINTER(C.c_void_p)))
    else:
        lo = (C.c_void_p * max(T, 1))(*[_ptr(t, None, "lo table") for t in split_lo])
        keep.append(lo)
        s = _SplitTables(T, dim, C.cast(rows, C.POINTER(C.c_int64)),
                         C.cast(ptrs, C.POINTER(C.c_void_p)), C.cast(lo, C.POINTER(C.c_void_p)))
    return s, keep


def _split_struct_fwd(hi):
    if isinstance(hi, SplitTables):
        return hi.struct, hi
    if isinstance(hi, Tables):
        raise TypeError("FP32 Tables given where split tables are expected")
    T = len(hi)
    _check_tables(hi, "hi table")
    rows = (C.c_int64 * max(T, 1))(*[int(t.shape[0]) for t in hi])
    ptrs = (C.c_void_p * max(T, 1))(*[_ptr(t, None, "hi table") for t in hi])
    s = _SplitTables(T, int(hi[0].shape[1]) if T else 0, C.cast(rows, C.POINTER(C.c_int64)),
                     C.cast(ptrs, C.POINTER(C.c_void_p)), None)
    return s, [rows, ptrs]


class Tables:
    """FP32 tables (a list of [M_t, E] GPU tensors) with their C descriptor
    checked and built once.  Every entry point that takes a list of tables
    also takes a Tables, and then skips rebuilding the descriptor: the
    per-call cost of the binding drops to the argument checks of the other
    buffers.  The tensors must keep their storage while it is in use."""

    def __init__(self, weights):
        self.tensors = list(weights)
        self.dim = _check_tables(self.tensors)
        self.struct, self._keep = _tables_struct(self.tensors)
        self.rows_addr = C.cast(self.struct.rows, C.c_void_p).value

    def __len__(self):
        return len(self.tensors)

    def __getitem__(self, i):
        return self.tensors[i]

    def __iter__(self):
        return iter(self.tensors)


class SplitTables:
    """Split tables (BF16 high halves `hi`, 16-bit low halves `lo`) with their
    C descriptor built once; taken wherever `hi` is (its `lo` argument is
    then ignored)."""

    def __init__(self, hi, lo):
        self.hi, self.lo = list(hi), list(lo)
        self.dim = _check_tables(self.hi, "hi table")
        self.struct, self._keep = _tables_struct(self.hi, split_lo=self.lo)
        self.rows_addr = C.cast(self.struct.rows, C.c_void_p).value

    def __len__(self):
        return len(self.hi)

    def __getitem__(self, i):
        return self.hi[i]

    def __iter__(self):
        return iter(self.hi)


def _rows_arg(rows):
    """Rows per table as the C ABI takes them (a pointer to int64s), with the
    array it points into: built from a list of ints, or the descriptor's own
    when given Tables or SplitTables."""
    if isinstance(rows, (Tables, SplitTables)):
        return rows.rows_addr, rows
    r = (C.c_int64 * max(len(rows), 1))(*[int(x) for x in rows])
    return C.cast(r, C.c_void_p), r


_I32 = ("int32",)


def _status_ptr(d_status):
    _check_numel(d_status, 1, "d_status", exact=False)
    return _ptr(d_status, _dt(*_I32), "d_status")
_U16 = ("uint16", "int16")
_U32 = ("uint32", "int32")


# ---- entry points (same names as the C ABI) --------------------------------
def embbag_forward(weights, batch, indices, offsets, pooled_out, d_status=None, stream=None) -> int:
    """Algorithm 1 over FP32 tables ``weights`` (list of [M_t, E] tensors)."""
    _check_bags(len(weights), batch, offsets)
    _check_act(pooled_out, len(weights), batch, _check_tables(weights), "pooled_out")
    s, keep = _tables_struct(weights)
    return lib().embbag_forward(C.byref(s), int(batch), _ptr(indices, _dt(*_I32), "indices"),
                                _ptr(offsets, _dt(*_I32), "offsets"), int(indices.numel()),
                                _ptr(pooled_out, _dt("float32"), "pooled_out"),
                                _status_ptr(d_status), _stream(stream))


def embbag_forward_pooled(weights, batch, indices, offsets, pooled_out, per_sample_weights=None,
                          pooling=EMBBAG_POOL_SUM, d_status=None, stream=None) -> int:
    """Weighted-sum (one weight per look-up) or mean pooling over FP32 tables."""
    _check_bags(len(weights), batch, offsets)
    _check_act(pooled_out, len(weights), batch, _check_tables(weights), "pooled_out")
    _check_numel(per_sample_weights, indices.numel(), "per_sample_weights")
    s, keep = _tables_struct(weights)
    return lib().embbag_forward_pooled(C.byref(s), int(batch), _ptr(indices, _dt(*_I32), "indices"),
                                       _ptr(offsets, _dt(*_I32), "offsets"), int(indices.numel()),
                                       _ptr(per_sample_weights, _dt("float32"), "per_sample_weights"),
                                       int(pooling), _ptr(pooled_out, _dt("float32"), "pooled_out"),
                                       _status_ptr(d_status), _stream(stream))


def embbag_backward_sgd_pooled(grad_pooled, batch, indices, offsets, lr, weights, workspace,
                               per_sample_weights=None, pooling=EMBBAG_POOL_SUM, d_status=None,
                               stream=None) -> int:
    _check_bags(len(weights), batch, offsets)
    _check_act(grad_pooled, len(weights), batch, _check_tables(weights), "grad_pooled")
    _check_numel(per_sample_weights, indices.numel(), "per_sample_weights")
    s, keep = _tables_struct(weights)
    return lib().embbag_backward_sgd_pooled(
        _ptr(grad_pooled, _dt("float32"), "grad_pooled"), int(batch),
        _ptr(indices, _dt(*_I32), "indices"), _ptr(offsets, _dt(*_I32), "offsets"),
        int(indices.numel()), _ptr(per_sample_weights, _dt("float32"), "per_sample_weights"),
        int(pooling), float(lr), C.byref(s), _ptr(workspace, None, "workspace"),
        int(workspace.numel() * workspace.element_size()), _status_ptr(d_status),
        _stream(stream))


def embbag_backward_prepare_pooled(rows, dim, batch, indices, offsets, workspace,
                                   per_sample_weights=None, pooling=EMBBAG_POOL_SUM,
                                   d_status=None, stream=None) -> int:
    _check_bags(len(rows), batch, offsets)
    _check_numel(per_sample_weights, indices.numel(), "per_sample_weights")
    T = len(rows)
    r, keep = _rows_arg(rows)
    return lib().embbag_backward_prepare_pooled(
        T, r, int(dim), int(batch), _ptr(indices, _dt(*_I32), "indices"),
        _ptr(offsets, _dt(*_I32), "offsets"), int(indices.numel()),
        _ptr(per_sample_weights, _dt("float32"), "per_sample_weights"), int(pooling),
        _ptr(workspace, None, "workspace"), int(workspace.numel() * workspace.element_size()),
        _status_ptr(d_status), _stream(stream))


def embbag_backward_apply_sgd_pooled(grad_pooled, batch, offsets, num_indices, lr, weights,
                                     workspace, per_sample_weights=None,
                                     pooling=EMBBAG_POOL_SUM, stream=None) -> int:
    _check_bags(len(weights), batch, offsets)
    _check_act(grad_pooled, len(weights), batch, _check_tables(weights), "grad_pooled")
    _check_numel(per_sample_weights, int(num_indices), "per_sample_weights")
    s, keep = _tables_struct(weights)
    return lib().embbag_backward_apply_sgd_pooled(
        _ptr(grad_pooled, _dt("float32"), "grad_pooled"), int(batch),
        _ptr(offsets, _dt(*_I32), "offsets"), int(num_indices),
        _ptr(per_sample_weights, _dt("float32"), "per_sample_weights"), int(pooling), float(lr),
        C.byref(s), _ptr(workspace, None, "workspace"),
        int(workspace.numel() * workspace.element_size()), _stream(stream))


def embbag_forward_split_bf16(hi, batch, indices, offsets, pooled_out, d_status=None,
                              stream=None) -> int:
    _check_bags(len(hi), batch, offsets)
    _check_act(pooled_out, len(hi), batch, _check_tables(hi, "hi table"), "pooled_out")
    s, keep = _split_struct_fwd(hi)
    return lib().embbag_forward_split_bf16(C.byref(s), int(batch),
                                           _ptr(indices, _dt(*_I32), "indices"),
                                           _ptr(offsets, _dt(*_I32), "offsets"),
                                           int(indices.numel()),
                                           _ptr(pooled_out, _dt("float32"), "pooled_out"),
                                           _status_ptr(d_status), _stream(stream))


def embbag_backward_workspace_bytes(num_tables, batch, num_indices, dim) -> int:
    return int(lib().embbag_backward_workspace_bytes(int(num_tables), int(batch),
                                                     int(num_indices), int(dim)))


def embbag_backward_sgd(grad_pooled, batch, indices, offsets, lr, weights, workspace,
                        d_status=None, stream=None) -> int:
    """Fused backward + SGD; ``weights`` are updated in place."""
    _check_bags(len(weights), batch, offsets)
    _check_act(grad_pooled, len(weights), batch, _check_tables(weights), "grad_pooled")
    s, keep = _tables_struct(weights)
    return lib().embbag_backward_sgd(_ptr(grad_pooled, _dt("float32"), "grad_pooled"), int(batch),
                                     _ptr(indices, _dt(*_I32), "indices"),
                                     _ptr(offsets, _dt(*_I32), "offsets"), int(indices.numel()),
                                     float(lr), C.byref(s), _ptr(workspace, None, "workspace"),
                                     int(workspace.numel() * workspace.element_size()),
                                     _status_ptr(d_status), _stream(stream))


def embbag_backward_sgd_noalloc(grad_pooled, batch, indices, offsets, lr, weights,
                                d_status=None, stream=None) -> int:
    """embbag_backward_sgd with the library's fixed device scratch array as its
    workspace (no allocation; EMBBAG_ERR_WORKSPACE past its size)."""
    _check_bags(len(weights), batch, offsets)
    _check_act(grad_pooled, len(weights), batch, _check_tables(weights), "grad_pooled")
    s, keep = _tables_struct(weights)
    return lib().embbag_backward_sgd_noalloc(
        _ptr(grad_pooled, _dt("float32"), "grad_pooled"), int(batch),
        _ptr(indices, _dt(*_I32), "indices"), _ptr(offsets, _dt(*_I32), "offsets"),
        int(indices.numel()), float(lr), C.byref(s), _status_ptr(d_status), _stream(stream))


def embbag_backward_sgd_split_bf16(grad_pooled, batch, indices, offsets, lr, hi, lo, workspace,
                                   d_status=None, stream=None) -> int:
    _check_bags(len(hi), batch, offsets)
    _check_act(grad_pooled, len(hi), batch, _check_tables(hi, "hi table"), "grad_pooled")
    s, keep = _tables_struct(hi, split_lo=lo)
    return lib().embbag_backward_sgd_split_bf16(
        _ptr(grad_pooled, _dt("float32"), "grad_pooled"), int(batch),
        _ptr(indices, _dt(*_I32), "indices"), _ptr(offsets, _dt(*_I32), "offsets"),
        int(indices.numel()), float(lr), C.byref(s), _ptr(workspace, None, "workspace"),
        int(workspace.numel() * workspace.element_size()),
        _status_ptr(d_status), _stream(stream))


def embbag_backward_prepare(rows, dim, batch, indices, offsets, workspace, d_status=None,
                            stream=None) -> int:
    """Phase 1 of the backward: keys, validation and the sort, into ``workspace``."""
    _check_bags(len(rows), batch, offsets)
    T = len(rows)
    r, keep = _rows_arg(rows)
    return lib().embbag_backward_prepare(T, r, int(dim), int(batch),
                                         _ptr(indices, _dt(*_I32), "indices"),
                                         _ptr(offsets, _dt(*_I32), "offsets"),
                                         int(indices.numel()), _ptr(workspace, None, "workspace"),
                                         int(workspace.numel() * workspace.element_size()),
                                         _status_ptr(d_status), _stream(stream))


def embbag_backward_apply_sgd(grad_pooled, batch, num_indices, lr, weights, workspace,
                              stream=None) -> int:
    """Phase 2 of the backward: segment sums and the SGD apply on FP32 tables."""
    _check_act(grad_pooled, len(weights), batch, _check_tables(weights), "grad_pooled")
    s, keep = _tables_struct(weights)
    return lib().embbag_backward_apply_sgd(_ptr(grad_pooled, _dt("float32"), "grad_pooled"),
                                           int(batch), int(num_indices), float(lr), C.byref(s),
                                           _ptr(workspace, None, "workspace"),
                                           int(workspace.numel() * workspace.element_size()),
                                           _stream(stream))


def embbag_backward_apply_sgd_split_bf16(grad_pooled, batch, num_indices, lr, hi, lo, workspace,
                                         stream=None) -> int:
    _check_act(grad_pooled, len(hi), batch, _check_tables(hi, "hi table"), "grad_pooled")
    s, keep = _tables_struct(hi, split_lo=lo)
    return lib().embbag_backward_apply_sgd_split_bf16(
        _ptr(grad_pooled, _dt("float32"), "grad_pooled"), int(batch), int(num_indices), float(lr),
        C.byref(s), _ptr(workspace, None, "workspace"),
        int(workspace.numel() * workspace.element_size()), _stream(stream))


# BF16 activations: pooled outputs and their gradients as torch.bfloat16 (or
# 16-bit integer tensors holding BF16 bit patterns).
_BF16 = ("bfloat16",) + _U16


def embbag_forward_split_bf16_act(hi, batch, indices, offsets, pooled_out, d_status=None,
                                  stream=None) -> int:
    _check_bags(len(hi), batch, offsets)
    _check_act(pooled_out, len(hi), batch, _check_tables(hi, "hi table"), "pooled_out")
    s, keep = _split_struct_fwd(hi)
    return lib().embbag_forward_split_bf16_act(C.byref(s), int(batch),
                                               _ptr(indices, _dt(*_I32), "indices"),
                                               _ptr(offsets, _dt(*_I32), "offsets"),
                                               int(indices.numel()),
                                               _ptr(pooled_out, _dt(*_BF16), "pooled_out"),
                                               _status_ptr(d_status),
                                               _stream(stream))


def embbag_backward_sgd_split_bf16_act(grad_pooled, batch, indices, offsets, lr, hi, lo,
                                       workspace, d_status=None, stream=None) -> int:
    _check_bags(len(hi), batch, offsets)
    _check_act(grad_pooled, len(hi), batch, _check_tables(hi, "hi table"), "grad_pooled")
    s, keep = _tables_struct(hi, split_lo=lo)
    return lib().embbag_backward_sgd_split_bf16_act(
        _ptr(grad_pooled, _dt(*_BF16), "grad_pooled"), int(batch),
        _ptr(indices, _dt(*_I32), "indices"), _ptr(offsets, _dt(*_I32), "offsets"),
        int(indices.numel()), float(lr), C.byref(s), _ptr(workspace, None, "workspace"),
        int(workspace.numel() * workspace.element_size()),
        _status_ptr(d_status), _stream(stream))


def embbag_backward_apply_sgd_split_bf16_act(grad_pooled, batch, num_indices, lr, hi, lo,
                                             workspace, stream=None) -> int:
    _check_act(grad_pooled, len(hi), batch, _check_tables(hi, "hi table"), "grad_pooled")
    s, keep = _tables_struct(hi, split_lo=lo)
    return lib().embbag_backward_apply_sgd_split_bf16_act(
        _ptr(grad_pooled, _dt(*_BF16), "grad_pooled"), int(batch), int(num_indices), float(lr),
        C.byref(s), _ptr(workspace, None, "workspace"),
        int(workspace.numel() * workspace.element_size()), _stream(stream))


def embbag_split_fp32(w, hi, lo, stream=None) -> int:
    _check_numel(hi, w.numel(), "hi")
    _check_numel(lo, w.numel(), "lo")
    return lib().embbag_split_fp32(_ptr(w, _dt("float32"), "w"), _ptr(hi, _dt(*_U16), "hi"),
                                   _ptr(lo, _dt(*_U16), "lo"), int(w.numel()), _stream(stream))


def embbag_combine_fp32(hi, lo, w, stream=None) -> int:
    _check_numel(hi, w.numel(), "hi")
    _check_numel(lo, w.numel(), "lo")
    return lib().embbag_combine_fp32(_ptr(hi, _dt(*_U16), "hi"), _ptr(lo, _dt(*_U16), "lo"),
                                     _ptr(w, _dt("float32"), "w"), int(w.numel()), _stream(stream))


def embbag_dedup_workspace_bytes(num_tables, batch, num_indices) -> int:
    return int(lib().embbag_dedup_workspace_bytes(int(num_tables), int(batch), int(num_indices)))


def embbag_dedup(rows, batch, indices, offsets, sorted_keys, sorted_bags, unique_keys, seg_off,
                 d_num_unique, workspace, d_status=None, stream=None) -> int:
    _check_bags(len(rows), batch, offsets)
    for a, n in ((sorted_keys, "sorted_keys"), (sorted_bags, "sorted_bags"), (unique_keys, "unique_keys")):
        _check_numel(a, indices.numel(), n, exact=False)
    _check_numel(seg_off, indices.numel() + 1, "seg_off", exact=False)
    _check_numel(d_num_unique, 1, "d_num_unique", exact=False)
    T = len(rows)
    r, keep = _rows_arg(rows)
    return lib().embbag_dedup(T, r, int(batch),
                              _ptr(indices, _dt(*_I32), "indices"),
                              _ptr(offsets, _dt(*_I32), "offsets"), int(indices.numel()),
                              _ptr(sorted_keys, _dt(*_U32), "sorted_keys"),
                              _ptr(sorted_bags, _dt(*_U32), "sorted_bags"),
                              _ptr(unique_keys, _dt(*_U32), "unique_keys"),
                              _ptr(seg_off, _dt(*_I32), "seg_off"),
                              _ptr(d_num_unique, _dt(*_I32), "d_num_unique"),
                              _ptr(workspace, None, "workspace"),
                              int(workspace.numel() * workspace.element_size()),
                              _status_ptr(d_status), _stream(stream))


# ---- baselines: the paper's unfused designs (for measurement) --------------
def embbag_baseline_materialize(grad_pooled, num_tables, batch, dim, offsets, num_indices, dW,
                                d_status=None, stream=None) -> int:
    _check_bags(int(num_tables), batch, offsets)
    _check_act(grad_pooled, int(num_tables), batch, int(dim), "grad_pooled")
    _check_numel(dW, int(num_indices) * int(dim), "dW", exact=False)
    return lib().embbag_baseline_materialize(_ptr(grad_pooled, _dt("float32"), "grad_pooled"),
                                             int(num_tables), int(batch), int(dim),
                                             _ptr(offsets, _dt(*_I32), "offsets"),
                                             int(num_indices), _ptr(dW, _dt("float32"), "dW"),
                                             _status_ptr(d_status),
                                             _stream(stream))


def embbag_baseline_update_atomic(dW, batch, indices, offsets, lr, weights, d_status=None,
                                  stream=None) -> int:
    _check_bags(len(weights), batch, offsets)
    _check_numel(dW, indices.numel() * _check_tables(weights), "dW", exact=False)
    s, keep = _tables_struct(weights)
    return lib().embbag_baseline_update_atomic(_ptr(dW, _dt("float32"), "dW"), int(batch),
                                               _ptr(indices, _dt(*_I32), "indices"),
                                               _ptr(offsets, _dt(*_I32), "offsets"),
                                               int(indices.numel()), float(lr), C.byref(s),
                                               _status_ptr(d_status),
                                               _stream(stream))


def embbag_baseline_backward_sgd_atomic(grad_pooled, batch, indices, offsets, lr, weights,
                                        d_status=None, stream=None) -> int:
    _check_bags(len(weights), batch, offsets)
    _check_act(grad_pooled, len(weights), batch, _check_tables(weights), "grad_pooled")
    s, keep = _tables_struct(weights)
    return lib().embbag_baseline_backward_sgd_atomic(
        _ptr(grad_pooled, _dt("float32"), "grad_pooled"), int(batch),
        _ptr(indices, _dt(*_I32), "indices"), _ptr(offsets, _dt(*_I32), "offsets"),
        int(indices.numel()), float(lr), C.byref(s), _status_ptr(d_status),
        _stream(stream))


def embbag_baseline_update_owner(dW, batch, indices, offsets, lr, weights, owners,
                                 stream=None) -> int:
    _check_bags(len(weights), batch, offsets)
    _check_numel(dW, indices.numel() * _check_tables(weights), "dW", exact=False)
    s, keep = _tables_struct(weights)
    return lib().embbag_baseline_update_owner(_ptr(dW, _dt("float32"), "dW"), int(batch),
                                              _ptr(indices, _dt(*_I32), "indices"),
                                              _ptr(offsets, _dt(*_I32), "offsets"),
                                              int(indices.numel()), float(lr), C.byref(s),
                                              int(owners), _stream(stream))


def embbag_baseline_touch_rows(batch, num_indices, weights, workspace, stream=None) -> int:
    s, keep = _tables_struct(weights)
    return lib().embbag_baseline_touch_rows(int(batch), int(num_indices), C.byref(s),
                                            _ptr(workspace, None, "workspace"),
                                            int(workspace.numel() * workspace.element_size()),
                                            _stream(stream))


def embbag_baseline_touch_rows_split(batch, num_indices, hi, lo, workspace, stream=None) -> int:
    s, keep = _tables_struct(hi, split_lo=lo)
    return lib().embbag_baseline_touch_rows_split(int(batch), int(num_indices), C.byref(s),
                                                  _ptr(workspace, None, "workspace"),
                                                  int(workspace.numel() * workspace.element_size()),
                                                  _stream(stream))


def embbag_status_read(d_status, stream=None) -> int:
    return lib().embbag_status_read(_status_ptr(d_status), _stream(stream))


__all__ = [n for n in dir() if n.startswith("embbag_") or n.startswith("EMBBAG_")] + [
    "lib", "check", "EmbbagError", "LIB_PATH"]
