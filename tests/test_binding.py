"""The Python binding on the CPU: it only marshals arguments, so it must refuse
host tensors, non-contiguous tensors and wrong dtypes before any library call,
fail loudly when the library is missing, and raise EmbbagError on a bad status.
(No GPU here: nothing below reaches a HIP call.)"""
import numpy as np
import pytest
import torch

import paper_2005_04680_amd as pk


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(pk, "LIB_PATH", str(tmp_path / "libembbag.so"))
    monkeypatch.setattr(pk, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        pk.lib()


def test_host_tensors_are_refused():
    W = [torch.zeros((10, 8))]
    I = torch.zeros(4, dtype=torch.int32)
    O = torch.tensor([0, 4], dtype=torch.int32)
    Y = torch.zeros((1, 1, 8))
    with pytest.raises(TypeError, match="GPU tensor"):
        pk.embbag_forward(W, 1, I, O, Y)
    with pytest.raises(TypeError, match="GPU tensor"):
        pk.embbag_backward_sgd(Y, 1, I, O, 0.1, W, torch.zeros(1024, dtype=torch.uint8))
    with pytest.raises(TypeError, match="GPU tensor"):
        pk.embbag_forward_split_bf16([torch.zeros((10, 8), dtype=torch.int16)], 1, I, O, Y)
    with pytest.raises(TypeError, match="GPU tensor"):
        pk.embbag_split_fp32(torch.zeros(8), torch.zeros(8, dtype=torch.int16),
                             torch.zeros(8, dtype=torch.int16))


def test_status_codes_and_check():
    assert pk.embbag_status_string(pk.EMBBAG_OK) == "ok"
    assert "index" in pk.embbag_status_string(pk.EMBBAG_ERR_INDEX_RANGE)
    pk.check(pk.EMBBAG_OK)
    with pytest.raises(pk.EmbbagError) as e:
        pk.check(pk.EMBBAG_ERR_OFFSETS, "backward")
    assert e.value.code == pk.EMBBAG_ERR_OFFSETS and "offsets" in str(e.value)


def test_workspace_size_marshalling():
    n = pk.embbag_backward_workspace_bytes(16, 8192, 16 * 8192 * 100, 256)
    assert n > 16 * 8192 * 100 * 16  # two 64-bit key buffers at least
    assert pk.embbag_backward_workspace_bytes(0, 8, 10, 16) == 0  # invalid table count
    assert pk.embbag_dedup_workspace_bytes(4, 32, 512) > 0


class _FakeCuda:
    """Stands in for a GPU tensor so that the binding's dtype and layout checks
    run on the CPU; its address is never dereferenced."""

    def __init__(self, t):
        self._t = t
        self.is_cuda = True
        self.dtype = t.dtype
        self.shape = t.shape

    def is_contiguous(self):
        return self._t.is_contiguous()

    def data_ptr(self):
        return 4096  # a dummy address: the checks under test fail before any library call

    def numel(self):
        return self._t.numel()

    def element_size(self):
        return self._t.element_size()


def test_dtype_and_layout_checks():
    W = [_FakeCuda(torch.zeros((10, 8)))]
    O = _FakeCuda(torch.zeros(2, dtype=torch.int32))
    Y = _FakeCuda(torch.zeros((1, 1, 8)))
    with pytest.raises(TypeError, match="indices"):
        pk.embbag_forward(W, 1, _FakeCuda(torch.zeros(4, dtype=torch.int64)), O, Y)
    with pytest.raises(TypeError, match="contiguous"):
        pk.embbag_forward(W, 1, _FakeCuda(torch.zeros((4, 2), dtype=torch.int32).t()), O, Y)
    with pytest.raises(TypeError, match="pooled_out"):
        pk.embbag_forward_split_bf16_act([_FakeCuda(torch.zeros((10, 8), dtype=torch.int16))], 1,
                                         _FakeCuda(torch.zeros(4, dtype=torch.int32)), O, Y)


def test_shape_checks_before_any_library_call():
    """Sizes the C ABI takes on trust (it gets raw pointers) are checked here: a
    narrower table, a short or long offsets array, activations of the wrong size
    or mismatched split halves raise ValueError instead of reaching a kernel."""
    f32 = lambda *shape: _FakeCuda(torch.zeros(shape))
    i32 = lambda n: _FakeCuda(torch.zeros(n, dtype=torch.int32))
    i16 = lambda *shape: _FakeCuda(torch.zeros(shape, dtype=torch.int16))
    W = [f32(10, 8), f32(20, 8)]
    I, O, Y = i32(6), i32(2 * 3 + 1), f32(2, 3, 8)
    ws = _FakeCuda(torch.zeros(64, dtype=torch.uint8))
    with pytest.raises(ValueError, match="table 1"):
        pk.embbag_forward([f32(10, 8), f32(20, 4)], 3, I, O, Y)
    with pytest.raises(ValueError, match="table 0"):
        pk.embbag_forward([f32(10, 8), f32(80)], 3, I, O, Y)
    with pytest.raises(ValueError, match="offsets"):
        pk.embbag_forward(W, 3, I, i32(6), Y)
    with pytest.raises(ValueError, match="offsets"):
        pk.embbag_backward_prepare((10, 20), 8, 3, I, i32(8), ws)
    with pytest.raises(ValueError, match="pooled_out"):
        pk.embbag_forward(W, 3, I, O, f32(2, 3, 4))
    with pytest.raises(ValueError, match="grad_pooled"):
        pk.embbag_backward_sgd(f32(2, 2, 8), 3, I, O, 0.1, W, ws)
    with pytest.raises(ValueError, match="grad_pooled"):
        pk.embbag_backward_apply_sgd(f32(1, 3, 8), 3, 6, 0.1, W, ws)
    with pytest.raises(ValueError, match="per_sample_weights"):
        pk.embbag_forward_pooled(W, 3, I, O, Y, f32(5))
    with pytest.raises(ValueError, match="lo table 1"):
        pk.embbag_backward_sgd_split_bf16(Y, 3, I, O, 0.1, [i16(10, 8), i16(20, 8)],
                                          [i16(10, 8), i16(19, 8)], ws)
    with pytest.raises(ValueError, match="lo tables"):
        pk.embbag_backward_apply_sgd_split_bf16(Y, 3, 6, 0.1, [i16(10, 8), i16(20, 8)],
                                                [i16(10, 8)], ws)
    with pytest.raises(ValueError, match="seg_off"):
        pk.embbag_dedup((10, 20), 3, I, O, i32(6), i32(6), i32(6), i32(6), i32(1), ws)
    with pytest.raises(ValueError, match="lo"):
        pk.embbag_split_fp32(f32(16), i16(16), i16(8))
    with pytest.raises(ValueError, match="dW"):
        pk.embbag_baseline_materialize(Y, 2, 3, 8, O, 6, f32(5, 8))
    with pytest.raises(ValueError, match="d_status"):
        pk.embbag_forward(W, 3, I, O, Y, i32(0))


def test_prebuilt_descriptors_refuse_host_tensors_and_the_other_kind():
    """Tables / SplitTables check their tensors once, when built, and an entry
    point refuses the other kind before any library call."""
    with pytest.raises(TypeError, match="GPU tensor"):
        pk.Tables([torch.zeros((10, 8))])
    h = [torch.zeros((10, 8), dtype=torch.int16)]
    with pytest.raises(TypeError, match="GPU tensor"):
        pk.SplitTables(h, h)
    fp32 = pk.Tables.__new__(pk.Tables)  # as built, without touching a GPU
    fp32.tensors, fp32.dim, fp32.struct, fp32.rows_addr = [torch.zeros((10, 8))], 8, None, 0
    split = pk.SplitTables.__new__(pk.SplitTables)
    split.hi, split.lo, split.dim, split.struct, split.rows_addr = h, h, 8, None, 0
    with pytest.raises(TypeError, match="FP32 Tables"):
        pk._tables_struct(fp32, split_lo=None)
    with pytest.raises(TypeError, match="FP32 Tables"):
        pk._split_struct_fwd(fp32)
    with pytest.raises(TypeError, match="SplitTables"):
        pk._tables_struct(split)
    assert len(fp32) == 1 and fp32[0] is fp32.tensors[0]
    assert len(split) == 1 and split[0] is h[0]
