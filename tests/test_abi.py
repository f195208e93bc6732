"""The C ABI library loads, exports every declared entry point, and rejects bad
arguments on the host (no GPU needed: these calls return before any HIP call)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "embbag.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(embbag_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    import paper_2005_04680_amd as pk
    if not os.path.exists(pk.LIB_PATH):
        import paper_2005_04680_amd.build as b
        b.build()
    return pk.lib()


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("embbag_forward", "embbag_backward_sgd", "embbag_forward_split_bf16",
              "embbag_backward_sgd_split_bf16", "embbag_backward_workspace_bytes",
              "embbag_split_fp32", "embbag_combine_fp32", "embbag_dedup",
              "embbag_dedup_workspace_bytes", "embbag_status_read", "embbag_status_string"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    missing = [n for n in _declared() if not hasattr(L, n)]
    assert not missing, missing


def test_status_codes_match_oracle(L, oracle):
    import paper_2005_04680_amd as pk
    assert (pk.EMBBAG_OK, pk.EMBBAG_ERR_INVALID_ARG, pk.EMBBAG_ERR_WORKSPACE,
            pk.EMBBAG_ERR_INDEX_RANGE, pk.EMBBAG_ERR_OFFSETS) == (
        oracle.OK, oracle.ERR_INVALID_ARG, oracle.ERR_WORKSPACE, oracle.ERR_INDEX_RANGE,
        oracle.ERR_OFFSETS)
    text = open(HEADER).read()
    for name, val in (("EMBBAG_OK", 0), ("EMBBAG_ERR_INVALID_ARG", -1), ("EMBBAG_ERR_WORKSPACE", -2),
                      ("EMBBAG_ERR_INDEX_RANGE", -3), ("EMBBAG_ERR_OFFSETS", -4),
                      ("EMBBAG_ERR_HIP", -5)):
        assert re.search(rf"#define {name} \(?{val}\)?", text)
    assert pk.embbag_status_string(-3) == "index out of its table's range"
    assert pk.embbag_status_string(7) == "unknown status"


class _T(C.Structure):
    _fields_ = [("num_tables", C.c_int32), ("dim", C.c_int32),
                ("rows", C.POINTER(C.c_int64)), ("weights", C.POINTER(C.c_void_p))]


FAKE = 1 << 20  # a 256-byte aligned non-null address; never dereferenced on these paths


def _tables(rows, dim, ptrs=None):
    r = (C.c_int64 * len(rows))(*rows)
    p = (C.c_void_p * len(rows))(*(ptrs or [FAKE + 4096 * i for i in range(len(rows))]))
    return _T(len(rows), dim, C.cast(r, C.POINTER(C.c_int64)), C.cast(p, C.POINTER(C.c_void_p))), (r, p)


@pytest.mark.parametrize("rows,dim,batch,ns,expect", [
    ((10,), 6, 1, 1, -1),            # E % 4
    ((10,), 2048, 1, 1, -1),         # E > 1024
    ((10,), 0, 1, 1, -1),
    ((), 8, 1, 1, -1),               # T = 0
    ((10,) * 65, 8, 1, 1, -1),       # T > 64
    ((0,), 8, 1, 1, -1),             # empty table
    ((2 ** 31,), 8, 1, 1, -1),       # M_t > INT32_MAX
    ((2 ** 30, 2 ** 30), 8, 1, 1, -1),  # sum of rows > INT32_MAX
    ((10,), 8, -1, 1, -1),           # B < 0
    ((10,), 8, 1, -1, -1),           # NS < 0
    ((10,), 8, 1, 2 ** 31, -1),      # NS > INT32_MAX
    ((10,), 8, 0, 5, -4),            # T*B == 0 but NS > 0
])
def test_forward_argument_errors(L, rows, dim, batch, ns, expect):
    t, keep = _tables(list(rows) or [1], dim)
    if not rows:
        t.num_tables = 0
    rc = L.embbag_forward(C.byref(t), batch, FAKE, FAKE, ns, FAKE, None, None)
    assert rc == expect


def test_null_and_misaligned_pointers(L):
    t, keep = _tables([10, 10], 8)
    assert L.embbag_forward(None, 1, FAKE, FAKE, 1, FAKE, None, None) == -1
    assert L.embbag_forward(C.byref(t), 1, FAKE, None, 1, FAKE, None, None) == -1    # offsets
    assert L.embbag_forward(C.byref(t), 1, None, FAKE, 1, FAKE, None, None) == -1    # indices
    assert L.embbag_forward(C.byref(t), 1, FAKE, FAKE, 1, None, None, None) == -1    # output
    assert L.embbag_forward(C.byref(t), 1, FAKE, FAKE, 1, FAKE + 4, None, None) == -1  # align
    t2, keep2 = _tables([10, 10], 8, ptrs=[FAKE, FAKE + 8])                          # table align
    assert L.embbag_forward(C.byref(t2), 1, FAKE, FAKE, 1, FAKE, None, None) == -1
    t3, keep3 = _tables([10, 10], 8, ptrs=[FAKE, 0])
    assert L.embbag_forward(C.byref(t3), 1, FAKE, FAKE, 1, FAKE, None, None) == -1


def test_workspace_checks(L):
    need = L.embbag_backward_workspace_bytes(2, 4, 100, 8)
    assert need > 0 and need % 256 == 0
    assert L.embbag_backward_workspace_bytes(2, 4, 1000, 8) > need
    assert L.embbag_backward_workspace_bytes(0, 4, 100, 8) == 0
    assert L.embbag_backward_workspace_bytes(2, 4, 100, 6) == 0
    assert L.embbag_backward_workspace_bytes(2, -1, 100, 8) == 0
    t, keep = _tables([10, 10], 8)
    # too small, then misaligned: rejected before anything is launched
    assert L.embbag_backward_sgd(FAKE, 4, FAKE, FAKE, 100, C.c_float(0.1), C.byref(t), FAKE,
                                 need - 1, None, None) == -2
    assert L.embbag_backward_sgd(FAKE, 4, FAKE, FAKE, 100, C.c_float(0.1), C.byref(t), FAKE + 64,
                                 need, None, None) == -2
    assert L.embbag_backward_sgd(FAKE, 4, FAKE, FAKE, 100, C.c_float(0.1), C.byref(t), None,
                                 need, None, None) == -2
    assert L.embbag_backward_sgd(None, 4, FAKE, FAKE, 100, C.c_float(0.1), C.byref(t), FAKE,
                                 need, None, None) == -1
    dneed = L.embbag_dedup_workspace_bytes(2, 4, 100)
    assert dneed > 0
    rows = (C.c_int64 * 2)(10, 10)
    assert L.embbag_dedup(2, rows, 4, FAKE, FAKE, 100, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                          dneed - 256, None, None) == -2


def test_lookup_limit_is_int32_max(L):
    """Indices and offsets are int32, so 2^31 - 1 look-ups is the largest
    count: it passes the argument checks (a workspace of 0 bytes is then
    refused, before anything is launched) and 2^31 does not.  The oracle draws
    the line at the same count."""
    NS = 2 ** 31 - 1
    assert L.embbag_backward_workspace_bytes(1, 1, NS, 4) >= NS * 16
    assert L.embbag_backward_workspace_bytes(1, 1, NS + 1, 4) == 0
    assert L.embbag_dedup_workspace_bytes(1, 1, NS) > 0
    assert L.embbag_dedup_workspace_bytes(1, 1, NS + 1) == 0
    t, keep = _tables([10], 8)
    assert L.embbag_backward_sgd(FAKE, 1, FAKE, FAKE, NS, C.c_float(0.1), C.byref(t), FAKE,
                                 0, None, None) == -2
    assert L.embbag_backward_sgd(FAKE, 1, FAKE, FAKE, NS + 1, C.c_float(0.1), C.byref(t), FAKE,
                                 0, None, None) == -1
    assert L.embbag_forward(C.byref(t), 1, FAKE, FAKE, NS + 1, FAKE, None, None) == -1


def test_large_workspace_is_modest():
    """Large-shaped step: 16 tables x 8192 bags x 100 look-ups, E = 256: under
    0.6 GiB (two 64-bit key buffers, two weight buffers, digit counts, FP64
    carries) beside 98 GB of tables."""
    import paper_2005_04680_amd as pk
    n = pk.embbag_backward_workspace_bytes(16, 8192, 16 * 8192 * 100, 256)
    assert n < 614 * 2 ** 20
