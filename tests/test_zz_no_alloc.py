"""The no-allocation backward (embbag_backward_sgd_noalloc) through the C ABI
against the workspace entry point whose kernels it shares (embbag_backward_sgd):
bit for bit on two calls in a row, the second smaller (the library's scratch
array keeps the first call's contents), each also within the tolerance of the
CPU oracle with untouched rows keeping their bits.  A step too large for the
array is refused before anything runs; a data error writes nothing."""
import numpy as np
import pytest
import torch

import oracle
import paper_2005_04680_amd as pk
from embbag_data import random_bags
from gpu_util import DEV, GpuTables, assert_close, bits_equal, log, require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _case(seed, rows, dim, batch, maxp, hot):
    rng = np.random.default_rng(seed)
    W = [rng.uniform(-0.05, 0.05, size=(m, dim)).astype(np.float32) for m in rows]
    I, O = random_bags(rng, rows, batch, maxp, empty_frac=0.05, hot_frac=hot)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    return W, I, O, G


# (seed, rows, dim, batch, max look-ups per bag, hot fraction): the first is
# about 537K look-ups of E = 64 (a 31 MiB workspace), the second smaller
CASES = [(5, (40000,) * 8, 64, 2048, 64, 0.2), (6, (3000, 500, 70), 32, 300, 12, 0.4)]


def test_noalloc_matches_workspace_entry_point_twice():
    for seed, rows, dim, batch, maxp, hot in CASES:
        W, I, O, G = _case(seed, rows, dim, batch, maxp, hot)
        T = len(rows)
        need = pk.embbag_backward_workspace_bytes(T, batch, I.size, dim)
        log(f"[noalloc] T={T} E={dim} B={batch} NS={I.size} workspace={need / 2**20:.1f} MiB")
        assert 0 < need <= pk.EMBBAG_NOALLOC_SCRATCH_BYTES
        Id, Od, Gd = to_dev(I), to_dev(O), to_dev(G)
        ref = GpuTables(W)
        ws = torch.empty(need, dtype=torch.uint8, device=DEV)
        assert pk.embbag_backward_sgd(Gd, batch, Id, Od, 0.1, ref.w, ws, ref.status) == 0
        got = GpuTables(W)
        assert pk.embbag_backward_sgd_noalloc(Gd, batch, Id, Od, 0.1, got.w, got.status) == 0
        assert ref.read_status() == 0 and got.read_status() == 0
        Wref = [w.copy() for w in W]
        assert oracle.backward_sgd(G, batch, I, O, 0.1, Wref) == 0
        for t, (a, b) in enumerate(zip(got.host(), ref.host())):
            assert bits_equal(a, b), f"table {t}: no-allocation entry point differs"
            lo, hi = O[t * batch], O[(t + 1) * batch]
            touched = np.zeros(rows[t], bool)
            touched[I[lo:hi]] = True
            assert_close(a[touched], Wref[t][touched], f"table {t} touched rows")
            assert bits_equal(a[~touched], W[t][~touched]), f"table {t} untouched rows"


def test_noalloc_refuses_a_step_past_its_array():
    """16 tables x 8192 bags x 100 look-ups at E = 256 need 519 MiB: refused with
    EMBBAG_ERR_WORKSPACE, nothing enqueued, the table keeps its bits."""
    T, B, P, E = 16, 8192, 100, 256
    NS = T * B * P
    assert pk.embbag_backward_workspace_bytes(T, B, NS, E) > pk.EMBBAG_NOALLOC_SCRATCH_BYTES
    W = [torch.zeros((10, E), dtype=torch.float32, device=DEV) for _ in range(T)]
    I = torch.zeros(NS, dtype=torch.int32, device=DEV)
    O = torch.arange(0, NS + 1, P, dtype=torch.int32, device=DEV)
    G = torch.ones((T, B, E), dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    assert pk.embbag_backward_sgd_noalloc(G, B, I, O, 0.1, W, status) == pk.EMBBAG_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert all(int(torch.count_nonzero(w)) == 0 for w in W)
    assert pk.embbag_status_read(status) == 0


def test_noalloc_data_error_writes_nothing():
    W, I, O, G = _case(7, (500, 300), 16, 64, 10, 0.3)
    I[-1] = 300  # out of table 1's range
    got = GpuTables(W)
    assert pk.embbag_backward_sgd_noalloc(to_dev(G), 64, to_dev(I), to_dev(O), 0.1, got.w,
                                          got.status) == 0
    assert got.read_status() == pk.EMBBAG_ERR_INDEX_RANGE
    for a, b in zip(got.host(), W):
        assert bits_equal(a, b)
