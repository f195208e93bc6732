"""The paper's unfused update designs on the GPU (measured baselines):
Algorithm 2 (materialised dW), Algorithm 3 with FP32 atomics, the fused
atomic update, and Algorithm 4's row-range ownership; and the update's floor
(each touched row read and written back once)."""
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


def _case(seed, rows=(2000, 37, 900), dim=64, batch=300, maxp=10, hot=0.0):
    rng = np.random.default_rng(seed)
    W = [rng.uniform(-0.05, 0.05, (m, dim)).astype(np.float32) for m in rows]
    I, O = random_bags(rng, rows, batch, maxp, 0.1, hot)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    return W, I, O, G, batch, dim


@pytest.mark.parametrize("dim", [4, 8, 12, 16, 32, 64, 100, 128, 256, 260, 512, 1024])
def test_materialize_is_a_copy(dim):
    W, I, O, G, B, E = _case(1, dim=dim)
    T = len(W)
    dW = torch.empty((I.size, E), dtype=torch.float32, device=DEV)
    assert pk.embbag_baseline_materialize(to_dev(G), T, B, E, to_dev(O), I.size, dW) == 0
    bag = np.searchsorted(O, np.arange(I.size), side="right") - 1
    assert bits_equal(dW.cpu().numpy(), G.reshape(-1, E)[bag])


@pytest.mark.parametrize("owners", [1, 7, 256])
@pytest.mark.parametrize("dim", [16, 256, 1024])
def test_owner_update_equals_sequential_fp32(owners, dim):
    """Algorithm 4 applies each row's look-ups in increasing s in FP32: bit for
    bit the oracle's literal reading of Algorithms 2 and 3."""
    W, I, O, G, B, E = _case(2 + owners, dim=dim, hot=0.3)
    T = len(W)
    log(f"[owner] owners={owners} dim={dim} NS={I.size}")
    gt = GpuTables(W)
    dW = torch.empty((I.size, E), dtype=torch.float32, device=DEV)
    assert pk.embbag_baseline_materialize(to_dev(G), T, B, E, to_dev(O), I.size, dW) == 0
    assert pk.embbag_baseline_update_owner(dW, B, to_dev(I), to_dev(O), 0.1, gt.w, owners) == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd(G, B, I, O, 0.1, Wref, literal=True) == 0
    for a, b in zip(gt.host(), Wref):
        assert bits_equal(a, b)


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("dim", [8, 64, 260, 1024])
def test_atomic_update_within_tolerance(fused, dim):
    W, I, O, G, B, E = _case(3, dim=dim)
    T = len(W)
    gt = GpuTables(W)
    if fused:
        assert pk.embbag_baseline_backward_sgd_atomic(to_dev(G), B, to_dev(I), to_dev(O), 0.1,
                                                      gt.w, gt.status) == 0
    else:
        dW = torch.empty((I.size, E), dtype=torch.float32, device=DEV)
        assert pk.embbag_baseline_materialize(to_dev(G), T, B, E, to_dev(O), I.size, dW) == 0
        assert pk.embbag_baseline_update_atomic(dW, B, to_dev(I), to_dev(O), 0.1, gt.w,
                                                gt.status) == 0
    assert gt.read_status() == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd(G, B, I, O, 0.1, Wref) == 0
    for t, (a, b) in enumerate(zip(gt.host(), Wref)):
        assert_close(a, b, f"atomic table {t}")


@pytest.mark.parametrize("dim", [16, 64, 256, 1024])
def test_touch_rows_keeps_every_bit(dim):
    """The floor kernel writes back what it read: the tables keep their bits,
    and the prepared workspace still drives an update that matches the oracle."""
    W, I, O, G, B, E = _case(11 + dim, dim=dim, hot=0.3)
    rows = [w.shape[0] for w in W]
    gt = GpuTables(W)
    Id, Od = to_dev(I), to_dev(O)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(len(W), B, I.size, E), dtype=torch.uint8,
                     device=DEV)
    assert pk.embbag_backward_prepare(rows, E, B, Id, Od, ws, gt.status) == 0
    for _ in range(2):
        assert pk.embbag_baseline_touch_rows(B, I.size, gt.w, ws) == 0
    for a, b in zip(gt.host(), W):
        assert bits_equal(a, b)
    assert pk.embbag_backward_apply_sgd(to_dev(G), B, I.size, 0.1, gt.w, ws) == 0
    assert gt.read_status() == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd(G, B, I, O, 0.1, Wref) == 0
    for t, (a, b) in enumerate(zip(gt.host(), Wref)):
        assert_close(a, b, f"table {t} after touch + apply")


@pytest.mark.parametrize("dim", [16, 64, 256, 1024])
def test_touch_rows_split_keeps_every_bit(dim):
    """The split floor writes back both halves it read: hi and lo keep their
    bits, and the prepared workspace still drives a split update that matches
    the oracle's."""
    W, I, O, G, B, E = _case(17 + dim, dim=dim, hot=0.3)
    rows = [w.shape[0] for w in W]
    gt = GpuTables(W, split=True)
    hi0 = [h.clone() for h in gt.w]
    lo0 = [l.clone() for l in gt.lo]
    Id, Od = to_dev(I), to_dev(O)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(len(W), B, I.size, E), dtype=torch.uint8,
                     device=DEV)
    assert pk.embbag_backward_prepare(rows, E, B, Id, Od, ws, gt.status) == 0
    for _ in range(2):
        assert pk.embbag_baseline_touch_rows_split(B, I.size, gt.w, gt.lo, ws) == 0
    for a, b in zip(gt.w + gt.lo, hi0 + lo0):
        assert torch.equal(a, b)
    assert pk.embbag_backward_apply_sgd_split_bf16(to_dev(G), B, I.size, 0.1, gt.w, gt.lo, ws) == 0
    assert gt.read_status() == 0
    his, los = zip(*[oracle.split(w) for w in W])
    his, los = [h.copy() for h in his], [l.copy() for l in los]
    assert oracle.backward_sgd_split(G, B, I, O, 0.1, his, los) == 0
    for t in range(len(W)):
        got = oracle.combine(gt.w[t].cpu().numpy().view(np.uint16), gt.lo[t].cpu().numpy().view(np.uint16))
        want = oracle.combine(his[t], los[t])
        assert_close(got, want, f"split table {t} after touch + apply")


def test_touch_rows_split_writes_nothing_without_a_prepare():
    """A workspace with no sort result for these sizes: the split floor leaves
    the halves alone."""
    W, I, O, G, B, E = _case(5, dim=64)
    gt = GpuTables(W, split=True)
    hi0 = [h.clone() for h in gt.w]
    lo0 = [l.clone() for l in gt.lo]
    ws = torch.zeros(pk.embbag_backward_workspace_bytes(len(W), B, I.size, E), dtype=torch.uint8,
                     device=DEV)
    assert pk.embbag_baseline_touch_rows_split(B, I.size, gt.w, gt.lo, ws) == 0
    torch.cuda.synchronize()
    for a, b in zip(gt.w + gt.lo, hi0 + lo0):
        assert torch.equal(a, b)
    assert (pk.embbag_baseline_touch_rows_split(B, I.size, gt.w, gt.lo, ws[:256]) ==
            pk.EMBBAG_ERR_WORKSPACE)
    assert pk.embbag_baseline_touch_rows_split(-1, I.size, gt.w, gt.lo, ws) == pk.EMBBAG_ERR_INVALID_ARG


def test_touch_rows_argument_errors():
    W, I, O, G, B, E = _case(4)
    gt = GpuTables(W)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(len(W), B, I.size, E), dtype=torch.uint8,
                     device=DEV)
    assert pk.embbag_baseline_touch_rows(B, I.size, gt.w, ws[:256]) == pk.EMBBAG_ERR_WORKSPACE
    assert pk.embbag_baseline_touch_rows(-1, I.size, gt.w, ws) == pk.EMBBAG_ERR_INVALID_ARG
