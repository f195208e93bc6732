"""Randomized GPU parity: 48 seeded cases with random table counts and sizes,
embedding widths, batch sizes, bag-size mixes (empty, single, long), duplicate
rates and storage (FP32 or split), each run forward + fused backward through
the C ABI and compared with the oracle (pooled outputs and every updated row
within tolerance, untouched rows bit-identical), and the dedup bit-exact."""
import numpy as np
import pytest

import oracle
from gpu_util import GpuTables, assert_close, bits_equal, gpu_dedup, log, require_gpu

pytestmark = pytest.mark.gpu

DIMS = [4, 8, 12, 16, 20, 32, 48, 64, 100, 128, 160, 256, 384, 512, 768, 1024]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _case(seed):
    rng = np.random.default_rng(10_000 + seed)
    T = int(rng.integers(1, 9))
    rows = tuple(int(m) for m in rng.integers(1, 20000, T))
    E = int(rng.choice(DIMS))
    B = int(rng.integers(1, 400))
    kind = rng.integers(0, 4)
    if kind == 0:
        sizes = rng.integers(0, 3, T * B)            # mostly tiny bags
    elif kind == 1:
        sizes = rng.integers(0, 60, T * B)
    elif kind == 2:
        sizes = rng.poisson(20, T * B)
    else:
        sizes = np.where(rng.random(T * B) < 0.05, rng.integers(200, 800, T * B), 1)
    sizes[rng.random(T * B) < rng.uniform(0, 0.3)] = 0
    hot = rng.uniform(0, 0.7)
    I = []
    for k, n in enumerate(sizes):
        m = rows[k // B]
        idx = rng.integers(0, m, n)
        idx[rng.random(n) < hot] = int(rng.integers(0, m))
        I.append(idx)
    I = np.concatenate(I).astype(np.int32)
    O = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    W = [rng.uniform(-0.05, 0.05, (m, E)).astype(np.float32) for m in rows]
    G = rng.standard_normal((T, B, E)).astype(np.float32)
    split = bool(rng.random() < 0.3)
    return rows, E, B, I, O, W, G, split


@pytest.mark.parametrize("seed", range(48))
def test_random_case(seed):
    rows, E, B, I, O, W, G, split = _case(seed)
    log(f"[fuzz] seed={seed} T={len(rows)} E={E} B={B} NS={I.size} split={split}")
    gt = GpuTables(W, split=split)
    rc, Y = gt.forward(B, I, O)
    assert rc == 0 and gt.read_status() == 0
    if split:
        rc, Yref = oracle.forward_split([oracle.split(w)[0] for w in W], B, I, O)
    else:
        rc, Yref = oracle.forward(W, B, I, O)
    assert rc == 0
    Yg = Y.cpu().numpy()
    assert_close(Yg, Yref, f"seed {seed} pooled")
    # the forward sums each bag in FP64 in look-up order and rounds once, like
    # the oracle: the pooled outputs are the same bits
    assert bits_equal(Yg, Yref), f"seed {seed}: pooled outputs not bit-identical"
    assert gt.backward(G, B, I, O, 0.1) == 0 and gt.read_status() == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd(G, B, I, O, 0.1, Wref) == 0
    for t, (wg, wr, w0) in enumerate(zip(gt.host(), Wref, W)):
        touched = np.zeros(rows[t], bool)
        touched[I[O[t * B]:O[(t + 1) * B]]] = True
        assert_close(wg[touched], wr[touched], f"seed {seed} table {t}")
        assert bits_equal(wg[~touched], w0[~touched]), f"seed {seed} table {t} untouched"
    rc, dref = oracle.dedup(rows, B, I, O)
    rc2, st, d = gpu_dedup(rows, B, I, O)
    assert rc == rc2 == st == 0 and d["num_unique"] == dref["num_unique"]
    for k in ("sorted_keys", "sorted_bags", "unique_keys", "seg_off"):
        assert np.array_equal(d[k], dref[k]), f"seed {seed} {k}"
