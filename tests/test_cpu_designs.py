"""The paper's multi-core CPU designs (context for the benchmark) against the
oracle's literal FP32 readings of Algorithms 1 and 2-4: the same sums in the
same order, so bit for bit, whatever the thread count."""
import numpy as np
import pytest

import cpu_designs
import oracle
from embbag_data import random_bags


@pytest.fixture(scope="module", autouse=True)
def _built():
    from cpu_designs import build
    build.build()


def _case(seed, rows, batch, dim, pool, empty, hot):
    rng = np.random.default_rng(seed)
    W = [rng.uniform(-0.5, 0.5, (m, dim)).astype(np.float32) for m in rows]
    I, O = random_bags(rng, rows, batch, pool, empty, hot)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    return W, I, O, G


CASES = [
    (1, (1000, 5, 70000), 90, 16, 30, 0.1, 0.3),   # mixed row counts, empty bags
    (2, (3,), 200, 8, 50, 0.0, 0.6),                # 3 rows for up to 8 owners
    (3, (5000, 20000), 64, 64, 200, 0.2, 0.5),      # long bags, hot rows
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("threads", [1, 3, 8])
def test_forward_equals_the_literal_reading(case, threads):
    seed, rows, batch, dim, pool, empty, hot = case
    W, I, O, _ = _case(seed, rows, batch, dim, pool, empty, hot)
    rc, Y = cpu_designs.forward(W, batch, I, O, threads)
    assert rc == 0
    rc, Yref = oracle.forward(W, batch, I, O, literal=True)
    assert rc == 0
    assert np.array_equal(Y.reshape(-1).view(np.uint32), Yref.reshape(-1).view(np.uint32))


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("threads", [1, 3, 8])
def test_owner_update_equals_the_literal_reading(case, threads):
    seed, rows, batch, dim, pool, empty, hot = case
    W, I, O, G = _case(seed, rows, batch, dim, pool, empty, hot)
    Wc = [w.copy() for w in W]
    assert cpu_designs.backward_sgd(G, batch, I, O, 0.1, Wc, threads) == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd(G, batch, I, O, 0.1, Wref, literal=True) == 0
    for a, b in zip(Wc, Wref):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_bad_arguments():
    W = [np.zeros((4, 8), np.float32)]
    O = np.zeros(3, np.int32)
    assert cpu_designs.forward(W, 2, np.zeros(0, np.int32), O, 0)[0] == -1
    assert cpu_designs.backward_sgd(np.zeros((1, 2, 8), np.float32), 2, np.zeros(0, np.int32), O,
                                    0.1, W, 0) == -1
