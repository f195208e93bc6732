"""Property-based pins of the oracle (hypothesis): for arbitrary small shapes
(E in {4, 8, 16}, mixed table sizes, variable and empty bags, heavy duplicate
rows) the forward equals the dense product A_t W_t of Section II and the
update equals W - lr A_t^T dY, both evaluated in float64 by numpy, within one
float32 ulp; the dedup equals numpy's stable argsort and unique."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

LR = np.float64(np.float32(0.1))


@st.composite
def cases(draw):
    T = draw(st.integers(1, 4))
    rows = tuple(draw(st.integers(1, 40)) for _ in range(T))
    E = draw(st.sampled_from([4, 8, 16]))
    B = draw(st.integers(1, 12))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    rng = np.random.default_rng(seed)
    sizes = rng.integers(0, 9, T * B)
    sizes[rng.random(T * B) < 0.2] = 0  # empty bags
    hot = draw(st.floats(0.0, 0.8))
    I = []
    for k, n in enumerate(sizes):
        m = rows[k // B]
        idx = rng.integers(0, m, n)
        idx[rng.random(n) < hot] = 0  # duplicate-heavy row 0
        I.append(idx)
    I = np.concatenate(I).astype(np.int32) if I else np.zeros(0, np.int32)
    O = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    W = [rng.uniform(-1, 1, (m, E)).astype(np.float32) for m in rows]
    G = rng.standard_normal((T, B, E)).astype(np.float32)
    return rows, E, B, I, O, W, G


def _dense_A(m, B, t, I, O):
    A = np.zeros((B, m))
    for b in range(B):
        k = t * B + b
        for s in range(O[k], O[k + 1]):
            A[b, I[s]] += 1.0
    return A


def _within_ulp(got, ref):
    got = np.asarray(got, np.float32)
    ref32 = np.asarray(ref, np.float64).astype(np.float32)
    sp = np.spacing(np.maximum(np.abs(got), np.abs(ref32)))
    return np.all(np.abs(got.astype(np.float64) - np.asarray(ref, np.float64)) <= sp)


SETTINGS = settings(max_examples=60, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])


@SETTINGS
@given(cases())
def test_forward_is_the_dense_product(oracle, case):
    rows, E, B, I, O, W, G = case
    rc, Y = oracle.forward(W, B, I, O)
    assert rc == oracle.OK
    for t, m in enumerate(rows):
        ref = _dense_A(m, B, t, I, O) @ W[t].astype(np.float64)
        assert _within_ulp(Y[t], ref)
        empty = O[t * B + 1:(t + 1) * B + 1] == O[t * B:(t + 1) * B]
        assert np.all(Y[t][empty].view(np.uint32) == 0)  # +0.0


@SETTINGS
@given(cases())
def test_update_is_the_dense_transpose(oracle, case):
    rows, E, B, I, O, W, G = case
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, B, I, O, 0.1, W1) == oracle.OK
    for t, m in enumerate(rows):
        A = _dense_A(m, B, t, I, O)
        ref = W[t].astype(np.float64) - LR * (A.T @ G[t].astype(np.float64))
        touched = A.sum(axis=0) > 0
        assert _within_ulp(W1[t][touched], ref[touched])
        assert np.array_equal(W1[t][~touched].view(np.uint32), W[t][~touched].view(np.uint32))


@SETTINGS
@given(cases())
def test_dedup_is_numpy_stable_sort_and_unique(oracle, case):
    rows, E, B, I, O, W, G = case
    rc, d = oracle.dedup(rows, B, I, O)
    assert rc == oracle.OK
    base = np.concatenate([[0], np.cumsum(rows)])[:-1]
    bag = np.searchsorted(O, np.arange(I.size), side="right") - 1
    key = (base[bag // B] + I).astype(np.uint32)
    perm = np.argsort(key, kind="stable")
    assert np.array_equal(d["sorted_keys"], key[perm])
    assert np.array_equal(d["sorted_bags"], bag[perm].astype(np.uint32))
    uk, first = np.unique(key, return_index=True)
    assert np.array_equal(d["unique_keys"], uk)
    starts = np.searchsorted(key[perm], uk, side="left")
    assert np.array_equal(d["seg_off"], np.concatenate([starts, [I.size]]).astype(np.int32))
