"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test checks the oracle against brute force, a library routine, a closed
form or an invariant that follows from the paper's definitions:
  * Section II: L = A^T W with A the multiplicity matrix of the bags;
  * Algorithm 1 (forward), Algorithms 2-4 (backward and sparse SGD update);
  * Section VII (Split-SGD-BF16).
"""
import numpy as np
import pytest
import torch

from embbag_data import get_config, make_batch, make_grads, random_bags, table_values_np

RTOL, ATOL = 1e-5, 1e-6


def _tables(rng, rows, dim, scale=1.0):
    return [(rng.uniform(-scale, scale, size=(m, dim))).astype(np.float32) for m in rows]


def _dense_A(rows_t, batch, t, indices, offsets):
    """Multiplicity matrix A_t[b, r] = number of times bag (t, b) reads row r."""
    A = np.zeros((batch, rows_t), dtype=np.float64)
    for b in range(batch):
        k = t * batch + b
        for s in range(offsets[k], offsets[k + 1]):
            A[b, indices[s]] += 1.0
    return A


def _ulp_close(a, b, ulps=1):
    """|a - b| <= ulps * spacing(max(|a|,|b|)) elementwise, float32."""
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    sp = np.spacing(np.maximum(np.abs(a), np.abs(b)).astype(np.float32))
    return np.all(np.abs(a.astype(np.float64) - b.astype(np.float64)) <= ulps * sp.astype(np.float64))


CASES = [
    # (rows, dim, batch, max_pool, empty_frac, hot_frac, seed)
    ((50, 7, 1), 4, 6, 5, 0.2, 0.0, 1),
    ((30, 40), 16, 9, 12, 0.1, 0.3, 2),
    ((13,), 8, 17, 3, 0.3, 0.5, 3),
    ((100, 100, 3), 12, 5, 20, 0.0, 0.2, 4),
]


# ----------------------------------------------------------------------------
# forward (Algorithm 1; L = A^T W)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("case", CASES)
def test_forward_matches_dense_multiplicity_product(oracle, case):
    rows, dim, batch, maxp, ef, hf, seed = case
    rng = np.random.default_rng(seed)
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, maxp, ef, hf)
    rc, Y = oracle.forward(W, batch, I, O)
    assert rc == oracle.OK
    for t in range(len(rows)):
        ref = _dense_A(rows[t], batch, t, I, O) @ W[t].astype(np.float64)
        assert _ulp_close(Y[t], ref.astype(np.float32), ulps=1)


@pytest.mark.parametrize("case", CASES)
def test_forward_matches_torch_embedding_bag(oracle, case):
    rows, dim, batch, maxp, ef, hf, seed = case
    rng = np.random.default_rng(seed + 100)
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, maxp, ef, hf)
    rc, Y = oracle.forward(W, batch, I, O)
    assert rc == oracle.OK
    for t in range(len(rows)):
        lo, hi = O[t * batch], O[(t + 1) * batch]
        idx = torch.from_numpy(I[lo:hi].astype(np.int64))
        offs = torch.from_numpy((O[t * batch:(t + 1) * batch] - lo).astype(np.int64))
        ref = torch.nn.functional.embedding_bag(idx, torch.from_numpy(W[t]), offs, mode="sum")
        np.testing.assert_allclose(Y[t], ref.numpy(), rtol=RTOL, atol=ATOL)


def test_forward_hand_example(oracle):
    # Integer-valued rows make every sum exact:
    #   table 0 rows: [1,2,3,4], [10,20,30,40], [-5,0,5,100]
    #   bag 0 = {0, 2, 2} -> [1-10, 2+0, 3+10, 4+200] = [-9, 2, 13, 204]
    #   bag 1 = {}        -> [0, 0, 0, 0]
    #   table 1 rows: [0.5,0.5,0.5,0.5], [2,4,8,16]
    #   bag 2 = {1}       -> [2, 4, 8, 16]
    #   bag 3 = {0, 1, 0} -> [3, 5, 9, 17]
    W0 = np.array([[1, 2, 3, 4], [10, 20, 30, 40], [-5, 0, 5, 100]], np.float32)
    W1 = np.array([[0.5] * 4, [2, 4, 8, 16]], np.float32)
    I = np.array([0, 2, 2, 1, 0, 1, 0], np.int32)
    O = np.array([0, 3, 3, 4, 7], np.int32)
    rc, Y = oracle.forward([W0, W1], 2, I, O)
    assert rc == oracle.OK
    expect = np.array([[[-9, 2, 13, 204], [0, 0, 0, 0]],
                       [[2, 4, 8, 16], [3, 5, 9, 17]]], np.float32)
    assert np.array_equal(Y, expect)


def test_forward_exact_special_cases(oracle):
    rng = np.random.default_rng(7)
    W = _tables(rng, (20,), 8)
    # bag0: single look-up (row copy); bag1: [r, r] (= 2 W[r], exact); bag2: empty
    I = np.array([5, 9, 9], np.int32)
    O = np.array([0, 1, 3, 3], np.int32)
    rc, Y = oracle.forward(W, 3, I, O)
    assert rc == oracle.OK
    assert np.array_equal(Y[0, 0].view(np.uint32), W[0][5].view(np.uint32))
    assert np.array_equal(Y[0, 1], 2.0 * W[0][9])
    assert np.array_equal(Y[0, 2].view(np.uint32), np.zeros(8, np.uint32))  # +0.0


def test_forward_permutation_within_bag(oracle):
    rng = np.random.default_rng(8)
    rows = (200,)
    W = _tables(rng, rows, 16)
    I, O = random_bags(rng, rows, 20, 30, 0.0, 0.2)
    rc, Y = oracle.forward(W, 20, I, O)
    I2 = I.copy()
    for k in range(20):
        seg = I2[O[k]:O[k + 1]]
        I2[O[k]:O[k + 1]] = rng.permutation(seg)
    rc2, Y2 = oracle.forward(W, 20, I2, O)
    assert rc == rc2 == oracle.OK
    np.testing.assert_allclose(Y, Y2, rtol=RTOL, atol=ATOL)


# ----------------------------------------------------------------------------
# integer work of the backward (bag ids, keys, stable sort, unique)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("case", CASES)
def test_dedup_matches_numpy(oracle, case):
    rows, dim, batch, maxp, ef, hf, seed = case
    rng = np.random.default_rng(seed + 200)
    I, O = random_bags(rng, rows, batch, maxp, ef, hf)
    rc, d = oracle.dedup(rows, batch, I, O)
    assert rc == oracle.OK
    NS = I.size
    s = np.arange(NS)
    bag = np.searchsorted(O, s, side="right") - 1
    rowbase = np.concatenate([[0], np.cumsum(rows)])
    key = rowbase[bag // batch] + I
    perm = np.argsort(key, kind="stable")
    assert np.array_equal(d["sorted_keys"], key[perm].astype(np.uint32))
    assert np.array_equal(d["sorted_bags"], bag[perm].astype(np.uint32))
    uk, first, counts = np.unique(key, return_index=False, return_counts=True), None, None
    uk, counts = np.unique(key, return_counts=True)
    assert d["num_unique"] == uk.size
    assert np.array_equal(d["unique_keys"], uk.astype(np.uint32))
    assert np.array_equal(d["seg_off"], np.concatenate([[0], np.cumsum(counts)]).astype(np.int32))
    # invariants: keys non-decreasing, ties in increasing position, counts sum to NS
    sk = d["sorted_keys"].astype(np.int64)
    assert np.all(np.diff(sk) >= 0)
    assert d["seg_off"][-1] == NS
    assert d["num_unique"] <= min(NS, sum(rows))


def test_dedup_tie_order_is_lookup_order(oracle):
    # two look-ups of the same row from bags 3 and 1 (in that positional order
    # they appear as bag 1 first because bags are laid out in order) plus a
    # within-bag duplicate: ties must keep increasing look-up position.
    rows = (10,)
    I = np.array([4, 2, 4, 4, 7, 2], np.int32)
    O = np.array([0, 2, 4, 6], np.int32)       # bags: {4,2} {4,4} {7,2}
    rc, d = oracle.dedup(rows, 3, I, O)
    assert rc == oracle.OK
    assert d["sorted_keys"].tolist() == [2, 2, 4, 4, 4, 7]
    assert d["sorted_bags"].tolist() == [0, 2, 0, 1, 1, 2]
    assert d["unique_keys"].tolist() == [2, 4, 7]
    assert d["seg_off"].tolist() == [0, 2, 5, 6]


# ----------------------------------------------------------------------------
# fused backward + sparse SGD (Algorithms 2-4)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("case", CASES)
def test_update_matches_dense_brute_force(oracle, case):
    rows, dim, batch, maxp, ef, hf, seed = case
    rng = np.random.default_rng(seed + 300)
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, maxp, ef, hf)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    lr = 0.1
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, batch, I, O, lr, W1) == oracle.OK
    for t in range(len(rows)):
        A = _dense_A(rows[t], batch, t, I, O)
        grad = A.T @ G[t].astype(np.float64)                 # dense A^T dY
        touched = A.sum(axis=0) > 0
        ref = W[t].astype(np.float64) - np.float64(np.float32(lr)) * grad
        assert _ulp_close(W1[t][touched], ref[touched].astype(np.float32), ulps=1)
        assert np.array_equal(W1[t][~touched].view(np.uint32), W[t][~touched].view(np.uint32))


@pytest.mark.parametrize("case", CASES)
def test_update_matches_torch_index_add(oracle, case):
    rows, dim, batch, maxp, ef, hf, seed = case
    rng = np.random.default_rng(seed + 400)
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, maxp, ef, hf)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    lr = 0.1
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, batch, I, O, lr, W1) == oracle.OK
    for t in range(len(rows)):
        lo, hi = O[t * batch], O[(t + 1) * batch]
        bag = np.searchsorted(O, np.arange(lo, hi), side="right") - 1 - t * batch
        ref = torch.from_numpy(W[t].copy())
        src = -lr * torch.from_numpy(G[t])[torch.from_numpy(bag)]
        ref.index_add_(0, torch.from_numpy(I[lo:hi].astype(np.int64)), src)
        np.testing.assert_allclose(W1[t], ref.numpy(), rtol=RTOL, atol=ATOL)


def test_update_hand_example(oracle):
    # lr = 0.5, integer-valued data: every result is exact.
    #   W rows: r0 = [1,1,1,1], r1 = [2,2,2,2], r2 = [3,3,3,3]
    #   bag0 = {0, 2, 0} with dY0 = [2, 4, 6, 8]
    #   bag1 = {2}       with dY1 = [-2, 0, 2, 4]
    #   row 0: G = 2*dY0 = [4, 8, 12, 16]  -> W = [1-2, 1-4, 1-6, 1-8] = [-1,-3,-5,-7]
    #   row 2: G = dY0 + dY1 = [0,4,8,12]  -> W = [3, 1, -1, -3]
    #   row 1: untouched
    W = [np.array([[1] * 4, [2] * 4, [3] * 4], np.float32)]
    G = np.array([[[2, 4, 6, 8], [-2, 0, 2, 4]]], np.float32)
    I = np.array([0, 2, 0, 2], np.int32)
    O = np.array([0, 3, 4], np.int32)
    assert oracle.backward_sgd(G, 2, I, O, 0.5, W) == oracle.OK
    assert W[0].tolist() == [[-1, -3, -5, -7], [2, 2, 2, 2], [3, 1, -1, -3]]


def test_update_invariants(oracle):
    rng = np.random.default_rng(11)
    rows = (64, 9)
    dim, batch = 8, 12
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, 6, 0.2, 0.3)
    G = rng.standard_normal((2, batch, dim)).astype(np.float32)
    # lr = 0 leaves every bit in place
    W0 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, batch, I, O, 0.0, W0) == oracle.OK
    for a, b in zip(W0, W):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    # conservation: sum over rows of (W' - W) = -lr * sum over look-ups of dY[bag]
    lr = 0.25
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, batch, I, O, lr, W1) == oracle.OK
    for t in range(2):
        lo, hi = O[t * batch], O[(t + 1) * batch]
        bag = np.searchsorted(O, np.arange(lo, hi), side="right") - 1
        lhs = (W1[t].astype(np.float64) - W[t]).sum(axis=0)
        rhs = -lr * G.reshape(-1, dim)[bag].astype(np.float64).sum(axis=0)
        np.testing.assert_allclose(lhs, rhs, rtol=1e-5, atol=1e-5)


def test_update_single_hit_and_double_hit(oracle):
    rng = np.random.default_rng(12)
    W = _tables(rng, (10,), 4)
    g = rng.standard_normal(4).astype(np.float32)
    lr = np.float32(0.1)
    # row 3 hit once; row 6 hit twice by the same bag -> W - 2 lr g
    I = np.array([3, 6, 6], np.int32)
    O = np.array([0, 1, 3], np.int32)
    G = np.stack([g, g])[None]
    W1 = [W[0].copy()]
    assert oracle.backward_sgd(G, 2, I, O, float(lr), W1) == oracle.OK
    once = (W[0][3] - lr * g).astype(np.float32)       # FP32 evaluation
    assert _ulp_close(W1[0][3], once, ulps=1)
    twice = W[0][6].astype(np.float64) - 2 * np.float64(lr) * g.astype(np.float64)
    assert _ulp_close(W1[0][6], twice.astype(np.float32), ulps=1)


def test_literal_order_within_tolerance(oracle):
    """Algorithms 1 and 3 in FP32 sequential order land within the tolerance."""
    cfg = get_config("tiny")
    rng = np.random.default_rng(13)
    W = [table_values_np(cfg.seed, t, np.arange(cfg.rows[t]), cfg.dim, cfg.value_scale[t])
         for t in range(cfg.num_tables)]
    I, O = make_batch(cfg, 0)
    G = make_grads(cfg, 0)
    rc, Y = oracle.forward(W, cfg.batch, I, O)
    rc2, Y2 = oracle.forward(W, cfg.batch, I, O, literal=True)
    assert rc == rc2 == oracle.OK
    np.testing.assert_allclose(Y2, Y, rtol=RTOL, atol=ATOL)
    Wa = [w.copy() for w in W]
    Wb = [w.copy() for w in W]
    assert oracle.backward_sgd(G, cfg.batch, I, O, cfg.lr, Wa) == oracle.OK
    assert oracle.backward_sgd(G, cfg.batch, I, O, cfg.lr, Wb, literal=True) == oracle.OK
    for a, b in zip(Wa, Wb):
        np.testing.assert_allclose(b, a, rtol=RTOL, atol=ATOL)
    del rng


def _fp32_forward_in_order(W, batch, I, O):
    """Algorithm 1 with an FP32 accumulator, look-ups in increasing s: numpy
    float32 additions, one look-up at a time (IEEE single rounding each step)."""
    T, E = len(W), W[0].shape[1]
    Y = np.zeros((T, batch, E), np.float32)
    for k in range(T * batch):
        t, b = divmod(k, batch)
        y = np.zeros(E, np.float32)
        for s in range(O[k], O[k + 1]):
            y = (y + W[t][I[s]]).astype(np.float32)
        Y[t, b] = y
    return Y


def _fp32_update_in_order(G, batch, I, O, lr, W, reverse=False):
    """Algorithm 2 then Algorithm 3 applied one look-up at a time in increasing
    s, in FP32: w <- w + fl(alpha * dW[s]) with alpha = -lr (Section III-A;
    within one row this is also Algorithm 4's order).  `reverse` walks the
    look-ups from the last one instead (only to show that order matters)."""
    T, E = len(W), W[0].shape[1]
    alpha = np.float32(-lr)
    out = [w.copy() for w in W]
    ks = range(T * batch - 1, -1, -1) if reverse else range(T * batch)
    for k in ks:
        t, b = divmod(k, batch)
        g = G[t, b].astype(np.float32)
        ss = range(O[k], O[k + 1])
        for s in (reversed(ss) if reverse else ss):
            step = (alpha * g).astype(np.float32)
            out[t][I[s]] = (out[t][I[s]] + step).astype(np.float32)
    return out


def test_literal_readings_absorb_in_order(oracle):
    """Worked example where FP32 order decides the bits.  Forward: a bag reads
    a row of 1.0 and then four rows of 2^-24 (half an ulp of 1): each addition
    ties and rounds back to 1.0, so Algorithm 1 in FP32 gives exactly 1.0,
    while the small rows first (reversed order) give 1 + 2^-22 and an FP64
    accumulator 1 + 2^-22 too.  Update: a zero row receives a step of +1 and
    then four steps of +2^-25 (lr = 1): sequential FP32 keeps 1.0 (each step is
    a quarter ulp), reversed order or an FP64 sum gives 1 + 2^-23."""
    E = 4
    W = [np.array([[1.0] * E, [2.0 ** -24] * E, [0.0] * E], np.float32)]
    I = np.array([0, 1, 1, 1, 1], np.int32)
    O = np.array([0, 5], np.int32)
    rc, Y = oracle.forward(W, 1, I, O, literal=True)
    assert rc == oracle.OK
    assert np.array_equal(Y[0, 0].view(np.uint32), np.full(E, np.float32(1.0)).view(np.uint32))
    rc, Yd = oracle.forward(W, 1, I, O)  # the FP64 definition: exact sum, rounded once
    assert rc == oracle.OK and np.all(Yd[0, 0] == np.float32(1.0 + 4 * 2.0 ** -24))
    # update: bag 0 = [row 2], bag 1 = [row 2] x 4; dY chosen so that -lr*g is
    # +1 for bag 0 and +2^-25 for bag 1
    I = np.array([2, 2, 2, 2, 2], np.int32)
    O = np.array([0, 1, 5], np.int32)
    G = np.array([[[-1.0] * E, [-(2.0 ** -25)] * E]], np.float32)
    Wl = [W[0].copy()]
    assert oracle.backward_sgd(G, 2, I, O, 1.0, Wl, literal=True) == oracle.OK
    assert np.array_equal(Wl[0][2], np.full(E, np.float32(1.0)))
    assert np.array_equal(Wl[0][:2], W[0][:2])
    Wd = [W[0].copy()]
    assert oracle.backward_sgd(G, 2, I, O, 1.0, Wd) == oracle.OK
    assert np.all(Wd[0][2] == np.float32(1.0 + 2.0 ** -23))


@pytest.mark.parametrize("seed", [21, 22, 23])
def test_literal_readings_follow_fp32_order(oracle, seed):
    """The literal readings are Algorithm 1 and Algorithm 3 in FP32, look-ups in
    increasing s: bit for bit what a numpy float32 loop in that order gives,
    on values whose magnitudes span ten decades (so sums depend on order:
    the test also checks that reversed order changes some bits)."""
    rng = np.random.default_rng(seed)
    rows, dim, batch = (40, 9), 8, 12
    mag = lambda *sh: (10.0 ** rng.uniform(-8, 2, sh)) * rng.choice([-1.0, 1.0], sh)
    W = [mag(m, dim).astype(np.float32) for m in rows]
    I, O = random_bags(rng, rows, batch, 24, 0.1, 0.5)
    G = mag(len(rows), batch, dim).astype(np.float32)
    lr = 0.37
    rc, Y = oracle.forward(W, batch, I, O, literal=True)
    assert rc == oracle.OK
    Yexp = _fp32_forward_in_order(W, batch, I, O)
    assert np.array_equal(Y.view(np.uint32), Yexp.view(np.uint32))
    Irev = np.concatenate([I[O[k]:O[k + 1]][::-1] for k in range(len(O) - 1)]).astype(np.int32)
    assert not np.array_equal(_fp32_forward_in_order(W, batch, Irev, O), Yexp)
    Wl = [w.copy() for w in W]
    assert oracle.backward_sgd(G, batch, I, O, lr, Wl, literal=True) == oracle.OK
    Wexp = _fp32_update_in_order(G, batch, I, O, lr, W)
    for a, b in zip(Wl, Wexp):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    Wrev = _fp32_update_in_order(G, batch, I, O, lr, W, reverse=True)
    assert any(not np.array_equal(a, b) for a, b in zip(Wrev, Wexp))


# ----------------------------------------------------------------------------
# validation and status codes
# ----------------------------------------------------------------------------
def test_status_codes(oracle):
    rows = (10, 5)
    I = np.array([1, 2, 3, 4], np.int32)
    O = np.array([0, 1, 2, 3, 4], np.int32)
    assert oracle.validate(rows, 8, 2, I, O) == oracle.OK
    assert oracle.validate(rows, 6, 2, I, O) == oracle.ERR_INVALID_ARG     # E % 4
    assert oracle.validate(rows, 2048, 2, I, O) == oracle.ERR_INVALID_ARG  # E > 1024
    assert oracle.validate(rows, 8, -1, I, O) == oracle.ERR_INVALID_ARG
    assert oracle.validate(rows, 8, 2, I, O, num_tables=0) == oracle.ERR_INVALID_ARG
    assert oracle.validate((10, 0), 8, 2, I, O) == oracle.ERR_INVALID_ARG
    # indices and offsets are int32: more than 2^31 - 1 look-ups is an argument
    # error, found before the arrays are read; 2^31 - 1 itself passes the
    # argument checks (here the offsets then disagree with it)
    assert oracle.validate(rows, 8, 2, I, O, num_indices=2 ** 31) == oracle.ERR_INVALID_ARG
    assert oracle.validate(rows, 8, 2, I, O, num_indices=2 ** 31 - 1) == oracle.ERR_OFFSETS
    bad = O.copy(); bad[0] = 1
    assert oracle.validate(rows, 8, 2, I, bad) == oracle.ERR_OFFSETS
    bad = np.array([0, 2, 1, 3, 4], np.int32)
    assert oracle.validate(rows, 8, 2, I, bad) == oracle.ERR_OFFSETS
    bad = np.array([0, 1, 2, 3, 3], np.int32)
    assert oracle.validate(rows, 8, 2, I, bad) == oracle.ERR_OFFSETS      # O[TB] != NS
    badI = I.copy(); badI[3] = 5                                          # table 1 has 5 rows
    assert oracle.validate(rows, 8, 2, badI, O) == oracle.ERR_INDEX_RANGE
    badI = I.copy(); badI[0] = -1
    assert oracle.validate(rows, 8, 2, badI, O) == oracle.ERR_INDEX_RANGE
    # offsets are checked before indices
    both = np.array([0, 2, 1, 3, 4], np.int32)
    assert oracle.validate(rows, 8, 2, badI, both) == oracle.ERR_OFFSETS


def test_errors_leave_tables_untouched(oracle):
    rng = np.random.default_rng(14)
    W = _tables(rng, (10, 5), 8)
    G = rng.standard_normal((2, 2, 8)).astype(np.float32)
    I = np.array([1, 2, 3, 5], np.int32)      # 5 is out of range for table 1
    O = np.array([0, 1, 2, 3, 4], np.int32)
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, 2, I, O, 0.1, W1) == oracle.ERR_INDEX_RANGE
    for a, b in zip(W1, W):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_empty_inputs(oracle):
    W = [np.ones((4, 4), np.float32)]
    rc, Y = oracle.forward(W, 3, np.zeros(0, np.int32), np.zeros(4, np.int32))
    assert rc == oracle.OK and np.array_equal(Y.view(np.uint32), np.zeros_like(Y).view(np.uint32))
    rc, Y = oracle.forward(W, 0, np.zeros(0, np.int32), np.zeros(1, np.int32))
    assert rc == oracle.OK and Y.shape == (1, 0, 4)
    W1 = [W[0].copy()]
    G = np.ones((1, 3, 4), np.float32)
    assert oracle.backward_sgd(G, 3, np.zeros(0, np.int32), np.zeros(4, np.int32), 0.1, W1) == 0
    assert np.array_equal(W1[0], W[0])


# ----------------------------------------------------------------------------
# Split-SGD-BF16 (Section VII)
# ----------------------------------------------------------------------------
@pytest.mark.slow
def test_split_roundtrip_exhaustive(oracle):
    assert oracle.split_roundtrip_mismatches(0, 1 << 32) == 0


def test_split_roundtrip_sampled(oracle):
    assert oracle.split_roundtrip_mismatches(0, 1 << 20) == 0
    assert oracle.split_roundtrip_mismatches((1 << 32) - (1 << 20), 1 << 20) == 0
    assert oracle.split_roundtrip_mismatches(0x3F800000 - 4096, 8192) == 0


def test_split_hi_is_bf16_truncation(oracle):
    rng = np.random.default_rng(15)
    w = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.float32([0.0, -0.0, 1.0, -1.0, 3.14159, 1e-30, -1e30])])
    hi, lo = oracle.split(w)
    hv = (hi.astype(np.uint32) << 16).view(np.float32)
    # hi is a BF16 number: a round trip through torch.bfloat16 keeps it
    t = torch.from_numpy(hv)
    assert torch.equal(t.to(torch.bfloat16).to(torch.float32), t)
    # ... and it is w truncated toward zero: same sign, |hv| <= |w| < next BF16 up
    assert np.all(np.signbit(hv) == np.signbit(w))
    assert np.all(np.abs(hv) <= np.abs(w))
    nz = w != 0
    assert np.all(np.abs(w[nz] - hv[nz]) < np.abs(hv[nz]) * 2.0 ** -7)
    # torch's round-to-nearest BF16 is either the truncation or the next value away from zero
    rne = torch.from_numpy(w).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.all((rne == hv) | (np.abs(rne) > np.abs(hv)))


def test_split_forward_reads_high_half_only(oracle):
    rng = np.random.default_rng(16)
    rows = (40, 25)
    W = _tables(rng, rows, 8)
    I, O = random_bags(rng, rows, 7, 6, 0.1, 0.2)
    his, los = zip(*[oracle.split(w) for w in W])
    rc, Ys = oracle.forward_split(list(his), 7, I, O)
    masked = [(w.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32) for w in W]
    rc2, Y = oracle.forward(masked, 7, I, O)
    assert rc == rc2 == oracle.OK
    assert np.array_equal(Ys.view(np.uint32), Y.view(np.uint32))
    # garbage in the low halves changes nothing in the forward
    rc3, Ys3 = oracle.forward_split(list(his), 7, I, O)
    assert np.array_equal(Ys3, Ys)


def test_split_update_equals_fp32_update(oracle):
    rng = np.random.default_rng(17)
    rows = (60, 33)
    W = _tables(rng, rows, 12)
    I, O = random_bags(rng, rows, 9, 8, 0.1, 0.3)
    G = rng.standard_normal((2, 9, 12)).astype(np.float32)
    hi, lo = zip(*[oracle.split(w) for w in W])
    hi, lo = [h.copy() for h in hi], [l.copy() for l in lo]
    assert oracle.backward_sgd_split(G, 9, I, O, 0.1, hi, lo) == oracle.OK
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, 9, I, O, 0.1, W1) == oracle.OK
    for h, l, w in zip(hi, lo, W1):
        assert np.array_equal(oracle.combine(h, l).view(np.uint32), w.view(np.uint32))


# ----------------------------------------------------------------------------
# BF16 activations (Section VII: forward and backward in BF16, update in FP32)
# ----------------------------------------------------------------------------
def _torch_bf16_bits(x):
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _torch_bf16_widen(h):
    return torch.from_numpy(h.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()


def test_bf16_round_matches_torch(oracle):
    rng = np.random.default_rng(18)
    ties = (rng.integers(0, 1 << 16, 50000).astype(np.uint32) << 16) | np.uint32(0x8000)
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32) * np.float32(1e-3),
        rng.integers(0, 1 << 32, 200000, dtype=np.uint64).astype(np.uint32).view(np.float32),
        ties.view(np.float32),  # exact midpoints, odd and even last bit, both signs
        np.float32([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, 3.4028235e38, -3.4028235e38,
                    1e-45, -1e-45, 1.1754944e-38, 1.0, -1.0]),
    ])
    x = x[~np.isnan(x)]
    assert np.array_equal(oracle.bf16_round(x), _torch_bf16_bits(x))
    # halfway between the largest finite BF16 and 2^128 rounds to infinity (ties to even)
    assert oracle.bf16_round(np.uint32([0x7F7F8000]).view(np.float32))[0] == 0x7F80
    assert oracle.bf16_round(np.uint32([0x7F7E8000]).view(np.float32))[0] == 0x7F7E
    assert np.isnan(oracle.bf16_widen(oracle.bf16_round(np.float32([np.nan]))))[0]


def test_bf16_widen_matches_torch(oracle):
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    w = oracle.bf16_widen(h)
    ref = _torch_bf16_widen(h)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(w), nan)
    assert np.array_equal(w[~nan].view(np.uint32), ref[~nan].view(np.uint32))
    assert np.array_equal(oracle.bf16_round(w[~nan]), h[~nan])  # BF16 values round to themselves


@pytest.mark.parametrize("case", CASES)
def test_bf16_act_forward_matches_torch(oracle, case):
    rows, dim, batch, maxp, ef, hf, seed = case
    rng = np.random.default_rng(seed + 300)
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, maxp, ef, hf)
    his = [oracle.split(w)[0] for w in W]
    rc, Yb = oracle.forward_split_bf16_act(his, batch, I, O)
    assert rc == oracle.OK and Yb.dtype == np.uint16
    for t in range(len(rows)):
        # sums of BF16 values (8 significant bits) over a 2^-32 range are exact in float64
        Wt = torch.from_numpy(_torch_bf16_widen(his[t])).double()
        lo, hi = O[t * batch], O[(t + 1) * batch]
        idx = torch.from_numpy(I[lo:hi].astype(np.int64))
        offs = torch.from_numpy((O[t * batch:(t + 1) * batch] - lo).astype(np.int64))
        y = torch.nn.functional.embedding_bag(idx, Wt, offs, mode="sum").float()
        assert np.array_equal(Yb[t], _torch_bf16_bits(y.numpy()))


def test_bf16_act_update_uses_the_exactly_widened_gradient(oracle):
    rng = np.random.default_rng(20)
    rows, E, B = (60, 33), 12, 9
    W = _tables(rng, rows, E)
    I, O = random_bags(rng, rows, B, 8, 0.1, 0.3)
    Gb = _torch_bf16_bits(rng.standard_normal((2, B, E)).astype(np.float32))
    Gw = _torch_bf16_widen(Gb)
    hi, lo = zip(*[oracle.split(w) for w in W])
    h1, l1 = [h.copy() for h in hi], [l.copy() for l in lo]
    assert oracle.backward_sgd_split_bf16_act(Gb, B, I, O, 0.1, h1, l1) == oracle.OK
    # dense brute force on the widened gradient: W - lr * A^T G in float64
    for t in range(2):
        A = _dense_A(rows[t], B, t, I, O)
        ref = W[t].astype(np.float64) - np.float64(np.float32(0.1)) * (A.T @ Gw[t].astype(np.float64))
        got = oracle.combine(h1[t], l1[t])
        touched = A.sum(axis=0) > 0
        assert _ulp_close(got[touched], ref[touched].astype(np.float32))
        assert np.array_equal(got[~touched].view(np.uint32), W[t][~touched].view(np.uint32))


# ----------------------------------------------------------------------------
# weighted and mean pooling (Section II's L = A^T W with weights a_p)
# ----------------------------------------------------------------------------
def _dense_A_weighted(rows_t, batch, t, indices, offsets, weights=None, mean=False):
    A = np.zeros((batch, rows_t), dtype=np.float64)
    for b in range(batch):
        k = t * batch + b
        n = offsets[k + 1] - offsets[k]
        for s in range(offsets[k], offsets[k + 1]):
            c = 1.0 if weights is None else float(weights[s])
            if mean:
                c /= n
            A[b, indices[s]] += c
    return A


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("mode", ["weighted", "mean"])
def test_weighted_and_mean_match_dense_and_torch(oracle, case, mode):
    rows, dim, batch, maxp, ef, hf, seed = case
    rng = np.random.default_rng(seed + 500)
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, maxp, ef, hf)
    a = rng.uniform(-2, 2, I.size).astype(np.float32) if mode == "weighted" else None
    m = oracle.POOL_MEAN if mode == "mean" else oracle.POOL_SUM
    rc, Y = oracle.forward_weighted(W, batch, I, O, a, m)
    assert rc == oracle.OK
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd_weighted(G, batch, I, O, 0.1, W1, a, m) == oracle.OK
    for t in range(len(rows)):
        A = _dense_A_weighted(rows[t], batch, t, I, O, a, mode == "mean")
        assert _ulp_close(Y[t], (A @ W[t].astype(np.float64)).astype(np.float32), ulps=1)
        grad = A.T @ G[t].astype(np.float64)
        touched = np.zeros(rows[t], bool)
        touched[I[O[t * batch]:O[(t + 1) * batch]]] = True
        ref = W[t].astype(np.float64) - np.float64(np.float32(0.1)) * grad
        assert _ulp_close(W1[t][touched], ref[touched].astype(np.float32), ulps=1)
        assert np.array_equal(W1[t][~touched].view(np.uint32), W[t][~touched].view(np.uint32))
        # library routine
        lo, hi = O[t * batch], O[(t + 1) * batch]
        idx = torch.from_numpy(I[lo:hi].astype(np.int64))
        offs = torch.from_numpy((O[t * batch:(t + 1) * batch] - lo).astype(np.int64))
        psw = None if a is None else torch.from_numpy(a[lo:hi])
        ref_t = torch.nn.functional.embedding_bag(idx, torch.from_numpy(W[t]), offs,
                                                  mode="mean" if mode == "mean" else "sum",
                                                  per_sample_weights=psw)
        np.testing.assert_allclose(Y[t], ref_t.numpy(), rtol=RTOL, atol=ATOL)


def test_weighted_special_cases(oracle):
    rng = np.random.default_rng(31)
    rows, dim, batch = (40, 25), 8, 7
    W = _tables(rng, rows, dim)
    I, O = random_bags(rng, rows, batch, 6, 0.2, 0.3)
    # unit weights reproduce the plain sum bit for bit
    rc, Y1 = oracle.forward_weighted(W, batch, I, O, np.ones(I.size, np.float32))
    rc2, Y0 = oracle.forward(W, batch, I, O)
    assert rc == rc2 == 0 and np.array_equal(Y1.view(np.uint32), Y0.view(np.uint32))
    G = rng.standard_normal((2, batch, dim)).astype(np.float32)
    Wa, Wb = [w.copy() for w in W], [w.copy() for w in W]
    assert oracle.backward_sgd_weighted(G, batch, I, O, 0.1, Wa, np.ones(I.size, np.float32)) == 0
    assert oracle.backward_sgd(G, batch, I, O, 0.1, Wb) == 0
    for a_, b_ in zip(Wa, Wb):
        assert np.array_equal(a_.view(np.uint32), b_.view(np.uint32))
    # mean of n copies of one row is that row; an empty bag is +0.0
    I2 = np.array([3, 3, 3, 5], np.int32)
    O2 = np.array([0, 3, 3, 4], np.int32)
    rc, Ym = oracle.forward_weighted([W[0]], 3, I2, O2, None, oracle.POOL_MEAN)
    assert rc == 0
    assert np.array_equal(Ym[0, 0], W[0][3]) and np.array_equal(Ym[0, 2], W[0][5])
    assert np.array_equal(Ym[0, 1].view(np.uint32), np.zeros(dim, np.uint32))
    # a zero weight contributes nothing: same as dropping that look-up (forward and update)
    a = rng.uniform(0.5, 2.0, I.size).astype(np.float32)
    zero = rng.random(I.size) < 0.3
    a[zero] = 0.0
    keep = ~zero
    bag = np.searchsorted(O, np.arange(I.size), side="right") - 1
    O3 = np.zeros_like(O)
    O3[1:] = np.cumsum(np.bincount(bag[keep], minlength=O.size - 1))
    rc, Yz = oracle.forward_weighted(W, batch, I, O, a)
    rc2, Yd = oracle.forward_weighted(W, batch, np.ascontiguousarray(I[keep]), O3,
                                      np.ascontiguousarray(a[keep]))
    assert rc == rc2 == 0 and np.array_equal(Yz.view(np.uint32), Yd.view(np.uint32))
    Wa, Wb = [w.copy() for w in W], [w.copy() for w in W]
    assert oracle.backward_sgd_weighted(G, batch, I, O, 0.1, Wa, a) == 0
    assert oracle.backward_sgd_weighted(G, batch, np.ascontiguousarray(I[keep]), O3, 0.1, Wb,
                                        np.ascontiguousarray(a[keep])) == 0
    for a_, b_ in zip(Wa, Wb):
        assert np.array_equal(a_.view(np.uint32), b_.view(np.uint32))
    # weights with mean pooling are rejected (torch allows weights with sum only)
    assert oracle.forward_weighted(W, batch, I, O, np.ones(I.size, np.float32),
                                   oracle.POOL_MEAN)[0] == oracle.ERR_INVALID_ARG
