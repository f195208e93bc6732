"""GPU parity at the full benchmark sizes, in the launch configuration bench.py
times (prepare + apply on one stream, tables filled on the device).

The Large-shaped (98.3 GB) and MLPerf-style (~94 GB) tables do not fit the
host, so the oracle runs in touched-rows mode: it gets a compact copy of every
table holding only the rows the batch names (regenerated from the
counter-based generator, never read back from the GPU path), with indices
remapped monotonically, so sums, sort order and segments are unchanged.
Checked: every pooled output and every touched row (within tolerance), 10^4
sampled untouched rows per table group (bit-identical), the full integer
dedup (bit-exact), and the device fill against the host generator.  The
split-storage runs (Section VII) check FP32 and BF16 pooled outputs and the
update driven by an FP32 (Large-shaped) or BF16 (MLPerf-style) gradient.

Two more runs go to the size limits of one call (2^31 - 1 - 2^16 look-ups,
then also T*B + 1 = 2^31 - 1 offsets) with inputs whose every expected value
has an exact closed form, checked bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2005_04680_amd as pk
from embbag_data import (fill_table_torch, fill_tables_torch, get_config, make_batch, make_grads,
                         make_weights, table_rows_torch, table_values_np)
from gpu_util import (DEV, assert_bf16_bracket, assert_close, bf16_bits, bits_equal, gpu_dedup, log,
                      require_gpu, to_bf16_bits)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _run(name):
    cfg = get_config(name)
    T, B, E, P, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.pooling, cfg.num_indices
    log(f"[full] {name}: filling {cfg.table_bytes / 1e9:.1f} GB on the device")
    W = [torch.empty((m, E), dtype=torch.float32, device=DEV) for m in cfg.rows]
    fill_tables_torch(cfg, W)
    I, O = make_batch(cfg, 0, device=DEV)
    G = make_grads(cfg, 0)
    rng = np.random.default_rng(7)

    # the device fill is the host generator, bit for bit (sampled rows)
    for t in (0, T - 1):
        r = np.unique(rng.integers(0, cfg.rows[t], 64))
        host = table_values_np(cfg.seed, t, r, E, cfg.value_scale[t])
        dev = W[t][torch.from_numpy(r).to(DEV)].cpu().numpy()
        assert bits_equal(dev, host), f"device fill differs from the host generator, table {t}"

    # compact tables for the oracle: touched rows + sampled untouched rows
    log(f"[full] {name}: building compact tables")
    sel, I_c, untouched = [], np.empty_like(I), []
    for t in range(T):
        lo, hi = t * B * P, (t + 1) * B * P
        touched = np.unique(I[lo:hi])
        cand = rng.integers(0, cfg.rows[t], 2000)
        cand = np.setdiff1d(np.unique(cand), touched)[: max(1, 10000 // T)]
        rows = np.union1d(touched, cand)
        I_c[lo:hi] = np.searchsorted(rows, I[lo:hi])
        sel.append(rows)
        untouched.append(cand)
    W_c = [table_rows_torch(cfg.seed, t, torch.from_numpy(sel[t]).to(DEV), E,
                            cfg.value_scale[t]).cpu().numpy() for t in range(T)]

    # GPU path, as bench.py runs it
    log(f"[full] {name}: GPU forward + backward")
    Id, Od, Gd = (torch.from_numpy(a).to(DEV) for a in (I, O, G))
    Y = torch.empty((T, B, E), dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(T, B, NS, E), dtype=torch.uint8, device=DEV)
    assert pk.embbag_forward(W, B, Id, Od, Y, status) == 0
    assert pk.embbag_backward_prepare(cfg.rows, E, B, Id, Od, ws, status) == 0
    assert pk.embbag_backward_apply_sgd(Gd, B, NS, cfg.lr, W, ws) == 0
    assert pk.embbag_status_read(status) == 0
    Y = Y.cpu().numpy()
    W_gpu = [W[t][torch.from_numpy(sel[t]).to(DEV)].cpu().numpy() for t in range(T)]
    del W
    torch.cuda.empty_cache()

    log(f"[full] {name}: oracle forward ({NS} look-ups)")
    rc, Y_ref = oracle.forward(W_c, B, I_c, O)
    assert rc == 0
    assert_close(Y, Y_ref, f"{name} pooled")
    assert bits_equal(Y, Y_ref), f"{name}: pooled outputs not bit-identical"
    log(f"[full] {name}: oracle backward")
    W_ref = [w.copy() for w in W_c]
    assert oracle.backward_sgd(G, B, I_c, O, cfg.lr, W_ref) == 0
    for t in range(T):
        is_u = np.isin(sel[t], untouched[t])
        assert_close(W_gpu[t][~is_u], W_ref[t][~is_u], f"{name} table {t} touched rows")
        assert bits_equal(W_gpu[t][is_u], W_c[t][is_u]), f"{name} table {t} untouched rows changed"

    log(f"[full] {name}: dedup, bit-exact")
    rc, d_ref = oracle.dedup(cfg.rows, B, I, O)
    assert rc == 0
    rc, st, d = gpu_dedup(cfg.rows, B, I, O)
    assert rc == 0 and st == 0 and d["num_unique"] == d_ref["num_unique"]
    for k in ("sorted_keys", "sorted_bags", "unique_keys", "seg_off"):
        assert np.array_equal(d[k], d_ref[k]), k
    log(f"[full] {name}: ok, U = {d['num_unique']}")


def _run_split(name, grad_bf16):
    """Split-SGD-BF16 storage at full size: FP32 and BF16 pooled outputs from
    the hi halves, then the update driven by an FP32 or a BF16 gradient."""
    cfg = get_config(name)
    T, B, E, P, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.pooling, cfg.num_indices
    log(f"[full] {name}: filling {cfg.table_bytes / 1e9:.1f} GB of hi/lo halves on the device")
    hi = [torch.empty((m, E), dtype=torch.int16, device=DEV) for m in cfg.rows]
    lo = [torch.empty((m, E), dtype=torch.int16, device=DEV) for m in cfg.rows]
    for t, m in enumerate(cfg.rows):
        tmp = torch.empty((m, E), dtype=torch.float32, device=DEV)
        fill_table_torch(cfg, t, tmp)
        assert pk.embbag_split_fp32(tmp, hi[t], lo[t]) == 0
        del tmp
    I, O = make_batch(cfg, 0, device=DEV)
    G = make_grads(cfg, 0)
    rng = np.random.default_rng(8)

    # the device halves are the host generator's values, split on the host
    for t in (0, T - 1):
        r = np.unique(rng.integers(0, cfg.rows[t], 64))
        h_ref, l_ref = oracle.split(table_values_np(cfg.seed, t, r, E, cfg.value_scale[t]))
        rd = torch.from_numpy(r).to(DEV)
        assert bits_equal(hi[t][rd].cpu().numpy().view(np.uint16), h_ref), f"hi, table {t}"
        assert bits_equal(lo[t][rd].cpu().numpy().view(np.uint16), l_ref), f"lo, table {t}"

    log(f"[full] {name}: building compact tables")
    sel, I_c, untouched = [], np.empty_like(I), []
    for t in range(T):
        a, b = t * B * P, (t + 1) * B * P
        touched = np.unique(I[a:b])
        cand = rng.integers(0, cfg.rows[t], 2000)
        cand = np.setdiff1d(np.unique(cand), touched)[: max(1, 10000 // T)]
        rows = np.union1d(touched, cand)
        I_c[a:b] = np.searchsorted(rows, I[a:b])
        sel.append(rows)
        untouched.append(cand)
    hl_c = [oracle.split(table_rows_torch(cfg.seed, t, torch.from_numpy(sel[t]).to(DEV), E,
                                          cfg.value_scale[t]).cpu().numpy()) for t in range(T)]
    hi_c = [h for h, _ in hl_c]
    lo_c = [l for _, l in hl_c]

    log(f"[full] {name}: GPU forward (FP32 and BF16 outputs) + backward "
        f"({'BF16' if grad_bf16 else 'FP32'} gradient)")
    Id, Od = (torch.from_numpy(a).to(DEV) for a in (I, O))
    Y = torch.empty((T, B, E), dtype=torch.float32, device=DEV)
    Yb = torch.empty((T, B, E), dtype=torch.bfloat16, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(T, B, NS, E), dtype=torch.uint8, device=DEV)
    assert pk.embbag_forward_split_bf16(hi, B, Id, Od, Y, status) == 0
    assert pk.embbag_forward_split_bf16_act(hi, B, Id, Od, Yb, status) == 0
    assert pk.embbag_backward_prepare(cfg.rows, E, B, Id, Od, ws, status) == 0
    if grad_bf16:
        Gb = to_bf16_bits(G)
        Gd = torch.from_numpy(Gb.view(np.int16)).to(DEV).view(torch.bfloat16)
        assert pk.embbag_backward_apply_sgd_split_bf16_act(Gd, B, NS, cfg.lr, hi, lo, ws) == 0
    else:
        Gd = torch.from_numpy(G).to(DEV)
        assert pk.embbag_backward_apply_sgd_split_bf16(Gd, B, NS, cfg.lr, hi, lo, ws) == 0
    assert pk.embbag_status_read(status) == 0
    Y = Y.cpu().numpy()
    Yb = bf16_bits(Yb)
    got = []
    for t in range(T):
        rd = torch.from_numpy(sel[t]).to(DEV)
        got.append((hi[t][rd].cpu().numpy().view(np.uint16), lo[t][rd].cpu().numpy().view(np.uint16)))
    del hi, lo
    torch.cuda.empty_cache()

    log(f"[full] {name}: oracle forward ({NS} look-ups)")
    rc, Y_ref = oracle.forward_split(hi_c, B, I_c, O)
    assert rc == 0
    assert_close(Y, Y_ref, f"{name} pooled")
    assert bits_equal(Y, Y_ref), f"{name}: pooled outputs not bit-identical"
    ndiff = assert_bf16_bracket(Yb, Y_ref, f"{name} pooled bf16")
    log(f"[full] {name}: BF16 outputs differing from the rounded oracle value: {ndiff} of {Yb.size}")
    if P == 1:
        assert ndiff == 0
    log(f"[full] {name}: oracle backward")
    h_ref, l_ref = [h.copy() for h in hi_c], [l.copy() for l in lo_c]
    if grad_bf16:
        assert oracle.backward_sgd_split_bf16_act(Gb, B, I_c, O, cfg.lr, h_ref, l_ref) == 0
    else:
        assert oracle.backward_sgd_split(G, B, I_c, O, cfg.lr, h_ref, l_ref) == 0
    for t in range(T):
        is_u = np.isin(sel[t], untouched[t])
        w_gpu = oracle.combine(*got[t])
        w_ref = oracle.combine(h_ref[t], l_ref[t])
        assert_close(w_gpu[~is_u], w_ref[~is_u], f"{name} table {t} touched rows")
        assert bits_equal(got[t][0][is_u], hi_c[t][is_u]), f"{name} table {t} untouched hi changed"
        assert bits_equal(got[t][1][is_u], lo_c[t][is_u]), f"{name} table {t} untouched lo changed"
    log(f"[full] {name}: ok")


def _run_pooled(name, pooling):
    """Weighted-sum or mean pooling (f1) at full size, as bench.py --pooling runs it."""
    cfg = get_config(name)
    T, B, E, P, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.pooling, cfg.num_indices
    log(f"[full] {name} {pooling}: filling {cfg.table_bytes / 1e9:.1f} GB on the device")
    W = [torch.empty((m, E), dtype=torch.float32, device=DEV) for m in cfg.rows]
    fill_tables_torch(cfg, W)
    I, O = make_batch(cfg, 0, device=DEV)
    G = make_grads(cfg, 0)
    a = make_weights(cfg, 0) if pooling == "weighted" else None
    pool = pk.EMBBAG_POOL_MEAN if pooling == "mean" else pk.EMBBAG_POOL_SUM
    om = oracle.POOL_MEAN if pooling == "mean" else oracle.POOL_SUM
    rng = np.random.default_rng(9)
    sel, I_c, untouched = [], np.empty_like(I), []
    for t in range(T):
        lo, hi = t * B * P, (t + 1) * B * P
        touched = np.unique(I[lo:hi])
        cand = rng.integers(0, cfg.rows[t], 2000)
        cand = np.setdiff1d(np.unique(cand), touched)[: max(1, 10000 // T)]
        rows = np.union1d(touched, cand)
        I_c[lo:hi] = np.searchsorted(rows, I[lo:hi])
        sel.append(rows)
        untouched.append(cand)
    W_c = [table_rows_torch(cfg.seed, t, torch.from_numpy(sel[t]).to(DEV), E,
                            cfg.value_scale[t]).cpu().numpy() for t in range(T)]
    log(f"[full] {name} {pooling}: GPU forward + backward")
    Id, Od, Gd = (torch.from_numpy(x).to(DEV) for x in (I, O, G))
    ad = None if a is None else torch.from_numpy(a).to(DEV)
    Y = torch.empty((T, B, E), dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(T, B, NS, E), dtype=torch.uint8, device=DEV)
    assert pk.embbag_forward_pooled(W, B, Id, Od, Y, ad, pool, status) == 0
    assert pk.embbag_backward_prepare_pooled(cfg.rows, E, B, Id, Od, ws, ad, pool, status) == 0
    assert pk.embbag_backward_apply_sgd_pooled(Gd, B, Od, NS, cfg.lr, W, ws, ad, pool) == 0
    assert pk.embbag_status_read(status) == 0
    Y = Y.cpu().numpy()
    W_gpu = [W[t][torch.from_numpy(sel[t]).to(DEV)].cpu().numpy() for t in range(T)]
    del W
    torch.cuda.empty_cache()
    log(f"[full] {name} {pooling}: oracle")
    rc, Y_ref = oracle.forward_weighted(W_c, B, I_c, O, a, om)
    assert rc == 0
    assert_close(Y, Y_ref, f"{name} {pooling} pooled")
    assert bits_equal(Y, Y_ref), f"{name} {pooling}: pooled outputs not bit-identical"
    W_ref = [w.copy() for w in W_c]
    assert oracle.backward_sgd_weighted(G, B, I_c, O, cfg.lr, W_ref, a, om) == 0
    for t in range(T):
        is_u = np.isin(sel[t], untouched[t])
        assert_close(W_gpu[t][~is_u], W_ref[t][~is_u], f"{name} {pooling} table {t} touched rows")
        assert bits_equal(W_gpu[t][is_u], W_c[t][is_u]), f"{name} table {t} untouched rows changed"
    log(f"[full] {name} {pooling}: ok")


def test_large_weighted_full_size():
    _run_pooled("large", "weighted")


def test_large_mean_full_size():
    _run_pooled("large", "mean")


def test_large_full_size():
    _run("large")


def test_mlperf_full_size():
    _run("mlperf")


def test_large_split_full_size():
    _run_split("large_split", grad_bf16=False)


def test_mlperf_split_full_size():
    _run_split("mlperf_split", grad_bf16=True)


def test_maximum_lookup_count():
    """The most look-ups one call accepts, 2^31 - 1 (indices and offsets are
    int32), through the forward and the fused backward: every kernel's
    position arithmetic at its limit, where the last radix tile, reduce chunk
    and index window run past 2^31 - 1.  One table of 1024 rows, E = 4, bags of 2048 look-ups (the last one
    2047) with row s mod 1024, so every full bag reads each row twice.  Weights
    are small integers and gradients binary fractions, so every expected value
    has a closed form that is exact in FP32: each pooled output and every
    updated row must match bit for bit, and no pooled row may stay unwritten."""
    NS = 2 ** 31 - 1
    P, M, E, lr = 2048, 1024, 4, 0.5
    B = (NS + P - 1) // P
    log(f"[full] maximum look-up count: NS={NS}, B={B}, M={M}, E={E}")
    Wh = ((np.arange(M)[:, None] * 7 + np.arange(E)[None, :] * 3) % 17 - 8).astype(np.float32)
    W = torch.from_numpy(Wh).to(DEV)
    I = torch.arange(NS, dtype=torch.int32, device=DEV).bitwise_and_(M - 1)
    O = torch.clamp(torch.arange(B + 1, dtype=torch.int64, device=DEV) * P, max=NS).to(torch.int32)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    Y = torch.full((1, B, E), float("nan"), dtype=torch.float32, device=DEV)
    pk.check(pk.embbag_forward([W], B, I, O, Y, status), "forward")
    pk.check(pk.embbag_status_read(status), "forward status")
    full = 2.0 * Wh.astype(np.float64).sum(0)
    Yexp = np.broadcast_to(full, (B, E)).copy()
    Yexp[B - 1] -= Wh[M - 1]  # the last bag misses row 1023's second read
    Yg = Y.cpu().numpy().reshape(B, E)
    assert bits_equal(Yg, Yexp.astype(np.float32)), "pooled outputs"

    k = np.arange(B, dtype=np.float64)
    dY = (((k % 5) - 2) * 2.0 ** -6)[:, None] + np.arange(E)[None, :] * 2.0 ** -8
    dYd = torch.from_numpy(dY.astype(np.float32)).reshape(1, B, E).to(DEV)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(1, B, NS, E), dtype=torch.uint8,
                     device=DEV)
    pk.check(pk.embbag_backward_sgd(dYd, B, I, O, lr, [W], ws, status), "backward_sgd")
    pk.check(pk.embbag_status_read(status), "backward status")
    mult = np.full(M, 2.0)
    mult[M - 1] = 1.0  # row 1023 is read once by the last bag
    G = 2.0 * dY[:B - 1].sum(0)[None, :] + mult[:, None] * dY[B - 1][None, :]
    Wexp = (Wh.astype(np.float64) - lr * G).astype(np.float32)
    assert bits_equal(W.cpu().numpy(), Wexp), "updated rows"
    del I, O, Y, ws
    torch.cuda.empty_cache()


def test_maximum_lookups_and_bags_together():
    """Both limits in one call: 2^31 - 1 look-ups and T*B + 1 = 2^31 - 1
    offsets (2 tables of 2^30 - 1 bags, one look-up per bag, the last bag
    two).  This is where the key build's validation slices pass 2^31 offsets.
    Look-up s of table t reads row (s - t*B) mod 768; B and 768 are multiples
    of 3, so gradients that depend on the bag index mod 3 give each row a sum
    with a closed form (the last bag's second look-up is added on its own).  Weights are small integers and gradients
    binary fractions: every pooled output (compared on the device, slice by
    slice) and every updated row must match bit for bit.  About 140 GB of
    device memory."""
    T, B, M, E, lr = 2, 2 ** 30 - 1, 768, 4, 0.5
    NS, TB = 2 ** 31 - 1, 2 * (2 ** 30 - 1)
    log(f"[full] maximum look-ups and bags: NS={NS}, T*B+1={TB + 1}, M={M}, E={E}")
    rng = np.random.default_rng(31)
    Wh = rng.integers(-8, 9, (T, M, E)).astype(np.float32)
    W = [torch.from_numpy(Wh[t]).to(DEV) for t in range(T)]
    I = torch.arange(NS, dtype=torch.int32, device=DEV)
    I[B:] -= B
    I.remainder_(M)
    O = torch.arange(TB + 1, dtype=torch.int32, device=DEV)
    O[TB] = NS  # the last bag holds look-ups TB - 1 and TB
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    Y = torch.full((T, B, E), float("nan"), dtype=torch.float32, device=DEV)
    pk.check(pk.embbag_forward(W, B, I, O, Y, status), "forward")
    pk.check(pk.embbag_status_read(status), "forward status")
    Wd = torch.from_numpy(Wh).to(DEV)
    Yf = Y.view(TB, E)
    step = 1 << 26
    for lo in range(0, TB, step):
        k = torch.arange(lo, min(lo + step, TB), dtype=torch.int64, device=DEV)
        t = torch.div(k, B, rounding_mode="floor")
        exp = Wd[t, (k - t * B) % M]
        exp[k == TB - 1] += Wd[1, B % M]
        got = Yf[lo:lo + k.numel()]
        assert torch.equal(got.view(torch.int32), exp.view(torch.int32)), f"pooled outputs in [{lo}, +{k.numel()})"
    del Y, Yf

    dY = torch.empty((T, B, E), dtype=torch.float32, device=DEV)
    dYf = dY.view(TB, E)
    col = torch.arange(E, dtype=torch.float32, device=DEV) * 2.0 ** -6
    for lo in range(0, TB, step):
        k = torch.arange(lo, min(lo + step, TB), dtype=torch.int64, device=DEV)
        dYf[lo:lo + k.numel()] = (((k % 3) - 1).to(torch.float32) * 2.0 ** -4)[:, None] + col[None, :]
    ws = torch.empty(pk.embbag_backward_workspace_bytes(T, B, NS, E), dtype=torch.uint8,
                     device=DEV)
    pk.check(pk.embbag_backward_sgd(dY, B, I, O, lr, W, ws, status), "backward_sgd")
    pk.check(pk.embbag_status_read(status), "backward status")
    r = np.arange(M)
    for t in range(T):
        # the first B look-ups of each table: look-up s' in bag t*B + s',
        # row s' mod M, and bag and row agree mod 3
        cnt = np.where(r < B, (B - r + M - 1) // M, 0).astype(np.float64)
        G = cnt[:, None] * ((((r % 3) - 1) * 2.0 ** -4)[:, None] + np.arange(E)[None, :] * 2.0 ** -6)
        if t == T - 1:  # look-up TB (local B) in bag TB - 1: row B mod M
            G[B % M] += (((TB - 1) % 3) - 1) * 2.0 ** -4 + np.arange(E) * 2.0 ** -6
        Wexp = (Wh[t].astype(np.float64) - lr * G).astype(np.float32)
        assert bits_equal(W[t].cpu().numpy(), Wexp), f"updated rows of table {t}"
    del I, O, dY, dYf, ws
    torch.cuda.empty_cache()
