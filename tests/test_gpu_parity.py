"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Floating point: |gpu - oracle| <= 1e-6 + 1e-5 |oracle| elementwise for pooled
outputs and updated rows; rows no look-up names must keep their bits.
Integer work (sorted keys/bags, unique keys, segment offsets, U): bit-exact.
BF16 pooled outputs: each value lies between the BF16 roundings of
oracle -/+ that tolerance (rounding is monotone), and equals the rounding of
the oracle's value wherever the sum is exact (one-term bags).
"""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
import paper_2005_04680_amd as pk
from embbag_data import get_config, make_batch, make_grads, random_bags, scaled, table_values_np
from gpu_util import (DEV, GpuTables, assert_bf16_bracket, assert_close, bf16_bits, bits_equal,
                      gpu_dedup, log, require_gpu, to_bf16_bits, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _tables(rng, rows, dim, scale):
    return [rng.uniform(-scale, scale, size=(m, dim)).astype(np.float32) for m in rows]


def check_step(W, batch, I, O, G, lr, split=False, what=""):
    """Forward + fused backward on the GPU vs the oracle; returns GPU tables."""
    log(f"[parity] {what} T={len(W)} E={W[0].shape[1]} B={batch} NS={I.size} split={split}")
    gt = GpuTables(W, split=split)
    rc, Y = gt.forward(batch, I, O)
    assert rc == 0
    if split:
        his = [oracle.split(w)[0] for w in W]
        orc, Yref = oracle.forward_split(his, batch, I, O)
    else:
        orc, Yref = oracle.forward(W, batch, I, O)
    assert orc == 0
    assert_close(Y.cpu().numpy(), Yref, f"{what} pooled")
    assert gt.backward(G, batch, I, O, lr) == 0
    assert gt.read_status() == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd(G, batch, I, O, lr, Wref) == 0
    Wg = gt.host()
    for t in range(len(W)):
        lo_, hi_ = O[t * batch], O[(t + 1) * batch]
        touched = np.zeros(W[t].shape[0], bool)
        touched[I[lo_:hi_]] = True
        assert_close(Wg[t][touched], Wref[t][touched], f"{what} table {t} touched rows")
        assert bits_equal(Wg[t][~touched], W[t][~touched]), f"{what} table {t} untouched rows changed"
    return gt


# ---------------------------------------------------------------------------
# Tiny workload (4 x 1000 x 16, B=32, P=4)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("batch_id", [0, 1])
def test_tiny(batch_id):
    cfg = get_config("tiny")
    W = [table_values_np(cfg.seed, t, np.arange(cfg.rows[t]), cfg.dim, cfg.value_scale[t])
         for t in range(cfg.num_tables)]
    I, O = make_batch(cfg, batch_id)
    G = make_grads(cfg, batch_id)
    check_step(W, cfg.batch, I, O, G, cfg.lr, what=f"tiny/{batch_id}")


# ---------------------------------------------------------------------------
# Every row geometry (lanes per row x column groups per lane), variable bags,
# empty bags, duplicate-heavy rows, ragged tails
# ---------------------------------------------------------------------------
DIMS = [4, 8, 12, 16, 20, 32, 64, 100, 128, 256, 260, 512, 768, 1024]


@pytest.mark.parametrize("dim", DIMS)
def test_row_geometries(dim):
    rng = np.random.default_rng(1000 + dim)
    rows = (300, 57, 1000)
    W = _tables(rng, rows, dim, 0.05)
    I, O = random_bags(rng, rows, 37, 20, empty_frac=0.15, hot_frac=0.2)
    G = rng.standard_normal((len(rows), 37, dim)).astype(np.float32)
    check_step(W, 37, I, O, G, 0.1, what=f"dim{dim}")


@pytest.mark.parametrize("dim", DIMS)
def test_row_geometries_split(dim):
    rng = np.random.default_rng(2000 + dim)
    rows = (500, 77)
    W = _tables(rng, rows, dim, 0.05)
    I, O = random_bags(rng, rows, 29, 12, empty_frac=0.1, hot_frac=0.3)
    G = rng.standard_normal((len(rows), 29, dim)).astype(np.float32)
    check_step(W, 29, I, O, G, 0.1, split=True, what=f"split dim{dim}")


@pytest.mark.parametrize("pool,batch,hot", [(1, 5000, 0.5), (3, 3001, 0.0), (50, 700, 0.3),
                                            (200, 64, 0.6)])
def test_many_tiles_and_long_segments(pool, batch, hot):
    """NS spans many radix tiles and segment chunks; hot rows make segments that
    cross hundreds of chunks; bag sizes and the tail are ragged."""
    rng = np.random.default_rng(pool * 7 + batch)
    rows = (20000, 3, 5000)
    dim = 64
    W = _tables(rng, rows, dim, 0.01)
    I, O = random_bags(rng, rows, batch, pool, empty_frac=0.05, hot_frac=hot)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    check_step(W, batch, I, O, G, 0.1, what=f"tiles P<={pool}")


@pytest.mark.parametrize("dim,split", [(200, False), (256, False), (256, True)])
def test_long_bags_one_row_per_wavefront(dim, split):
    """Bags of up to 300 look-ups at E = 200 and 256 (one row per wavefront,
    10 row loads in flight per lane): an iteration's last slots take their
    indices from the next 64-entry window at every offset."""
    rng = np.random.default_rng(dim + 11 + split)
    rows = (5000, 300)
    batch = 97
    W = _tables(rng, rows, dim, 0.05)
    I, O = random_bags(rng, rows, batch, 300, empty_frac=0.05, hot_frac=0.2)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    check_step(W, batch, I, O, G, 0.1, split=split, what=f"long bags E={dim} split={split}")


def test_dispatch_block_order():
    """Grids large enough that the forward (16384 blocks) and the update (4272
    blocks) walk their blocks in dispatch order rather than in per-XCD ranges:
    4 tables x 65536 bags of 0-16 look-ups (2.19M) at E = 128, where eight
    tables' rows and dY would not fit half of the MALL.  Row 0 of each table
    takes 30% of its look-ups, a segment across thousands of chunks."""
    rng = np.random.default_rng(77)
    rows, batch, dim = (200000,) * 4, 65536, 128
    I, O = random_bags(rng, rows, batch, 16, 0.02, 0.3)
    W = _tables(rng, rows, dim, 0.01)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    check_step(W, batch, I, O, G, 0.1, what="dispatch order")


@pytest.mark.parametrize("dim,seed", [(16, 1), (64, 2), (64, 3), (256, 4)])
def test_segments_of_many_lengths(dim, seed):
    """Segments of every length from 1 to tens of thousands of look-ups, in random
    bags: they start and end at every offset within chunks and within the groups
    of chunks whose partials are pre-summed, and some fill several whole groups."""
    rng = np.random.default_rng(1000 + seed)
    M = 400
    mult = np.concatenate([rng.integers(1, 40, 200), rng.integers(40, 3000, 40),
                           rng.integers(3000, 40000, 6)])
    rows_used = rng.permutation(M)[:mult.size]
    look = np.repeat(rows_used, mult).astype(np.int32)
    rng.shuffle(look)
    NS = look.size
    batch = NS // 37 + 1
    cuts = np.sort(rng.integers(0, NS + 1, batch - 1))
    O = np.concatenate([[0], cuts, [NS]]).astype(np.int32)
    W = _tables(rng, (M,), dim, 0.01)
    G = rng.standard_normal((1, batch, dim)).astype(np.float32)
    check_step(W, batch, look, O, G, 0.1, what=f"segment lengths E={dim}")


@pytest.mark.parametrize("dim", [256, 512])
def test_segment_past_one_flag_read(dim):
    """One row takes 250K of ~345K look-ups: at E >= 256 (64 lanes per row, chunks
    of 128 look-ups) its segment fills about 120 groups of 16 chunks, more than
    the 64 group flags the fix-up reads at a time, so the fix-up reads the next
    64 flags after a read that found every group filled."""
    rng = np.random.default_rng(dim + 5)
    M = 64
    mult = np.concatenate([[250000], rng.integers(1, 3000, M - 1)])
    look = np.repeat(rng.permutation(M), mult).astype(np.int32)
    rng.shuffle(look)
    NS = look.size
    batch = NS // 50 + 1
    cuts = np.sort(rng.integers(0, NS + 1, batch - 1))
    O = np.concatenate([[0], cuts, [NS]]).astype(np.int32)
    W = _tables(rng, (M,), dim, 0.01)
    G = rng.standard_normal((1, batch, dim)).astype(np.float32)
    check_step(W, batch, look, O, G, 0.1, what=f"segment past one flag read E={dim}")


# chunk length of the sorted look-ups at these sizes (64 lanes per row: 128;
# 16 lanes: 32; 4 lanes: 8)
_CHUNK = {16: 8, 64: 32, 256: 128, 512: 128, 1024: 128}


@pytest.mark.parametrize("dim,split,mode", [(16, False, "sum"), (64, False, "sum"),
                                            (256, False, "sum"), (64, True, "sum"),
                                            (256, True, "sum"), (64, False, "weighted"),
                                            (256, False, "mean"), (256, False, "weighted"),
                                            (512, False, "sum"), (1024, True, "sum")])
def test_segments_around_the_chunk_length(dim, split, mode):
    """Segments of 1-3 look-ups, of 63-65 (a 64-lane row's window past a chunk
    end) and of one, two, three and sixteen chunk lengths and one look-up
    either side, in random order.  With 64 lanes per row, a segment that ends
    within the next chunk's first 64 look-ups is summed whole by the chunk
    where it begins (the next chunk starts after it); all others crossing a
    boundary go through the partial sums.  Every kind starts at every offset
    of a chunk."""
    import paper_2005_04680_amd as pk
    c = _CHUNK[dim]
    rng = np.random.default_rng(7 * dim + split + 3 * (mode != "sum"))
    kinds = np.array([1, 2, 3, 63, 64, 65, c - 1, c, c + 1, 2 * c - 1, 2 * c, 2 * c + 1,
                      3 * c + 5, 16 * c, 16 * c + 1, 17 * c + 3])
    nseg = 600 if dim >= 256 else 1500
    mult = rng.choice(kinds, nseg, p=np.r_[[0.15] * 3, [0.1] * 3, [0.2 / 7] * 7, [0.05 / 3] * 3])
    M = nseg + 50
    look = np.repeat(np.arange(nseg), mult).astype(np.int32)
    rng.shuffle(look)
    NS = look.size
    batch = NS // 37 + 1
    cuts = np.sort(rng.integers(0, NS + 1, batch - 1))
    O = np.concatenate([[0], cuts, [NS]]).astype(np.int32)
    W = _tables(rng, (M,), dim, 0.01)
    G = rng.standard_normal((1, batch, dim)).astype(np.float32)
    what = f"segments around C={c} E={dim} split={split} {mode}"
    if mode == "sum":
        check_step(W, batch, look, O, G, 0.1, split=split, what=what)
        return
    log(f"[parity] {what} NS={NS}")
    a = rng.uniform(-2, 2, NS).astype(np.float32) if mode == "weighted" else None
    pool = pk.EMBBAG_POOL_MEAN if mode == "mean" else pk.EMBBAG_POOL_SUM
    om = oracle.POOL_MEAN if mode == "mean" else oracle.POOL_SUM
    gt = GpuTables(W)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(1, batch, NS, dim), dtype=torch.uint8,
                     device=DEV)
    ad = None if a is None else to_dev(a)
    assert pk.embbag_backward_sgd_pooled(to_dev(G), batch, to_dev(look), to_dev(O), 0.1, gt.w,
                                         ws, ad, pool, gt.status) == 0
    assert gt.read_status() == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd_weighted(G, batch, look, O, 0.1, Wref, a, om) == 0
    Wg = gt.host()[0]
    touched = np.zeros(M, bool)
    touched[look] = True
    assert_close(Wg[touched], Wref[0][touched], what)
    assert bits_equal(Wg[~touched], W[0][~touched]), f"{what}: untouched rows changed"


def test_small_full():
    """Small-shaped workload at full size: 8 x 1e6 x 64, B=2048, P=32, Zipf(1.05)."""
    cfg = get_config("small")
    W = [table_values_np(cfg.seed, t, np.arange(cfg.rows[t]), cfg.dim, cfg.value_scale[t])
         for t in range(cfg.num_tables)]
    I, O = make_batch(cfg, 0)
    G = make_grads(cfg, 0)
    check_step(W, cfg.batch, I, O, G, cfg.lr, what="small")


def test_split_full():
    """Split-SGD-BF16 workload: Small-shaped tables stored as hi/lo halves."""
    cfg = get_config("split")
    W = [table_values_np(cfg.seed, t, np.arange(cfg.rows[t]), cfg.dim, cfg.value_scale[t])
         for t in range(cfg.num_tables)]
    I, O = make_batch(cfg, 0)
    G = make_grads(cfg, 0)
    check_step(W, cfg.batch, I, O, G, cfg.lr, split=True, what="split")


@pytest.mark.parametrize("dim,maxp", [(16, 30), (64, 30), (128, 1), (256, 12), (1024, 5),
                                      (4, 20), (8, 20), (12, 20), (20, 20), (32, 20), (100, 20),
                                      (260, 12), (512, 8), (768, 8)])
def test_split_bf16_activations(dim, maxp):
    """Section VII with BF16 activations: BF16 pooled outputs from the hi halves,
    the update driven by a BF16 gradient; two-phase equals fused."""
    rng = np.random.default_rng(900 + dim)
    rows, batch = (3000, 1500, 700), 97 if maxp > 1 else 2000
    W = _tables(rng, rows, dim, 0.5)
    I, O = random_bags(rng, rows, batch, maxp, 0.1, 0.3)
    T, NS = len(rows), I.size
    log(f"[parity] split bf16 act E={dim} B={batch} NS={NS} P<={maxp}")
    gt = GpuTables(W, split=True)
    Id, Od = to_dev(I), to_dev(O)
    Yb = torch.empty((T, batch, dim), dtype=torch.bfloat16, device=DEV)
    assert pk.embbag_forward_split_bf16_act(gt.w, batch, Id, Od, Yb, gt.status) == 0
    his, los = gt.host_split()
    rc, Y32 = oracle.forward_split(his, batch, I, O)
    assert rc == 0
    got = bf16_bits(Yb)
    ndiff = assert_bf16_bracket(got, Y32, f"E={dim} pooled bf16")
    if maxp == 1:  # one-term sums are exact: every value is the rounding of the oracle's
        rc, Yref = oracle.forward_split_bf16_act(his, batch, I, O)
        assert rc == 0 and ndiff == 0 and np.array_equal(got, Yref)
    Gb = to_bf16_bits(rng.standard_normal((T, batch, dim)).astype(np.float32))
    Gd = torch.from_numpy(Gb.view(np.int16)).to(DEV).view(torch.bfloat16)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(T, batch, NS, dim), dtype=torch.uint8,
                     device=DEV)
    two = GpuTables(dev_tables=[w.clone() for w in gt.w], dev_lo=[l.clone() for l in gt.lo],
                    split=True)
    assert pk.embbag_backward_sgd_split_bf16_act(Gd, batch, Id, Od, 0.1, gt.w, gt.lo, ws,
                                                 gt.status) == 0
    assert gt.read_status() == 0
    assert pk.embbag_backward_prepare(rows, dim, batch, Id, Od, ws, two.status) == 0
    assert pk.embbag_backward_apply_sgd_split_bf16_act(Gd, batch, NS, 0.1, two.w, two.lo, ws) == 0
    assert two.read_status() == 0
    h_ref, l_ref = [h.copy() for h in his], [l.copy() for l in los]
    assert oracle.backward_sgd_split_bf16_act(Gb, batch, I, O, 0.1, h_ref, l_ref) == 0
    Wg, W2 = gt.host(), two.host()
    for t in range(T):
        Wr = oracle.combine(h_ref[t], l_ref[t])
        touched = np.zeros(rows[t], bool)
        touched[I[O[t * batch]:O[(t + 1) * batch]]] = True
        assert_close(Wg[t][touched], Wr[touched], f"E={dim} table {t} touched rows")
        assert bits_equal(Wg[t][~touched], W[t][~touched]), f"table {t} untouched rows changed"
        assert bits_equal(W2[t], Wg[t]), f"table {t}: two-phase differs from fused"


def test_split_bf16_activation_argument_errors():
    rng = np.random.default_rng(950)
    W = _tables(rng, (50,), 8, 0.5)
    I, O = random_bags(rng, (50,), 4, 3, 0.0, 0.0)
    gt = GpuTables(W, split=True)
    Id, Od = to_dev(I), to_dev(O)
    Y32 = torch.empty((1, 4, 8), dtype=torch.float32, device=DEV)
    with pytest.raises(TypeError):  # the binding checks the dtype
        pk.embbag_forward_split_bf16_act(gt.w, 4, Id, Od, Y32, gt.status)
    Yb = torch.empty((1, 4, 8), dtype=torch.bfloat16, device=DEV)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(1, 4, I.size, 8), dtype=torch.uint8,
                     device=DEV)
    # misaligned BF16 gradient (2-byte offset) and a missing lo half are argument errors
    Gflat = torch.zeros(1 * 4 * 8 + 1, dtype=torch.bfloat16, device=DEV)
    lib = pk.lib()
    s, keep = pk._tables_struct(gt.w, split_lo=gt.lo)
    rc = lib.embbag_backward_sgd_split_bf16_act(
        Gflat.data_ptr() + 2, 4, Id.data_ptr(), Od.data_ptr(), I.size, C.c_float(0.1), C.byref(s),
        ws.data_ptr(), ws.numel(), None, pk._stream(None))
    assert rc == pk.EMBBAG_ERR_INVALID_ARG
    s2, keep2 = pk._split_struct_fwd(gt.w)  # no lo halves
    rc = lib.embbag_backward_apply_sgd_split_bf16_act(Gflat.data_ptr(), 4, I.size, C.c_float(0.1),
                                                      C.byref(s2), ws.data_ptr(), ws.numel(),
                                                      pk._stream(None))
    assert rc == pk.EMBBAG_ERR_INVALID_ARG
    assert pk.embbag_forward_split_bf16_act(gt.w, 4, Id, Od, Yb, gt.status) == 0
    assert gt.read_status() == 0


# ---------------------------------------------------------------------------
# Integer work: bit-exact
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("case", ["tiny", "random", "p1_hot", "small", "mlperf_scaled",
                                  "tile1024", "tile2048", "tile4096", "one_pass", "digits7",
                                  "four_passes", "hot_17bit", "hot_24bit", "hot_2m",
                                  "empty_tables", "many_small_tables"])
def test_dedup_bit_exact(case):
    rng = np.random.default_rng(5)
    if case == "tiny":
        cfg = get_config("tiny")
        rows, batch = cfg.rows, cfg.batch
        I, O = make_batch(cfg, 0)
    elif case == "random":
        rows, batch = (1000, 5, 70000), 900
        I, O = random_bags(rng, rows, batch, 30, 0.1, 0.2)
    elif case == "p1_hot":
        rows, batch = (10, 1000000), 50000
        I, O = random_bags(rng, rows, batch, 1, 0.0, 0.4)
    elif case == "small":
        cfg = get_config("small")
        rows, batch = cfg.rows, cfg.batch
        I, O = make_batch(cfg, 1)
    elif case == "mlperf_scaled":
        cfg = scaled(get_config("mlperf"), batch=8192)
        rows, batch = cfg.rows, cfg.batch
        I, O = make_batch(cfg, 0)
    elif case.startswith("hot_"):
        # row 0 of each table takes half or more of its look-ups (runs of equal
        # digits spanning many radix tiles in every pass): 17-bit keys (two
        # passes), 24-bit keys (three passes), and 21-bit keys over 2M look-ups
        rows, batch, pool, hot = {"hot_17bit": ((100000, 31072), 3000, 20, 0.5),
                                  "hot_24bit": ((8000000, 8777215), 3000, 20, 0.5),
                                  "hot_2m": ((2 ** 20, 2 ** 20), 16000, 130, 0.6)}[case]
        I, O = random_bags(rng, rows, batch, pool, 0.05, hot)
    elif case in ("one_pass", "digits7", "four_passes"):
        # key widths the other cases miss (the dedup needs row counts only, no
        # tables): 9-bit keys sorted in one pass, 21-bit keys in three passes of
        # 7 bits, and 31-bit keys (a table of 1.6G rows) in four passes of 8 bits
        rows, batch, pool = {"one_pass": ((300, 200), 3000, 40),
                             "digits7": ((1500000, 500000), 20000, 50),
                             "four_passes": ((1600000000, 1000, 3), 5000, 60)}[case]
        I, O = random_bags(rng, rows, batch, pool, 0.05, 0.3)
    elif case == "empty_tables":
        # tables whose bags are all empty between tables whose look-ups end
        # inside a radix tile, and a table of one row
        rows, batch = (50, 7, 3000, 1, 100000, 9), 400
        I, O = random_bags(rng, rows, batch, 12, 0.1, 0.2)
        sizes = np.diff(O.astype(np.int64)).reshape(len(rows), batch)
        drop = np.isin(np.arange(len(rows)), (1, 5))
        I = I[np.repeat(np.repeat(~drop, batch), sizes.reshape(-1))]
        sizes[drop] = 0
        O = np.zeros(len(rows) * batch + 1, np.int64)
        np.cumsum(sizes.reshape(-1), out=O[1:])
        O = O.astype(np.int32)
    elif case == "many_small_tables":
        # 64 tables, most with fewer look-ups than a radix tile, so that most
        # tiles hold look-ups of several tables
        rows = tuple(int(r) for r in rng.integers(1, 300000, 64))
        batch = 37
        I, O = random_bags(rng, rows, batch, 70, 0.2, 0.25)
    else:
        # radix tiles of 1024, 2048 and 4096 keys: 12-bit keys (6-bit digits)
        # over 300K look-ups; 17-bit keys (9-bit digits) over 400K and 3M
        rows, batch, pool = {"tile1024": ((3000, 1000), 10000, 60),
                             "tile2048": ((100000, 31072), 8000, 100),
                             "tile4096": ((100000, 31072), 30000, 200)}[case]
        I, O = random_bags(rng, rows, batch, pool, 0.05, 0.3)
    log(f"[dedup] {case} NS={I.size}")
    rc, d_ref = oracle.dedup(rows, batch, I, O)
    assert rc == 0
    rc, status, d = gpu_dedup(rows, batch, I, O)
    assert rc == 0 and status == 0
    assert d["num_unique"] == d_ref["num_unique"]
    for k in ("sorted_keys", "sorted_bags", "unique_keys", "seg_off"):
        assert np.array_equal(d[k], d_ref[k]), k


# ---------------------------------------------------------------------------
# Invariants, determinism, edge cases, errors
# ---------------------------------------------------------------------------
def test_lr_zero_and_determinism():
    rng = np.random.default_rng(9)
    rows = (4000, 4000)
    W = _tables(rng, rows, 128, 0.1)
    I, O = random_bags(rng, rows, 500, 40, 0.05, 0.3)
    G = rng.standard_normal((2, 500, 128)).astype(np.float32)
    g0 = GpuTables(W)
    assert g0.backward(G, 500, I, O, 0.0) == 0
    for a, b in zip(g0.host(), W):
        assert bits_equal(a, b)
    ga, gb = GpuTables(W), GpuTables(W)
    assert ga.backward(G, 500, I, O, 0.1) == 0
    assert gb.backward(G, 500, I, O, 0.1) == 0
    for a, b in zip(ga.host(), gb.host()):
        assert bits_equal(a, b)
    _, Ya = ga.forward(500, I, O)
    _, Yb = gb.forward(500, I, O)
    assert bits_equal(Ya.cpu().numpy(), Yb.cpu().numpy())


def test_exact_special_cases():
    rng = np.random.default_rng(10)
    W = _tables(rng, (50,), 64, 1.0)
    I = np.array([7, 9, 9], np.int32)
    O = np.array([0, 1, 3, 3], np.int32)
    gt = GpuTables(W)
    rc, Y = gt.forward(3, I, O)
    Y = Y.cpu().numpy()
    assert bits_equal(Y[0, 0], W[0][7])              # single look-up = row copy
    assert np.array_equal(Y[0, 1], 2 * W[0][9])      # [r, r] = 2 W[r]
    assert bits_equal(Y[0, 2], np.zeros(64, np.float32))  # empty bag = +0.0


def test_empty_inputs():
    W = [np.ones((10, 16), np.float32)]
    gt = GpuTables(W)
    I = np.zeros(0, np.int32)
    O = np.zeros(6, np.int32)
    rc, Y = gt.forward(5, I, O)
    assert rc == 0 and bits_equal(Y.cpu().numpy(), np.zeros((1, 5, 16), np.float32))
    G = np.ones((1, 5, 16), np.float32)
    assert gt.backward(G, 5, I, O, 0.1) == 0
    assert gt.read_status() == 0
    assert bits_equal(gt.host()[0], W[0])
    # B = 0
    rc, _ = gt.forward(0, I, np.zeros(1, np.int32))
    assert rc == 0 and gt.read_status() == 0


def test_index_out_of_range_is_reported_and_writes_nothing():
    rng = np.random.default_rng(11)
    rows = (100, 20)
    W = _tables(rng, rows, 32, 0.1)
    I, O = random_bags(rng, rows, 50, 10, 0.0, 0.0)
    I[O[60] + 1] = 20           # a bag of table 1, row 20 of 20
    G = rng.standard_normal((2, 50, 32)).astype(np.float32)
    assert oracle.validate(rows, 32, 50, I, O) == oracle.ERR_INDEX_RANGE
    gt = GpuTables(W)
    rc, _ = gt.forward(50, I, O)
    assert rc == 0 and gt.read_status() == oracle.ERR_INDEX_RANGE
    gt.reset_status()
    assert gt.backward(G, 50, I, O, 0.1) == 0
    assert gt.read_status() == oracle.ERR_INDEX_RANGE
    for a, b in zip(gt.host(), W):
        assert bits_equal(a, b)
    I[5] = -3
    gt.reset_status()
    assert gt.backward(G, 50, I, O, 0.1) == 0
    assert gt.read_status() == oracle.ERR_INDEX_RANGE


@pytest.mark.parametrize("kind", ["index", "offsets"])
def test_data_errors_on_the_split_and_bf16_paths_write_nothing(kind):
    rng = np.random.default_rng(13)
    rows, E, B = (100, 20), 64, 50
    W = _tables(rng, rows, E, 0.1)
    I, O = random_bags(rng, rows, B, 10, 0.0, 0.0)
    if kind == "index":
        I[O[60] + 1] = 20       # row 20 of a 20-row table
        expect = oracle.ERR_INDEX_RANGE
    else:
        O[30] = O[31] + 1       # decreasing offsets
        expect = oracle.ERR_OFFSETS
    assert oracle.validate(rows, E, B, I, O) == expect
    gt = GpuTables(W, split=True)
    his0, los0 = gt.host_split()
    Id, Od = to_dev(I), to_dev(O)
    Gb = to_bf16_bits(rng.standard_normal((2, B, E)).astype(np.float32))
    Gd = torch.from_numpy(Gb.view(np.int16)).to(DEV).view(torch.bfloat16)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(2, B, I.size, E), dtype=torch.uint8,
                     device=DEV)
    Yb = torch.empty((2, B, E), dtype=torch.bfloat16, device=DEV)
    assert pk.embbag_forward_split_bf16_act(gt.w, B, Id, Od, Yb, gt.status) == 0
    assert gt.read_status() == expect
    gt.reset_status()
    assert pk.embbag_backward_sgd_split_bf16_act(Gd, B, Id, Od, 0.1, gt.w, gt.lo, ws,
                                                 gt.status) == 0
    assert gt.read_status() == expect
    gt.reset_status()
    assert gt.backward(make_grads_like(rng, 2, B, E), B, I, O, 0.1) == 0
    assert gt.read_status() == expect
    his, los = gt.host_split()
    for a, b, c, d in zip(his, his0, los, los0):
        assert bits_equal(a, b) and bits_equal(c, d)


def make_grads_like(rng, T, B, E):
    return rng.standard_normal((T, B, E)).astype(np.float32)


@pytest.mark.parametrize("dim", [8, 1024])
def test_sixty_four_tables(dim):
    """The largest table count the boundary accepts, tables of 1 to 5000 rows."""
    rng = np.random.default_rng(64 + dim)
    rows = tuple(int(m) for m in rng.integers(1, 5000, 64))
    rows = (1,) + rows[1:]
    batch = 40
    W = _tables(rng, rows, dim, 0.05)
    I, O = random_bags(rng, rows, batch, 12, 0.1, 0.2)
    G = rng.standard_normal((64, batch, dim)).astype(np.float32)
    check_step(W, batch, I, O, G, 0.1, what=f"64 tables E={dim}")
    check_step(W, batch, I, O, G, 0.1, split=True, what=f"64 split tables E={dim}")


@pytest.mark.parametrize("kind", ["first", "decreasing", "last", "both"])
def test_bad_offsets_are_reported_and_write_nothing(kind):
    rng = np.random.default_rng(12)
    rows = (100, 20)
    W = _tables(rng, rows, 16, 0.1)
    I, O = random_bags(rng, rows, 40, 10, 0.0, 0.0)
    G = rng.standard_normal((2, 40, 16)).astype(np.float32)
    O = O.copy()
    if kind == "first":
        O[0] = 1
    elif kind == "decreasing":
        O[30] = O[31] + 1
    elif kind == "last":
        O[-1] -= 1
    else:
        O[30] = O[31] + 1
        I[0] = 100
    assert oracle.validate(rows, 16, 40, I, O) == oracle.ERR_OFFSETS
    gt = GpuTables(W)
    rc, _ = gt.forward(40, I, O)
    assert rc == 0 and gt.read_status() == oracle.ERR_OFFSETS
    gt.reset_status()
    assert gt.backward(G, 40, I, O, 0.1) == 0
    assert gt.read_status() == oracle.ERR_OFFSETS
    for a, b in zip(gt.host(), W):
        assert bits_equal(a, b)


def test_split_helpers_bit_exact():
    import paper_2005_04680_amd as pk
    rng = np.random.default_rng(13)
    w = np.concatenate([rng.standard_normal(1 << 20).astype(np.float32),
                        rng.integers(0, 2 ** 32, 4099, dtype=np.uint64).astype(np.uint32).view(np.float32)])
    hi_ref, lo_ref = oracle.split(w)
    wd = to_dev(w)
    hi = torch.empty(w.size, dtype=torch.int16, device=DEV)
    lo = torch.empty(w.size, dtype=torch.int16, device=DEV)
    assert pk.embbag_split_fp32(wd, hi, lo) == 0
    assert np.array_equal(hi.cpu().numpy().view(np.uint16), hi_ref)
    assert np.array_equal(lo.cpu().numpy().view(np.uint16), lo_ref)
    back = torch.empty_like(wd)
    assert pk.embbag_combine_fp32(hi, lo, back) == 0
    assert bits_equal(back.cpu().numpy(), w)


# ---------------------------------------------------------------------------
# Two-phase backward (prepare = index work, apply = segment sums + SGD)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("split", [False, True])
def test_prepare_apply_equals_fused(split):
    import paper_2005_04680_amd as pk
    rng = np.random.default_rng(21)
    rows = (3000, 17, 900)
    dim = 64
    W = _tables(rng, rows, dim, 0.05)
    I, O = random_bags(rng, rows, 300, 25, 0.05, 0.3)
    G = rng.standard_normal((3, 300, dim)).astype(np.float32)
    fused = GpuTables(W, split=split)
    assert fused.backward(G, 300, I, O, 0.1) == 0
    two = GpuTables(W, split=split)
    Id, Od, Gd = to_dev(I), to_dev(O), to_dev(G)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(3, 300, I.size, dim), dtype=torch.uint8,
                     device=DEV)
    assert pk.embbag_backward_prepare(rows, dim, 300, Id, Od, ws, two.status) == 0
    if split:
        rc = pk.embbag_backward_apply_sgd_split_bf16(Gd, 300, I.size, 0.1, two.w, two.lo, ws)
    else:
        rc = pk.embbag_backward_apply_sgd(Gd, 300, I.size, 0.1, two.w, ws)
    assert rc == 0 and two.read_status() == 0
    for a, b in zip(fused.host(), two.host()):
        assert bits_equal(a, b)


@pytest.mark.parametrize("split", [False, True])
def test_prebuilt_descriptors_give_the_same_bits(split):
    """The same step through Tables / SplitTables (descriptor built once) and
    through plain lists: bit-identical outputs and tables."""
    rng = np.random.default_rng(31 + split)
    rows = (500, 40, 1200)
    W = _tables(rng, rows, 64, 0.05)
    batch = 50
    I, O = random_bags(rng, rows, batch, 12, empty_frac=0.1, hot_frac=0.3)
    G = rng.standard_normal((len(rows), batch, 64)).astype(np.float32)
    Id, Od, Gd = to_dev(I), to_dev(O), to_dev(G)
    a, b = GpuTables(W, split=split), GpuTables(W, split=split)
    desc = pk.SplitTables(b.w, b.lo) if split else pk.Tables(b.w)
    Ya = torch.empty((len(rows), batch, 64), dtype=torch.float32, device=DEV)
    Yb = torch.empty_like(Ya)
    wsa = torch.empty(pk.embbag_backward_workspace_bytes(len(rows), batch, I.size, 64),
                      dtype=torch.uint8, device=DEV)
    wsb = torch.empty_like(wsa)
    if split:
        assert pk.embbag_forward_split_bf16(a.w, batch, Id, Od, Ya, a.status) == 0
        assert pk.embbag_forward_split_bf16(desc, batch, Id, Od, Yb, b.status) == 0
        assert pk.embbag_backward_prepare(list(rows), 64, batch, Id, Od, wsa, a.status) == 0
        assert pk.embbag_backward_prepare(desc, 64, batch, Id, Od, wsb, b.status) == 0
        assert pk.embbag_backward_apply_sgd_split_bf16(Gd, batch, I.size, 0.1, a.w, a.lo, wsa) == 0
        assert pk.embbag_backward_apply_sgd_split_bf16(Gd, batch, I.size, 0.1, desc, None, wsb) == 0
    else:
        assert pk.embbag_forward(a.w, batch, Id, Od, Ya, a.status) == 0
        assert pk.embbag_forward(desc, batch, Id, Od, Yb, b.status) == 0
        assert pk.embbag_backward_prepare(list(rows), 64, batch, Id, Od, wsa, a.status) == 0
        assert pk.embbag_backward_prepare(desc, 64, batch, Id, Od, wsb, b.status) == 0
        assert pk.embbag_backward_apply_sgd(Gd, batch, I.size, 0.1, a.w, wsa) == 0
        assert pk.embbag_backward_apply_sgd(Gd, batch, I.size, 0.1, desc, wsb) == 0
    assert a.read_status() == 0 and b.read_status() == 0
    assert torch.equal(Ya, Yb)
    for x, y in zip(a.w + (a.lo or []), b.w + (b.lo or [])):
        assert torch.equal(x, y)


@pytest.mark.parametrize("dim", [8, 64, 256])
def test_split_halves_not_16_byte_aligned(dim):
    """Split halves need only 8-byte alignment (the update reads and writes
    them 8 bytes per lane and half): halves placed 8 bytes past a 16-byte
    boundary give the oracle's result, and the floor kernel leaves them
    unchanged."""
    rng = np.random.default_rng(dim + 77)
    rows = (600, 50)
    W = _tables(rng, rows, dim, 0.05)
    batch = 40
    I, O = random_bags(rng, rows, batch, 20, empty_frac=0.1, hot_frac=0.3)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    his, los = zip(*[oracle.split(w) for w in W])
    hi_d, lo_d = [], []
    for h, l in zip(his, los):
        for src, out in ((h, hi_d), (l, lo_d)):
            buf = torch.empty(src.size + 4, dtype=torch.int16, device=DEV)
            v = buf[4:].view(src.shape)  # 8 bytes past a 256-byte-aligned start
            assert v.data_ptr() % 16 == 8
            v.copy_(torch.from_numpy(src.view(np.int16)).to(DEV))
            out.append(v)
    gt = GpuTables(None, split=True, dev_tables=hi_d, dev_lo=lo_d)
    Id, Od = to_dev(I), to_dev(O)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(len(rows), batch, I.size, dim),
                     dtype=torch.uint8, device=DEV)
    assert pk.embbag_backward_prepare(list(rows), dim, batch, Id, Od, ws, gt.status) == 0
    before = [x.clone() for x in hi_d + lo_d]
    assert pk.embbag_baseline_touch_rows_split(batch, I.size, hi_d, lo_d, ws) == 0
    for a, b in zip(hi_d + lo_d, before):
        assert torch.equal(a, b)
    assert pk.embbag_backward_apply_sgd_split_bf16(to_dev(G), batch, I.size, 0.1, hi_d, lo_d,
                                                   ws) == 0
    assert gt.read_status() == 0
    hr, lr_ = [h.copy() for h in his], [l.copy() for l in los]
    assert oracle.backward_sgd_split(G, batch, I, O, 0.1, hr, lr_) == 0
    for t in range(len(rows)):
        got = oracle.combine(hi_d[t].cpu().numpy().view(np.uint16),
                             lo_d[t].cpu().numpy().view(np.uint16))
        assert_close(got, oracle.combine(hr[t], lr_[t]), f"unaligned split table {t}")


def test_apply_needs_a_prepared_workspace():
    import paper_2005_04680_amd as pk
    rng = np.random.default_rng(22)
    rows = (500, 500)
    W = _tables(rng, rows, 32, 0.05)
    I, O = random_bags(rng, rows, 100, 10, 0.0, 0.2)
    G = rng.standard_normal((2, 100, 32)).astype(np.float32)
    gt = GpuTables(W)
    Id, Od, Gd = to_dev(I), to_dev(O), to_dev(G)
    # sized for one look-up more (the prepare for other sizes below)
    ws = torch.zeros(pk.embbag_backward_workspace_bytes(2, 100, I.size + 1, 32), dtype=torch.uint8,
                     device=DEV)
    # never prepared: nothing is written
    assert pk.embbag_backward_apply_sgd(Gd, 100, I.size, 0.1, gt.w, ws) == 0
    for a, b in zip(gt.host(), W):
        assert bits_equal(a, b)
    # prepared once, applied twice: two SGD steps with the same gradient
    assert pk.embbag_backward_prepare(rows, 32, 100, Id, Od, ws, gt.status) == 0
    assert pk.embbag_backward_apply_sgd(Gd, 100, I.size, 0.1, gt.w, ws) == 0
    assert pk.embbag_backward_apply_sgd(Gd, 100, I.size, 0.1, gt.w, ws) == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd(G, 100, I, O, 0.1, Wref) == 0
    assert oracle.backward_sgd(G, 100, I, O, 0.1, Wref) == 0
    for t, (a, b) in enumerate(zip(gt.host(), Wref)):
        assert_close(a, b, f"two applies table {t}")
    # a prepare for other sizes (one look-up more, in the last bag) leaves a
    # stamp the apply rejects
    I2 = np.concatenate([I, np.array([3], np.int32)])
    O2 = O.copy()
    O2[-1] += 1
    assert pk.embbag_backward_prepare(rows, 32, 100, to_dev(I2), to_dev(O2), ws, gt.status) == 0
    before = gt.host()
    assert pk.embbag_backward_apply_sgd(Gd, 100, I.size, 0.1, gt.w, ws) == 0
    for a, b in zip(gt.host(), before):
        assert bits_equal(a, b)
    assert pk.embbag_status_read(gt.status) == 0


def test_apply_rejects_a_prepare_for_another_dim():
    """The workspace layout depends on E (the carry regions come before the
    sorted weights), so a weighted prepare for E = 32 applied to E = 64 tables
    must write nothing; prepared for E = 64 the same apply is the oracle's."""
    import paper_2005_04680_amd as pk
    rng = np.random.default_rng(23)
    rows, batch = (300, 200), 50
    W = _tables(rng, rows, 64, 0.05)
    I, O = random_bags(rng, rows, batch, 12, 0.1, 0.3)
    G = rng.standard_normal((2, batch, 64)).astype(np.float32)
    a = rng.uniform(-2, 2, I.size).astype(np.float32)
    gt = GpuTables(W)
    Id, Od, Gd, ad = to_dev(I), to_dev(O), to_dev(G), to_dev(a)
    nbytes = max(pk.embbag_backward_workspace_bytes(2, batch, I.size, e) for e in (32, 64))
    ws = torch.zeros(nbytes, dtype=torch.uint8, device=DEV)
    assert pk.embbag_backward_prepare_pooled(rows, 32, batch, Id, Od, ws, ad,
                                             pk.EMBBAG_POOL_SUM, gt.status) == 0
    assert pk.embbag_backward_apply_sgd_pooled(Gd, batch, Od, I.size, 0.1, gt.w, ws, ad,
                                               pk.EMBBAG_POOL_SUM) == 0
    for x, y in zip(gt.host(), W):
        assert bits_equal(x, y)
    assert pk.embbag_backward_prepare_pooled(rows, 64, batch, Id, Od, ws, ad,
                                             pk.EMBBAG_POOL_SUM, gt.status) == 0
    assert pk.embbag_backward_apply_sgd_pooled(Gd, batch, Od, I.size, 0.1, gt.w, ws, ad,
                                               pk.EMBBAG_POOL_SUM) == 0
    assert pk.embbag_status_read(gt.status) == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd_weighted(G, batch, I, O, 0.1, Wref, a, oracle.POOL_SUM) == 0
    for t, (x, y) in enumerate(zip(gt.host(), Wref)):
        assert_close(x, y, f"weighted apply table {t}")


# ---------------------------------------------------------------------------
# Weighted-sum and mean pooling (Section II's weights a_p)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dim", [16, 64, 128, 256, 1024])
@pytest.mark.parametrize("mode", ["weighted", "mean"])
@pytest.mark.parametrize("maxp", [3, 40, 300])
def test_weighted_and_mean(dim, mode, maxp):
    pooled_case(dim, mode, maxp)


@pytest.mark.parametrize("dim", [d for d in DIMS if d not in (16, 64, 128, 256, 1024)])
@pytest.mark.parametrize("mode", ["weighted", "mean"])
def test_weighted_and_mean_every_width(dim, mode):
    """The pooled kernels at the row widths the test above skips (every lane
    and column-group geometry of the forward and the update)."""
    pooled_case(dim, mode, 40)


def pooled_case(dim, mode, maxp):
    import paper_2005_04680_amd as pk
    rng = np.random.default_rng(dim * 3 + maxp + (mode == "mean"))
    rows = (700, 40, 3000)
    batch = 61
    W = _tables(rng, rows, dim, 0.05)
    I, O = random_bags(rng, rows, batch, maxp, empty_frac=0.1, hot_frac=0.3)
    G = rng.standard_normal((len(rows), batch, dim)).astype(np.float32)
    a = rng.uniform(-2, 2, I.size).astype(np.float32) if mode == "weighted" else None
    pool = pk.EMBBAG_POOL_MEAN if mode == "mean" else pk.EMBBAG_POOL_SUM
    om = oracle.POOL_MEAN if mode == "mean" else oracle.POOL_SUM
    log(f"[pooled] {mode} dim={dim} maxp={maxp} NS={I.size}")
    gt = GpuTables(W)
    Id, Od, Gd = to_dev(I), to_dev(O), to_dev(G)
    ad = None if a is None else to_dev(a)
    Y = torch.empty((len(rows), batch, dim), dtype=torch.float32, device=DEV)
    assert pk.embbag_forward_pooled(gt.w, batch, Id, Od, Y, ad, pool, gt.status) == 0
    rc, Yref = oracle.forward_weighted(W, batch, I, O, a, om)
    assert rc == 0
    assert_close(Y.cpu().numpy(), Yref, f"{mode} pooled")
    ws = torch.empty(pk.embbag_backward_workspace_bytes(len(rows), batch, I.size, dim),
                     dtype=torch.uint8, device=DEV)
    two = GpuTables(W)  # the same update in two phases
    assert pk.embbag_backward_sgd_pooled(Gd, batch, Id, Od, 0.1, gt.w, ws, ad, pool, gt.status) == 0
    assert gt.read_status() == 0
    ws2 = torch.empty_like(ws)
    assert pk.embbag_backward_prepare_pooled(rows, dim, batch, Id, Od, ws2, ad, pool,
                                             two.status) == 0
    assert pk.embbag_backward_apply_sgd_pooled(Gd, batch, Od, I.size, 0.1, two.w, ws2, ad,
                                               pool) == 0
    assert two.read_status() == 0
    Wref = [w.copy() for w in W]
    assert oracle.backward_sgd_weighted(G, batch, I, O, 0.1, Wref, a, om) == 0
    for t, (wg, wr, w2) in enumerate(zip(gt.host(), Wref, two.host())):
        assert_close(wg, wr, f"{mode} table {t}")
        assert bits_equal(w2, wg), f"{mode} table {t}: two-phase differs from fused"
    # a weighted workspace is not taken for an unweighted apply, nor the reverse
    if mode == "weighted":
        before = gt.host()
        assert pk.embbag_backward_apply_sgd(Gd, batch, I.size, 0.1, gt.w, ws) == 0
        assert pk.embbag_backward_apply_sgd_pooled(Gd, batch, Od, I.size, 0.1, gt.w, ws, None,
                                                   pk.EMBBAG_POOL_MEAN) == 0
        for x, y in zip(gt.host(), before):
            assert bits_equal(x, y)
        assert pk.embbag_backward_prepare(rows, dim, batch, Id, Od, ws, gt.status) == 0
        assert pk.embbag_backward_apply_sgd_pooled(Gd, batch, Od, I.size, 0.1, gt.w, ws, ad,
                                                   pool) == 0
        for x, y in zip(gt.host(), before):
            assert bits_equal(x, y)


def test_pooled_argument_errors():
    import paper_2005_04680_amd as pk
    W = [np.ones((8, 16), np.float32)]
    gt = GpuTables(W)
    I = to_dev(np.array([1, 2], np.int32))
    O = to_dev(np.array([0, 1, 2], np.int32))
    a = to_dev(np.ones(2, np.float32))
    Y = torch.empty((1, 2, 16), dtype=torch.float32, device=DEV)
    assert pk.embbag_forward_pooled(gt.w, 2, I, O, Y, a, pk.EMBBAG_POOL_MEAN) == pk.EMBBAG_ERR_INVALID_ARG
    assert pk.embbag_forward_pooled(gt.w, 2, I, O, Y, None, 7) == pk.EMBBAG_ERR_INVALID_ARG
