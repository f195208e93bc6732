"""Seeded generators: table values, bag layouts, gradients.

Table values use a counter-based generator so that any single row can be
regenerated on its own (on the host, for the CPU checker of a 98 GB table)
or filled in parallel on the device, with identical bits:

    value(t, r, e) = a_t * v,   v = (2k + 1 - 2^24) / 2^24,   k = h >> 40
    h = SplitMix64 output number i of the stream seeded with ``tseed``,
        i = (t << 41) | (r << 10) | e

SplitMix64 is the generator of Steele, Lea and Flood, "Fast splittable
pseudorandom number generators" (OOPSLA 2014): output i of a stream with seed
x is mix(x + (i + 1) * 0x9E3779B97F4A7C15) with the 64-bit finaliser below.
v is an odd multiple of 2^-24 in (-1, 1) and exact in FP32; the product with
a_t (an FP32 number) is rounded once, so host and device agree bit for bit.

Zipf look-ups are drawn by inverting the truncated Zipf(s) CDF over ranks
1..M (a float64 cumulative table and a binary search), then mapped to rows by
a seeded affine bijection row = (a * (rank - 1) + c) mod M, gcd(a, M) = 1, so
the hot rows are spread over the table instead of sitting at its start.
"""
from __future__ import annotations

import math

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
_M64 = (1 << 64) - 1


def _signed(x: int) -> int:
    x &= _M64
    return x - (1 << 64) if x >= (1 << 63) else x


# --------------------------------------------------------------------------
# SplitMix64, numpy (uint64 arithmetic wraps modulo 2^64 by definition)
# --------------------------------------------------------------------------
def splitmix64_np(seed: int, i: np.ndarray) -> np.ndarray:
    """Output number ``i`` (uint64 array) of the SplitMix64 stream ``seed``."""
    i = np.asarray(i, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & _M64) + (i + np.uint64(1)) * np.uint64(GAMMA)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX2)
        z = z ^ (z >> np.uint64(31))
    return z


def table_seed(seed: int) -> int:
    ss = np.random.SeedSequence([seed, 0x7AB1E])
    return int(ss.generate_state(1, dtype=np.uint64)[0])


def _counter_np(t: int, rows: np.ndarray, dim: int) -> np.ndarray:
    rows = np.asarray(rows, dtype=np.uint64)
    e = np.arange(dim, dtype=np.uint64)
    return (np.uint64(t) << np.uint64(41)) | (rows[:, None] << np.uint64(10)) | e[None, :]


def table_values_np(seed: int, t: int, rows, dim: int, scale: float) -> np.ndarray:
    """FP32 values of rows ``rows`` of table ``t``: shape [len(rows), dim]."""
    h = splitmix64_np(table_seed(seed), _counter_np(t, rows, dim))
    k = (h >> np.uint64(40)).astype(np.int64)
    v = (2 * k + 1 - (1 << 24)).astype(np.float32) * np.float32(2.0 ** -24)
    return v * np.float32(scale)


# --------------------------------------------------------------------------
# SplitMix64, torch int64 (two's-complement wrap-around), for device fills
# --------------------------------------------------------------------------
def _mix_torch(z):
    import torch  # noqa: F401
    z = (z ^ ((z >> 30) & ((1 << 34) - 1))) * _signed(MIX1)
    z = (z ^ ((z >> 27) & ((1 << 37) - 1))) * _signed(MIX2)
    return z ^ ((z >> 31) & ((1 << 33) - 1))


def table_values_torch(seed: int, t: int, row_start: int, nrows: int, dim: int,
                       scale: float, device="cpu"):
    """Same values as :func:`table_values_np` for rows [row_start, row_start+nrows)."""
    import torch
    r = torch.arange(row_start, row_start + nrows, dtype=torch.int64, device=device)
    e = torch.arange(dim, dtype=torch.int64, device=device)
    i = ((t << 41) | (r[:, None] << 10)) | e[None, :]
    del r
    z = (i + 1) * _signed(GAMMA) + _signed(table_seed(seed))
    del i
    h = _mix_torch(z)
    del z
    k = (h >> 40) & ((1 << 24) - 1)
    del h
    v = (2 * k + 1 - (1 << 24)).to(torch.float32) * (2.0 ** -24)
    return v * float(np.float32(scale))


def table_rows_torch(seed: int, t: int, rows, dim: int, scale: float):
    """Same values as :func:`table_values_np` for arbitrary rows (torch, any device)."""
    import torch
    r = torch.as_tensor(rows, dtype=torch.int64)
    e = torch.arange(dim, dtype=torch.int64, device=r.device)
    i = ((t << 41) | (r[:, None] << 10)) | e[None, :]
    z = (i + 1) * _signed(GAMMA) + _signed(table_seed(seed))
    del i
    h = _mix_torch(z)
    del z
    k = (h >> 40) & ((1 << 24) - 1)
    del h
    v = (2 * k + 1 - (1 << 24)).to(torch.float32) * (2.0 ** -24)
    return v * float(np.float32(scale))


def fill_table_torch(cfg, t: int, w, chunk_elems: int = 1 << 26):
    """Fill a preallocated [M_t, E] FP32 tensor with table t's values (any device)."""
    m, e = w.shape
    step = max(1, chunk_elems // e)
    for r0 in range(0, m, step):
        n = min(step, m - r0)
        w[r0:r0 + n].copy_(table_values_torch(cfg.seed, t, r0, n, e, cfg.value_scale[t],
                                              device=w.device))


def fill_tables_torch(cfg, tables, chunk_elems: int = 1 << 26):
    """Fill preallocated [M_t, E] FP32 tensors in place (any device)."""
    for t, w in enumerate(tables):
        fill_table_torch(cfg, t, w, chunk_elems)


# --------------------------------------------------------------------------
# Look-up indices
# --------------------------------------------------------------------------
_CDF_CACHE: dict = {}


def zipf_cdf(m: int, s: float) -> np.ndarray:
    """Cumulative distribution of the truncated Zipf(s) over ranks 1..m."""
    key = (int(m), float(s))
    c = _CDF_CACHE.get(key)
    if c is None:
        k = np.arange(1, m + 1, dtype=np.float64)
        c = np.cumsum(k ** (-s))
        c /= c[-1]
        if len(_CDF_CACHE) > 4:
            _CDF_CACHE.clear()
        _CDF_CACHE[key] = c
    return c


def row_bijection(m: int, rng: np.random.Generator):
    """Seeded affine bijection on [0, m): returns (a, c) with gcd(a, m) == 1."""
    if m == 1:
        return 1, 0
    while True:
        a = int(rng.integers(1, m))
        if math.gcd(a, m) == 1:
            break
    c = int(rng.integers(0, m))
    return a, c


def _table_rng(cfg, stream: int, batch_id: int, t: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, stream, batch_id, t])))


def draw_rows(cfg, t: int, n: int, batch_id: int, device=None) -> np.ndarray:
    """n look-up rows of table t (int64 numpy array) for batch ``batch_id``."""
    m = int(cfg.rows[t])
    g = _table_rng(cfg, 1, batch_id, t)
    if cfg.dist == "uniform":
        return g.integers(0, m, n, dtype=np.int64)
    if cfg.dist != "zipf":
        raise ValueError(cfg.dist)
    u = g.random(n)
    cdf = zipf_cdf(m, cfg.zipf_s)
    if device is not None:
        import torch
        rank0 = torch.searchsorted(torch.from_numpy(cdf).to(device),
                                   torch.from_numpy(u).to(device), right=True).cpu().numpy()
    else:
        rank0 = np.searchsorted(cdf, u, side="right")
    rank0 = np.minimum(rank0, m - 1).astype(np.int64)
    if cfg.mapping == "identity":
        return rank0
    a, c = row_bijection(m, _table_rng(cfg, 4, 0, t))  # same bijection for every batch
    return (a * rank0 + c) % m


def make_batch(cfg, batch_id: int = 0, device=None):
    """Fixed-P bags: (indices int32 [T*B*P], offsets int32 [T*B+1]).

    Bag k = t*B + b holds indices[offsets[k]:offsets[k+1]], rows of table t.
    """
    n_t = cfg.batch * cfg.pooling
    parts = [draw_rows(cfg, t, n_t, batch_id, device=device) for t in range(cfg.num_tables)]
    indices = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
    offsets = np.arange(0, cfg.num_bags * cfg.pooling + 1, cfg.pooling, dtype=np.int64)
    if cfg.pooling == 0:
        offsets = np.zeros(cfg.num_bags + 1, dtype=np.int64)
    return indices, offsets.astype(np.int32)


def make_grads(cfg, batch_id: int = 0) -> np.ndarray:
    """Gradient of the pooled output, N(0,1) FP32, shape [T, B, E]."""
    out = np.empty((cfg.num_tables, cfg.batch, cfg.dim), dtype=np.float32)
    for t in range(cfg.num_tables):
        out[t] = _table_rng(cfg, 2, batch_id, t).standard_normal((cfg.batch, cfg.dim), dtype=np.float32)
    return out


def make_weights(cfg, batch_id: int = 0) -> np.ndarray:
    """Per-look-up weights a_s (Section II's non-zero entries of A), U(0.5, 1.5)
    FP32, one per look-up of make_batch's indices (table-major)."""
    n_t = cfg.batch * cfg.pooling
    out = np.empty(cfg.num_tables * n_t, dtype=np.float32)
    for t in range(cfg.num_tables):
        u = _table_rng(cfg, 3, batch_id, t).random(n_t, dtype=np.float32)
        out[t * n_t:(t + 1) * n_t] = u + np.float32(0.5)
    return out


def random_bags(rng: np.random.Generator, rows, batch: int, max_pool: int,
                empty_frac: float = 0.1, hot_frac: float = 0.0):
    """Variable-size bags for edge-case tests.

    Bag sizes are uniform in [1, max_pool], with a fraction ``empty_frac``
    forced empty; a fraction ``hot_frac`` of look-ups hit row 0 of their table
    (duplicate-heavy segments).  Returns (indices int32, offsets int32).
    """
    T = len(rows)
    sizes = rng.integers(1, max_pool + 1, size=T * batch) if max_pool > 0 else np.zeros(T * batch, np.int64)
    sizes[rng.random(T * batch) < empty_frac] = 0
    offsets = np.zeros(T * batch + 1, dtype=np.int64)
    np.cumsum(sizes, out=offsets[1:])
    idx = np.empty(int(offsets[-1]), dtype=np.int64)
    for t in range(T):
        lo, hi = offsets[t * batch], offsets[(t + 1) * batch]
        n = int(hi - lo)
        r = rng.integers(0, rows[t], n)
        if hot_frac > 0:
            r[rng.random(n) < hot_frac] = 0
        idx[lo:hi] = r
    return idx.astype(np.int32), offsets.astype(np.int32)


# --------------------------------------------------------------------------
# MLPerf-style table shapes
# --------------------------------------------------------------------------
def mlperf_rows(seed: int, num_tables: int = 26, lo: float = 10.0, hi: float = 4e7,
                dim: int = 128, target_bytes: float = 98e9, tol: float = 0.10):
    """Row counts drawn log-uniform in [lo, hi], conditioned on total FP32 bytes.

    Draws whole vectors of ``num_tables`` counts from one seeded stream and keeps
    the first whose tables take ``target_bytes`` +- ``tol`` (Table 2 of the paper
    lists 98 GB for the MLPerf tables).  Returns (rows int64 array, attempt).
    """
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 3])))
    for attempt in range(1, 1_000_000):
        x = np.exp(g.uniform(math.log(lo), math.log(hi), num_tables))
        rows = np.clip(np.floor(x), lo, hi).astype(np.int64)
        total = float(rows.sum()) * dim * 4
        if abs(total - target_bytes) <= tol * target_bytes:
            return rows, attempt
    raise RuntimeError("no draw met the size condition")
