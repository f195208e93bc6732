"""Workload shapes for the EmbeddingBag step.

The shapes follow the paper's Table 1 (Small, Large, MLPerf columns): number
of tables S, rows per table M, embedding dimension E, look-ups per bag P.
The graded single-GPU variants differ from the paper where noted:

* ``small``  : 8 tables x 1e6 rows x E=64, batch 2048, P=32, Zipf(1.05).
               (The paper's Small uses P=50 with uniform indices; that shape
               is kept as ``small_p50_uniform``.)
* ``large``  : 16 of the paper's 64 tables (one device's share when the 64
               tables are spread over four devices, as in Table 2's minimum
               of 4 sockets), 6e6 rows x E=256, batch 8192, P=100, Zipf(1.05).
* ``mlperf`` : 26 tables, E=128, rows log-uniform in [10, 4e7] conditioned so
               that all tables together take ~98 GB (Table 2), batch 65536,
               P=1, Zipf(1.2).
* ``split``  : ``small`` stored as Split-SGD-BF16 halves (Section VII);
  ``large_split`` and ``mlperf_split`` are the same storage at those shapes.
* ``tiny``   : 4 x 1000 x 16, batch 32, P=4, uniform; values U(-0.01, 0.01).

Table values are U(-a_t, a_t) with a_t = 1/sqrt(M_t) (0.01 for ``tiny``);
gradients of the pooled output are N(0, 1); the SGD learning rate is 0.1.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

BASE_SEED = 20050468


@dataclass(frozen=True)
class Config:
    name: str
    rows: tuple            # M_t per table
    dim: int               # E
    batch: int             # B (bags per table)
    pooling: int           # P (look-ups per bag, fixed)
    dist: str              # "uniform" | "zipf"
    zipf_s: float          # Zipf exponent (ignored for uniform)
    value_scale: tuple     # a_t: table values are U(-a_t, a_t)
    lr: float = 0.1
    seed: int = BASE_SEED
    split: bool = False    # Split-SGD-BF16 storage
    mapping: str = "affine"  # Zipf rank -> row: "affine" bijection or "identity"

    @property
    def num_tables(self) -> int:
        return len(self.rows)

    @property
    def num_bags(self) -> int:
        return self.num_tables * self.batch

    @property
    def num_indices(self) -> int:
        return self.num_bags * self.pooling

    @property
    def total_rows(self) -> int:
        return int(sum(self.rows))

    @property
    def table_bytes(self) -> int:
        per = 4  # FP32, or BF16 hi + 16-bit lo
        return self.total_rows * self.dim * per

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


def _uniform_scale(rows):
    return tuple(float(1.0 / math.sqrt(m)) for m in rows)


def _make(name: str, seed: int) -> Config:
    if name == "tiny":
        rows = (1000,) * 4
        return Config("tiny", rows, 16, 32, 4, "uniform", 0.0, (0.01,) * 4, seed=seed)
    if name == "small":
        rows = (1_000_000,) * 8
        return Config("small", rows, 64, 2048, 32, "zipf", 1.05, _uniform_scale(rows), seed=seed)
    if name == "split":
        return _make("small", seed).with_(name="split", split=True)
    if name == "large":
        rows = (6_000_000,) * 16
        return Config("large", rows, 256, 8192, 100, "zipf", 1.05, _uniform_scale(rows), seed=seed)
    if name == "mlperf":
        from .generators import mlperf_rows
        rows, _attempt = mlperf_rows(seed)
        rows = tuple(int(r) for r in rows)
        return Config("mlperf", rows, 128, 65536, 1, "zipf", 1.2, _uniform_scale(rows), seed=seed)
    if name == "large_split":
        return _make("large", seed).with_(name=name, split=True)
    if name == "mlperf_split":
        return _make("mlperf", seed).with_(name=name, split=True)
    if name == "small_p50_uniform":
        rows = (1_000_000,) * 8
        return Config(name, rows, 64, 2048, 50, "uniform", 0.0, _uniform_scale(rows), seed=seed)
    if name == "large_uniform":
        return _make("large", seed).with_(name=name, dist="uniform", zipf_s=0.0)
    raise KeyError(f"unknown config {name!r}; known: {CONFIG_NAMES}")


CONFIG_NAMES = ("tiny", "small", "large", "mlperf", "split", "large_split", "mlperf_split",
                "small_p50_uniform", "large_uniform")

_CACHE: dict = {}


def get_config(name: str, seed: int = BASE_SEED) -> Config:
    key = (name, seed)
    if key not in _CACHE:
        _CACHE[key] = _make(name, seed)
    return _CACHE[key]


def scaled(cfg: Config, *, batch: int | None = None, rows: int | None = None,
           tables: int | None = None, name: str | None = None) -> Config:
    """A smaller variant of ``cfg`` with the same distribution and dim.

    ``rows`` caps every table's row count (value scale follows 1/sqrt(M_t)
    unless the config uses a fixed scale); ``tables`` keeps the first tables.
    """
    r = list(cfg.rows)
    if tables is not None:
        r = r[:tables]
    if rows is not None:
        r = [min(m, rows) for m in r]
    if cfg.name.startswith("tiny"):
        scale = (0.01,) * len(r)
    else:
        scale = _uniform_scale(r)
    return cfg.with_(name=name or f"{cfg.name}_scaled", rows=tuple(r),
                     value_scale=scale, batch=batch or cfg.batch)
