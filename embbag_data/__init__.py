"""Seeded synthetic inputs for the EmbeddingBag step.

This package only draws inputs: table shapes, table values, bag layouts
(indices + offsets) and pooled-output gradients.  It holds none of the
method's arithmetic (no pooling, no sorting of lookups, no update), so both
the GPU path and the CPU oracle can be fed from it without sharing any of
their computation.
"""
from .configs import BASE_SEED, Config, get_config, CONFIG_NAMES, scaled
from .generators import (
    splitmix64_np,
    table_values_np,
    table_values_torch,
    table_rows_torch,
    fill_table_torch,
    fill_tables_torch,
    make_batch,
    make_grads,
    make_weights,
    random_bags,
    zipf_cdf,
    row_bijection,
    mlperf_rows,
)

__all__ = [
    "BASE_SEED", "Config", "get_config", "CONFIG_NAMES", "scaled",
    "splitmix64_np", "table_values_np", "table_values_torch", "table_rows_torch",
    "fill_table_torch", "fill_tables_torch", "make_batch", "make_grads", "make_weights",
    "random_bags",
    "zipf_cdf", "row_bijection", "mlperf_rows",
]
