"""Seeded input generators: determinism, published definitions, distributions."""
import math

import numpy as np
import pytest
import torch
from scipy import stats

from embbag_data import (get_config, make_batch, make_grads, mlperf_rows, row_bijection,
                         scaled, splitmix64_np, table_values_np, table_values_torch, zipf_cdf)
from embbag_data.generators import draw_rows


def test_splitmix64_published_values():
    # First outputs of SplitMix64 seeded with 1234567 (reference values of the
    # algorithm as published by Steele, Lea and Flood, 2014; they are the
    # standard test vector of the Java SplittableRandom / xoshiro seeding code).
    out = splitmix64_np(1234567, np.arange(5, dtype=np.uint64))
    assert out.tolist() == [6457827717110365317, 3203168211198807973, 9817491932198370423,
                            4593380528125082431, 16408922859458223821]


def test_table_values_host_and_torch_agree():
    cfg = get_config("small")
    for t in (0, 5):
        a = table_values_np(cfg.seed, t, np.arange(1000, 1300), cfg.dim, cfg.value_scale[t])
        b = table_values_torch(cfg.seed, t, 1000, 300, cfg.dim, cfg.value_scale[t]).numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_table_values_range_and_moments():
    cfg = get_config("tiny")
    w = table_values_np(cfg.seed, 1, np.arange(cfg.rows[1]), cfg.dim, cfg.value_scale[1])
    assert w.dtype == np.float32 and w.shape == (1000, 16)
    assert np.all(np.abs(w) < 0.01)
    assert abs(w.mean()) < 3 * 0.01 / math.sqrt(3 * w.size)
    assert abs(w.var() - 0.01 ** 2 / 3) < 0.05 * 0.01 ** 2 / 3
    # KS test against U(-0.01, 0.01)
    assert stats.kstest(w.ravel(), stats.uniform(loc=-0.01, scale=0.02).cdf).pvalue > 1e-4


def test_batches_deterministic_and_shaped():
    cfg = get_config("tiny")
    I1, O1 = make_batch(cfg, 3)
    I2, O2 = make_batch(cfg, 3)
    I3, _ = make_batch(cfg, 4)
    assert np.array_equal(I1, I2) and np.array_equal(O1, O2)
    assert not np.array_equal(I1, I3)
    assert I1.dtype == np.int32 and O1.dtype == np.int32
    assert I1.size == cfg.num_indices and O1.size == cfg.num_bags + 1
    assert np.array_equal(O1, np.arange(0, cfg.num_indices + 1, cfg.pooling))
    for t in range(cfg.num_tables):
        part = I1[t * cfg.batch * cfg.pooling:(t + 1) * cfg.batch * cfg.pooling]
        assert part.min() >= 0 and part.max() < cfg.rows[t]
    G = make_grads(cfg, 3)
    assert G.shape == (4, 32, 16) and G.dtype == np.float32
    assert np.array_equal(G, make_grads(cfg, 3))


def test_zipf_sampler_chi_square():
    cfg = scaled(get_config("small"), rows=50, tables=1).with_(mapping="identity")
    n = 200000
    ranks = draw_rows(cfg, 0, n, 0)
    p = np.arange(1, 51, dtype=np.float64) ** -1.05
    p /= p.sum()
    obs = np.bincount(ranks, minlength=50)
    assert stats.chisquare(obs, n * p).pvalue > 1e-4


def test_zipf_cdf_and_torch_search_agree():
    c = zipf_cdf(1000, 1.2)
    assert c[-1] == 1.0 and np.all(np.diff(c) > 0)
    u = np.random.default_rng(0).random(10000)
    a = np.searchsorted(c, u, side="right")
    b = torch.searchsorted(torch.from_numpy(c), torch.from_numpy(u), right=True).numpy()
    assert np.array_equal(a, b)


def test_row_bijection_is_a_permutation():
    rng = np.random.default_rng(1)
    for m in (1, 2, 10, 97, 1000, 6 * 1024):
        a, c = row_bijection(m, rng)
        r = (a * np.arange(m) + c) % m
        assert np.array_equal(np.sort(r), np.arange(m))


def test_mlperf_rows_condition():
    rows, attempt = mlperf_rows(20050468)
    assert rows.size == 26 and rows.min() >= 10 and rows.max() <= 4e7
    total = rows.sum() * 128 * 4
    assert abs(total - 98e9) <= 0.1 * 98e9
    rows2, attempt2 = mlperf_rows(20050468)
    assert np.array_equal(rows, rows2) and attempt == attempt2
    cfg = get_config("mlperf")
    assert cfg.rows == tuple(int(r) for r in rows)
    assert cfg.total_rows < 2 ** 31 - 1


@pytest.mark.parametrize("name", ["tiny", "small", "large", "mlperf", "split"])
def test_config_shapes(name):
    cfg = get_config(name)
    expect = {"tiny": (4, 16, 32, 4), "small": (8, 64, 2048, 32), "large": (16, 256, 8192, 100),
              "mlperf": (26, 128, 65536, 1), "split": (8, 64, 2048, 32)}[name]
    assert (cfg.num_tables, cfg.dim, cfg.batch, cfg.pooling) == expect
    assert cfg.num_indices < 2 ** 31 and cfg.num_bags < 2 ** 31
