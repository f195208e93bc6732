"""bench.py's command-line contract that needs no GPU: a run on more than one
GPU is refused with a JSON message and exit status 2, before any GPU work;
the byte models it reports have the sizes the workloads fix."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv],
                       capture_output=True, text=True, env={**os.environ, **env}, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_bytes_model_of_the_large_step():
    """B_alg per step at Large: every look-up's 1 KB row read once in the
    forward, the pooled outputs written, the indices and offsets read; the
    update reads dY once and reads and writes every touched row once."""
    sys.path.insert(0, ROOT)
    import bench
    from embbag_data import get_config
    cfg = get_config("large")
    T, B, E, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.num_indices
    U = 3_276_528
    fwd, bwd = bench.bytes_model(cfg, U, split=False)
    assert (T, B, E, NS) == (16, 8192, 256, 13_107_200)
    # rows read, indices, offsets, pooled outputs
    assert fwd == 13_421_772_800 + 52_428_800 + 524_292 + 134_217_728
    # dY, indices, offsets, touched rows read and written
    assert bwd == 134_217_728 + 52_428_800 + 524_292 + 2 * U * 1024
    # split rows: the forward reads 2-byte high halves; the update moves both halves
    fwd_s, bwd_s = bench.bytes_model(cfg, U, split=True)
    assert fwd_s == fwd - NS * E * 2 and bwd_s == bwd
