"""Write tests/golden/tiny_oracle.json from the CPU oracle alone.

The fixture records what the oracle computes for the Tiny workload (4 tables
x 1000 rows x E=16, batch 32, P=4, uniform indices, values U(-0.01, 0.01),
lr 0.1, N(0,1) pooled gradients, seed 20050468, batch 0).  The paper prints
no worked example for these operators, so this file is not a pin of the
oracle; it detects any later change to the oracle's arithmetic, which must
then be justified by the passage of the paper it follows.

Run: python tests/golden/make_golden.py
"""
import hashlib
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from embbag_data import get_config, make_batch, make_grads, table_values_np  # noqa: E402


def compute():
    cfg = get_config("tiny")
    W = [table_values_np(cfg.seed, t, np.arange(cfg.rows[t]), cfg.dim, cfg.value_scale[t])
         for t in range(cfg.num_tables)]
    I, O = make_batch(cfg, 0)
    G = make_grads(cfg, 0)
    rc, Y = oracle.forward(W, cfg.batch, I, O)
    assert rc == 0
    rc, d = oracle.dedup(cfg.rows, cfg.batch, I, O)
    assert rc == 0
    W1 = [w.copy() for w in W]
    assert oracle.backward_sgd(G, cfg.batch, I, O, cfg.lr, W1) == 0
    h = lambda a: hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
    return {
        "workload": "tiny, batch 0, seed 20050468",
        "num_unique": d["num_unique"],
        "sha256_pooled": h(Y),
        "sha256_sorted_keys": h(d["sorted_keys"]),
        "sha256_sorted_bags": h(d["sorted_bags"]),
        "sha256_tables_after": h(np.concatenate([w.ravel() for w in W1])),
        "pooled_bag0": [float(x) for x in Y[0, 0]],
        "table0_row_of_first_lookup_after": [float(x) for x in W1[0][I[0]]],
    }


if __name__ == "__main__":
    out = os.path.join(HERE, "tiny_oracle.json")
    with open(out, "w") as f:
        json.dump(compute(), f, indent=1)
    print(out)
