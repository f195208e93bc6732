#!/usr/bin/env python3
"""Benchmark of the EmbeddingBag training step on one MI355X.

A step is one pass of the whole hot path over one batch: the sum-pooled
forward (Algorithm 1) followed by the backward fused with the sparse SGD
update (Algorithms 2-3), on synthetic seeded data with inputs resident in
HBM.  Default workload: the Large-shaped tables (16 x 6e6 rows x E=256 FP32,
98.3 GB), batch 8192, 100 look-ups per bag, Zipf(1.05) indices, lr 0.1,
rotating over pre-generated batches.

Prints ONE JSON line: lookups/s (value), algorithmic HBM GB/s and % of the
8 TB/s peak for the whole step, the roofline record of the dominant kernel
(timed with HIP events on the launch stream), and the CPU oracle timed on a
bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "embedding lookups/sec and achieved HBM GB/s (fwd+bwd+update), % of HBM peak"


# The paper prints no EmbeddingBag throughput.  For its Small configuration
# (8 x 1M x 64, batch 2048, 50 uniform look-ups per bag, FP32) on one Xeon
# socket it gives a 38 ms optimised iteration with the embeddings at about 30%
# of it (Section VI), i.e. about 11 ms for their forward, backward and update.
# Context only: other hardware, and a derived, not a printed, number.
PAPER_CONTEXT = {
    "small_p50_uniform": {
        "value": round(2048 * 8 * 50 / (0.30 * 38e-3), -5), "unit": "lookups/s",
        "hardware": "one Xeon socket (SKX 8180 or CLX 8280), FP32",
        "derivation": "0.30 x 38 ms optimised Small iteration (Section VI), not printed as such",
    },
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def describe(cfg, act_bf16=False, pooling="sum"):
    kind = "split-BF16 hi/lo" if cfg.split else "FP32"
    act = ", BF16 pooled outputs and gradients" if act_bf16 else ""
    act += {"sum": "", "weighted": ", weighted sum (per-look-up weights U(0.5, 1.5))",
            "mean": ", mean pooling"}[pooling]
    if cfg.name.startswith("mlperf"):
        return (f"{cfg.name}: 26 tables, log-uniform rows in [10, 4e7], {kind} "
                f"({cfg.table_bytes / 1e9:.1f} GB), E=128, batch 65536, 1 look-up/bag, "
                f"Zipf(1.2){act}")
    dist = f"Zipf({cfg.zipf_s})" if cfg.dist == "zipf" else "uniform"
    return (f"{cfg.name}: {cfg.num_tables} tables x {cfg.rows[0]:.0e} rows x E={cfg.dim} {kind} "
            f"({cfg.table_bytes / 1e9:.1f} GB), batch {cfg.batch}, {cfg.pooling} look-ups/bag, "
            f"{dist}{act}")


def bytes_model(cfg, U, split, act_bf16=False, weighted=False):
    """Algorithmic HBM bytes of one step (forward, backward+update).  Row reads of
    the forward are s_w = 4 B (FP32) or 2 B (BF16 hi halves) per element; pooled
    outputs and their gradients s_y = 4 B or 2 B (BF16 activations); the update
    reads and writes 4 B per element of every touched row (FP32, or hi + lo)."""
    T, B, E, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.num_indices
    TB = T * B
    sw = 2 if split else 4
    sy = 2 if act_bf16 else 4
    fwd = NS * E * sw + 4 * NS + 4 * (TB + 1) + sy * TB * E
    bwd = sy * TB * E + 4 * NS + 4 * (TB + 1) + 2 * U * E * 4
    if weighted:  # one weight per look-up, read by the forward and by the update
        fwd += 4 * NS
        bwd += 4 * NS
    return fwd, bwd


def profiled_traffic(workload, call):
    """L2-to-fabric bytes per launch of one call ("forward", "prepare" or
    "apply", all its kernels) from profiles/traffic.json (copy-calibrated
    rocprofv3 FETCH_SIZE + WRITE_SIZE), or None when the record holds no such
    workload or the kernels' sources changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    r = rec.get("workloads", {}).get(workload, {}).get("calls", {}).get(call)
    if r is None:
        return None
    h = hashlib.sha256()
    for src in r["sources"]:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    if h.hexdigest() != r["source_sha256"]:
        return None
    return r["fetch_bytes"] + r["write_bytes"]


def workload_tag(cfg, act_bf16, pooling="sum"):
    return cfg.name + ("+bf16act" if act_bf16 else "") + ("" if pooling == "sum" else "+" + pooling)


def unique_count(cfg, I):
    """Touched (table, row) pairs of one batch (plain numpy on the host)."""
    n_t = cfg.batch * cfg.pooling
    return int(sum(np.unique(I[t * n_t:(t + 1) * n_t]).size for t in range(cfg.num_tables)))


def host_cpu():
    """CPU model and logical CPU count of this host (from /proc/cpuinfo)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{model}, {os.cpu_count()} logical CPUs, {host_ram_gb()} GB RAM"


def host_ram_gb():
    """Installed host memory in GB (MemTotal of /proc/meminfo), or None."""
    try:
        with open("/proc/meminfo") as f:
            for line in f:
                if line.startswith("MemTotal:"):
                    return round(int(line.split()[1]) * 1024 / 1e9, 1)
    except (OSError, ValueError, IndexError):
        pass
    return None


def host_tables(pk, torch, cfg):
    """Every table of the workload in host memory, filled from the counter-based
    generator on the device (for split storage: the hi and lo halves)."""
    from embbag_data import fill_table_torch
    out, out_lo = [], []
    for t, m in enumerate(cfg.rows):
        tmp = torch.empty((m, cfg.dim), dtype=torch.float32, device="cuda")
        fill_table_torch(cfg, t, tmp)
        if cfg.split:
            hi = torch.empty((m, cfg.dim), dtype=torch.int16, device="cuda")
            lo = torch.empty((m, cfg.dim), dtype=torch.int16, device="cuda")
            pk.check(pk.embbag_split_fp32(tmp, hi, lo), "split")
            del tmp
            out.append(hi.cpu().numpy().view(np.uint16))
            out_lo.append(lo.cpu().numpy().view(np.uint16))
            del hi, lo
        else:
            out.append(tmp.cpu().numpy())
            del tmp
    torch.cuda.synchronize()
    return out, out_lo


def cpu_baseline(pk, cfg, host_batches, sample_bags, act_bf16=False, pooling="sum",
                 budget_s=25.0):
    """The CPU oracle on the first `sample_bags` bags of every table of each of
    `host_batches` ((indices, grads, weights or None) on the host), forward +
    fused backward, single-threaded on one host core, stopping after the batch
    that takes it past `budget_s`.  Full-table mode (whole tables in host
    memory, the look-ups reading them at random as on the GPU) where host RAM
    holds 1.1x the tables; otherwise touched-rows mode (each table compacted to
    the rows the sample touches, regenerated from the counter-based generator:
    less memory, and more locality than the full tables would give)."""
    import torch

    import oracle
    from embbag_data import table_rows_torch

    # The paper's multi-core CPU designs on the same sample and tables, on all
    # the cores this process may use (FP32 tables with plain sums only).
    designs = not cfg.split and pooling == "sum"
    if designs:
        import cpu_designs

    P, B, T = cfg.pooling, cfg.batch, cfg.num_tables
    nb = min(sample_bags, B)
    ram = host_ram_gb()
    full = ram is not None and ram * 1e9 >= 1.1 * cfg.table_bytes
    mode = "full-table" if full else "touched-rows"
    t_fill = time.perf_counter()
    if full:
        full_w, full_lo = host_tables(pk, torch, cfg)
    t_fill = time.perf_counter() - t_fill
    dt, dt_f, dt_b, n_look, n_rows, n_batches = 0.0, 0.0, 0.0, 0, 0, 0
    dd_f, dd_b = 0.0, 0.0
    # one host core for the oracle's timed region (it is single-threaded)
    old_aff = os.sched_getaffinity(0)
    core = min(old_aff)
    nthreads = len(old_aff)
    os.sched_setaffinity(0, {core})
    for batch_I, G, A in host_batches:
        if dt > budget_s:
            break
        I_s, tabs, A_s = [], [], []
        for t in range(T):
            part = batch_I[t * B * P: t * B * P + nb * P]
            if A is not None:
                A_s.append(A[t * B * P: t * B * P + nb * P])
            if full:
                I_s.append(part)
                n_rows += np.unique(part).size
                continue
            rows, inv = np.unique(part, return_inverse=True)
            n_rows += rows.size
            I_s.append(inv.astype(np.int32))
            vals = table_rows_torch(cfg.seed, t, torch.from_numpy(rows).cuda(), cfg.dim,
                                    cfg.value_scale[t])
            tabs.append(vals.cpu().numpy())
        if full:
            tabs = full_w
        I_s = np.concatenate(I_s)
        O_s = np.arange(0, T * nb * P + 1, P, dtype=np.int32)
        G_s = np.ascontiguousarray(G[:, :nb, :])
        if cfg.split and full:
            his, los = full_w, full_lo
        elif cfg.split:
            his, los = zip(*[oracle.split(w) for w in tabs])
            his, los = list(his), list(los)
            del tabs
        if cfg.split and act_bf16:
            Gb = np.ascontiguousarray(torch.from_numpy(G_s).to(torch.bfloat16).view(torch.int16)
                                      .numpy().view(np.uint16))
            fwd = lambda: oracle.forward_split_bf16_act(his, nb, I_s, O_s)[0]
            bwd = lambda: oracle.backward_sgd_split_bf16_act(Gb, nb, I_s, O_s, cfg.lr, his, los)
        elif cfg.split:
            fwd = lambda: oracle.forward_split(his, nb, I_s, O_s)[0]
            bwd = lambda: oracle.backward_sgd_split(G_s, nb, I_s, O_s, cfg.lr, his, los)
        elif pooling != "sum":
            mode = oracle.POOL_MEAN if pooling == "mean" else oracle.POOL_SUM
            a = np.ascontiguousarray(np.concatenate(A_s)) if A_s else None
            fwd = lambda: oracle.forward_weighted(tabs, nb, I_s, O_s, a, mode)[0]
            bwd = lambda: oracle.backward_sgd_weighted(G_s, nb, I_s, O_s, cfg.lr, tabs, a, mode)
        else:
            fwd = lambda: oracle.forward(tabs, nb, I_s, O_s)[0]
            bwd = lambda: oracle.backward_sgd(G_s, nb, I_s, O_s, cfg.lr, tabs)
        t0 = time.perf_counter()
        rc1 = fwd()
        t1 = time.perf_counter()
        rc2 = bwd()
        t2 = time.perf_counter()
        dt_f += t1 - t0
        dt_b += t2 - t1
        dt += t2 - t0
        assert rc1 == 0 and rc2 == 0
        if designs:
            os.sched_setaffinity(0, old_aff)
            t0 = time.perf_counter()
            rc3 = cpu_designs.forward(tabs, nb, I_s, O_s, nthreads)[0]
            t1 = time.perf_counter()
            rc4 = cpu_designs.backward_sgd(G_s, nb, I_s, O_s, cfg.lr, tabs, nthreads)
            t2 = time.perf_counter()
            os.sched_setaffinity(0, {core})
            assert rc3 == 0 and rc4 == 0
            dd_f += t1 - t0
            dd_b += t2 - t1
        n_look += I_s.size
        n_batches += 1
    os.sched_setaffinity(0, old_aff)
    if full:
        del full_w, full_lo
    if n_batches == 0:
        return {"value": None, "unit": "lookups/s", "cores": 1, "kind": "oracle",
                "sample": "not timed (no sampled batches)"}
    where = (f"the whole tables in host memory ({cfg.table_bytes / 1e9:.1f} GB, filled in "
             f"{t_fill:.0f} s, not timed)" if full else
             f"tables compacted to the sampled look-ups' rows (host RAM {ram} GB < 1.1x "
             f"{cfg.table_bytes / 1e9:.1f} GB of tables)")
    sample = (f"{mode}: first {nb} of {B} bags of each of the {T} tables of batches "
              f"0-{n_batches - 1} ({n_look} look-ups, {n_rows} touched rows) on {where}")
    res = {"value": n_look / dt, "unit": "lookups/s", "cores": 1, "kind": "oracle",
           "mode": mode,
           "sample": f"{sample}, forward + fused backward/SGD, single-threaded, {dt:.2f} s",
           "host": host_cpu(), "core": core,
           "forward_lookups_per_s": round(n_look / dt_f, 1),
           "backward_sgd_lookups_per_s": round(n_look / dt_b, 1)}
    if designs:
        dd = dd_f + dd_b
        res["paper_designs"] = {
            "value": round(n_look / dd, 1), "unit": "lookups/s", "cores": nthreads,
            "kind": ("the paper's CPU designs, OpenMP, FP32: Algorithm 1 over the bags; "
                     "Algorithms 2-3 fused with Algorithm 4's row ownership"),
            "sample": f"{sample}, the same look-ups after the oracle's, {dd:.2f} s",
            "forward_lookups_per_s": round(n_look / dd_f, 1),
            "backward_sgd_lookups_per_s": round(n_look / dd_b, 1)}
    return res


def calibrate_gather(pk, torch, dev, reps=10):
    """Measured rates of the access patterns the step is made of, on this GPU:
    random whole-row reads (each row once; the library's forward with one
    look-up per bag, which reads the rows and writes them out densely, and
    torch.index_select as a library reference), the same rows in increasing
    order, and random whole-row read-modify-writes (the update's floor kernel,
    each row read and written back once), for 1 KB rows (E = 256) and 512 B rows
    (E = 128), 3.3M distinct rows of a 6.1 GB table.  Also random 512 B reads of
    every row of an 872 MB array (the MLPerf-shaped gradient, read once in a
    random order by the update)."""
    def timed(fn):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    g = torch.Generator(device=dev)
    g.manual_seed(20050468)
    out = {"calibration": "gather", "reps": reps}
    U = 3276528
    for E, M in ((256, 6_000_000), (128, 12_000_000)):
        row = 4 * E
        w = torch.empty((M, E), dtype=torch.float32, device=dev)
        w.normal_(generator=g)
        rows = torch.randperm(M, generator=g, device=dev)[:U].to(torch.int32)
        srt = torch.sort(rows).values
        O = torch.arange(U + 1, dtype=torch.int32, device=dev)
        Y = torch.empty((1, U, E), dtype=torch.float32, device=dev)
        status = torch.zeros(1, dtype=torch.int32, device=dev)
        r = {"row_bytes": row, "rows": U, "table_gb": round(M * row / 1e9, 2)}
        for name, idx in (("random", rows), ("sorted", srt)):
            ms = timed(lambda: pk.check(pk.embbag_forward([w], U, idx, O, Y, status), "forward"))
            r[f"read_{name}_ms"] = round(ms, 4)
            r[f"read_{name}_gbps"] = round(U * row / (ms * 1e-3) / 1e9, 1)
            r[f"read_{name}_plus_write_gbps"] = round(2 * U * row / (ms * 1e-3) / 1e9, 1)
        il = rows.to(torch.int64)
        ms = timed(lambda: torch.index_select(w, 0, il))
        r["index_select_random_plus_write_gbps"] = round(2 * U * row / (ms * 1e-3) / 1e9, 1)
        ws = torch.empty(pk.embbag_backward_workspace_bytes(1, U, U, E), dtype=torch.uint8,
                         device=dev)
        pk.check(pk.embbag_backward_prepare([M], E, U, rows, O, ws, status), "prepare")
        ms = timed(lambda: pk.check(pk.embbag_baseline_touch_rows(U, U, [w], ws), "touch"))
        r["rmw_random_ms"] = round(ms, 4)
        r["rmw_random_gbps"] = round(2 * U * row / (ms * 1e-3) / 1e9, 1)
        assert pk.embbag_status_read(status) == 0
        out[f"rows_{row}B"] = r
        del w, rows, srt, O, Y, ws, il
        torch.cuda.empty_cache()
    n, E = 65536 * 26, 128
    a = torch.empty((n, E), dtype=torch.float32, device=dev)
    a.normal_(generator=g)
    perm = torch.randperm(n, generator=g, device=dev)
    ms = timed(lambda: torch.index_select(a, 0, perm))
    out["perm_read_512B"] = {"array_mb": round(n * E * 4 / 1e6, 1),
                             "ms": round(ms, 4),
                             "read_gbps": round(n * E * 4 / (ms * 1e-3) / 1e9, 1),
                             "read_plus_write_gbps": round(2 * n * E * 4 / (ms * 1e-3) / 1e9, 1)}
    return out


def time_graph(torch, batches, prep, fwd, apply, K, warmup, fork=False):
    """The step (forward, prepare, apply) captured once per batch as a HIP graph;
    K replays rotating over the batches, timed with events on the replay stream.
    With `fork`, the prepare (which reads only the indices and offsets) is a
    branch of its own beside the forward, and the apply waits for both."""
    graphs = []
    side = torch.cuda.Stream() if fork else None
    for bt in batches:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            cap = torch.cuda.current_stream()
            if fork:
                side.wait_stream(cap)
                rp = prep(bt, side)
                rf = fwd(bt, cap)
                cap.wait_stream(side)
                rcs = (rf, rp, apply(bt, cap))
            else:
                rcs = (fwd(bt), prep(bt), apply(bt))
        assert rcs == (0, 0, 0), rcs
        graphs.append(g)
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        graphs[i % len(graphs)].replay()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(K):
        graphs[i % len(graphs)].replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    del graphs
    return {"ms_per_step": round(ms, 4), "replays": K, "graphs": len(batches),
            "prepare": "beside the forward" if fork else "after the forward"}


def time_floor(pk, torch, touch, bt, prep, stream, K):
    """Mean ms of the update's floor on the rows of batch `bt`: every touched
    row read and written back once (`touch`: embbag_baseline_touch_rows or its
    split-storage form, which leave the tables unchanged), K calls back to
    back on one prepared workspace between two events on `stream`."""
    pk.check(prep(bt), "prepare")
    pk.check(touch(), "touch rows")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(K):
        pk.check(touch(), "touch rows")
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / K


def time_baselines(pk, torch, cfg, tables, batches, stream, reps=3):
    """Average ms per step of the unfused designs, same workload and stream."""
    T, B, E, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.num_indices
    dW = torch.empty((NS, E), dtype=torch.float32, device=tables[0].device)
    res = {}

    def timed(fn, n):
        fn(batches[0])  # warm-up
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for i in range(n):
            fn(batches[i % len(batches)])
        ev1.record(stream)
        torch.cuda.synchronize()
        return round(ev0.elapsed_time(ev1) / n, 4)

    res["alg2_materialize_ms"] = timed(
        lambda bt: pk.check(pk.embbag_baseline_materialize(bt["G"], T, B, E, bt["O"], NS, dW)), reps)
    res["alg3_atomic_update_ms"] = timed(
        lambda bt: pk.check(pk.embbag_baseline_update_atomic(dW, B, bt["I"], bt["O"], cfg.lr,
                                                             tables)), reps)
    res["alg2_3_fused_atomic_ms"] = timed(
        lambda bt: pk.check(pk.embbag_baseline_backward_sgd_atomic(bt["G"], B, bt["I"], bt["O"],
                                                                   cfg.lr, tables)), reps)
    res["alg4_owner_update_ms"] = timed(
        lambda bt: pk.check(pk.embbag_baseline_update_owner(dW, B, bt["I"], bt["O"], cfg.lr,
                                                            tables, 256)), 1)
    res["note"] = ("unfused = alg2 + alg3 (or alg2 + alg4); the fused sort-and-segment backward "
                   "is bwd_prepare_ms + bwd_apply_ms")
    del dW
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="large",
                    choices=["tiny", "small", "large", "mlperf", "split", "large_split",
                             "mlperf_split", "small_p50_uniform", "large_uniform"])
    ap.add_argument("--pooling", default="sum", choices=["sum", "weighted", "mean"],
                    help="sum (the paper's default), weighted sum with per-look-up weights "
                         "U(0.5, 1.5), or mean (FP32 tables only)")
    ap.add_argument("--act", default="f32", choices=["f32", "bf16"],
                    help="pooled outputs and their gradients in FP32, or in BF16 (split-storage "
                         "configurations only: Section VII's BF16 activations)")
    ap.add_argument("--batches", type=int, default=8, help="pre-generated batches, rotated")
    ap.add_argument("--table-alloc", default="separate", choices=["separate", "one"],
                    help="FP32 tables as one device allocation each, or as row ranges of a "
                         "single allocation")
    ap.add_argument("--cpu-sample-bags", type=int, default=8192,
                    help="bags per table of each sampled batch the CPU oracle is timed on")
    ap.add_argument("--cpu-sample-batches", type=int, default=3,
                    help="batches the CPU oracle (and the paper's CPU designs) are timed on "
                         "(about 20 s of oracle time at Large)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--overlap-prepare", action="store_true",
                    help="run the backward's index phase on a second stream, overlapped with "
                         "the forward (measured slower on MI355X: both are memory-bound)")
    ap.add_argument("--baselines", action="store_true",
                    help="also time the paper's unfused update designs on the GPU: Algorithm 2 "
                         "(materialised dW) + Algorithm 3 (FP32 atomics), the fused atomic update, "
                         "and Algorithm 4 (row-range ownership, 256 owners)")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured as one HIP graph per batch and replayed "
                         "(for the launch-bound small workloads)")
    ap.add_argument("--calibrate-gather", action="store_true",
                    help="only measure random row reads and read-modify-writes of 1 KB and "
                         "512 B rows (the access patterns of the step) on this GPU")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 5 times (the reference "
                         "kernel that scales rocprofv3 FETCH_SIZE/WRITE_SIZE to bytes)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "the library runs on one GPU; --gpus must be 1 "
                                   "(the tables would shard table-wise across GPUs, with an "
                                   "all-to-all of pooled rows and gradients, but no multi-GPU "
                                   "path is implemented)"}))
        sys.exit(2)

    import torch

    import paper_2005_04680_amd as pk
    from embbag_data import (fill_table_torch, fill_tables_torch, get_config, make_batch,
                             make_grads, make_weights)

    pk.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_gather:
        print(json.dumps(calibrate_gather(pk, torch, dev)), flush=True)
        return
    if args.calibrate_copy:
        n = 1 << 28  # 1 GiB of FP32
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        dst.copy_(src)
        e0.record()
        for _ in range(5):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 5
        print(json.dumps({"calibration": "copy", "bytes_read_per_copy": 4 * n,
                          "bytes_written_per_copy": 4 * n, "copies": 6,
                          "ms_per_copy": round(ms, 4),
                          "gbps_read_plus_write": round(8 * n / (ms * 1e-3) / 1e9, 1)}),
              flush=True)
        return
    cfg = get_config(args.config)
    T, B, E, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.num_indices
    split = cfg.split
    act_bf16 = args.act == "bf16"
    if act_bf16 and not split:
        print(json.dumps({"error": "--act bf16 needs a split-storage configuration"}))
        sys.exit(2)
    pooled = args.pooling != "sum"
    if pooled and split:
        print(json.dumps({"error": "--pooling weighted/mean runs on FP32 tables"}))
        sys.exit(2)
    pool_code = pk.EMBBAG_POOL_MEAN if args.pooling == "mean" else pk.EMBBAG_POOL_SUM

    # ---- tables in HBM ----------------------------------------------------
    t0 = time.time()
    if split:
        hi = [torch.empty((m, E), dtype=torch.int16, device=dev) for m in cfg.rows]
        lo = [torch.empty((m, E), dtype=torch.int16, device=dev) for m in cfg.rows]
        for t, m in enumerate(cfg.rows):
            tmp = torch.empty((m, E), dtype=torch.float32, device=dev)
            fill_table_torch(cfg, t, tmp)
            pk.check(pk.embbag_split_fp32(tmp, hi[t], lo[t]), "split")
            del tmp
        tables = None
    elif args.table_alloc == "one":
        whole = torch.empty((sum(cfg.rows), E), dtype=torch.float32, device=dev)
        base = np.concatenate([[0], np.cumsum(cfg.rows)])
        tables = [whole[int(base[t]):int(base[t + 1])] for t in range(T)]
        fill_tables_torch(cfg, tables)
    else:
        tables = [torch.empty((m, E), dtype=torch.float32, device=dev) for m in cfg.rows]
        fill_tables_torch(cfg, tables)
    torch.cuda.synchronize()
    log(f"[bench] tables filled ({cfg.table_bytes / 1e9:.1f} GB) in {time.time() - t0:.1f}s")

    # ---- batches ----------------------------------------------------------
    t0 = time.time()
    batches = []
    for b in range(args.batches):
        I, O = make_batch(cfg, b, device=dev)
        G = make_grads(cfg, b)
        U = unique_count(cfg, I)
        Gd = torch.from_numpy(G).to(dev)
        if act_bf16:
            Gd = Gd.to(torch.bfloat16)  # the gradient a BF16 network hands over
        keep = b < args.cpu_sample_batches and not args.no_cpu_baseline
        A = make_weights(cfg, b) if args.pooling == "weighted" else None
        batches.append(dict(I=torch.from_numpy(I).to(dev), O=torch.from_numpy(O).to(dev),
                            G=Gd, U=U, I_host=I if keep else None, G_host=G if keep else None,
                            A=None if A is None else torch.from_numpy(A).to(dev),
                            A_host=A if keep else None))
    log(f"[bench] {args.batches} batches generated in {time.time() - t0:.1f}s; "
        f"U = {[x['U'] for x in batches]}")

    Y = torch.empty((T, B, E), dtype=torch.bfloat16 if act_bf16 else torch.float32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    ws = torch.empty(pk.embbag_backward_workspace_bytes(T, B, NS, E), dtype=torch.uint8, device=dev)
    # The tables' C descriptor, built once: per call the binding then checks
    # only the other buffers (a list would be checked and rebuilt each call).
    td = pk.SplitTables(hi, lo) if split else pk.Tables(tables)

    # (st: the stream to launch on; None: the current one, as under graph capture)
    def fwd(bt, st=None):
        if pooled:
            return pk.embbag_forward_pooled(td, B, bt["I"], bt["O"], Y, bt["A"], pool_code, status,
                                            st)
        if act_bf16:
            return pk.embbag_forward_split_bf16_act(td, B, bt["I"], bt["O"], Y, status, st)
        if split:
            return pk.embbag_forward_split_bf16(td, B, bt["I"], bt["O"], Y, status, st)
        return pk.embbag_forward(td, B, bt["I"], bt["O"], Y, status, st)

    def prep(bt, st=None):
        if pooled:
            return pk.embbag_backward_prepare_pooled(td, E, B, bt["I"], bt["O"], ws, bt["A"],
                                                     pool_code, status, st)
        return pk.embbag_backward_prepare(td, E, B, bt["I"], bt["O"], ws, status, st)

    def apply(bt, st=None):
        if pooled:
            return pk.embbag_backward_apply_sgd_pooled(bt["G"], B, bt["O"], NS, cfg.lr, td, ws,
                                                       bt["A"], pool_code, st)
        if act_bf16:
            return pk.embbag_backward_apply_sgd_split_bf16_act(bt["G"], B, NS, cfg.lr, td, None, ws,
                                                               st)
        if split:
            return pk.embbag_backward_apply_sgd_split_bf16(bt["G"], B, NS, cfg.lr, td, None, ws, st)
        return pk.embbag_backward_apply_sgd(bt["G"], B, NS, cfg.lr, td, ws, st)

    def bwd(bt):
        rc = prep(bt)
        return rc if rc else apply(bt)

    main = torch.cuda.current_stream()
    side = torch.cuda.Stream(device=dev) if args.overlap_prepare else main

    def step(bt, prev, evs=None):
        """One step: forward, prepare (on `side`, after `prev`), apply; returns
        the event after the apply.  `evs` (six timing events) bracket the calls."""
        e_f0, e_f1, e_p0, e_p1, e_a0, e_a1 = evs if evs is not None else tuple(
            torch.cuda.Event(enable_timing=False) for _ in range(6))
        # Forward first, as in a training step; the index phase needs only the
        # indices and offsets, so it follows (or, with --overlap-prepare, runs
        # beside) the forward, and its sorted look-ups are then still in the
        # MALL when the apply reads them.
        e_f0.record(main)
        pk.check(fwd(bt, main), "forward")
        e_f1.record(main)
        side.wait_event(prev)
        e_p0.record(side)
        pk.check(prep(bt, side), "prepare")
        e_p1.record(side)
        main.wait_event(e_p1)
        e_a0.record(main)
        pk.check(apply(bt, main), "apply")
        e_a1.record(main)
        return e_a1

    # warm-up in the same stream pattern as the timed steps
    prev = torch.cuda.Event()
    prev.record(main)
    for i in range(args.warmup):
        prev = step(batches[i % len(batches)], prev)
    torch.cuda.synchronize()
    pk.check(pk.embbag_status_read(status), "device status")

    # ---- timed steps ------------------------------------------------------
    # The backward's index phase (prepare) reads only indices and offsets, so
    # with --overlap-prepare it runs on a second stream while the forward
    # gathers rows; the apply phase waits for both, and the next step's
    # prepare waits for this step's apply, which still reads the workspace.
    K = args.steps
    ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(6)) for _ in range(K)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(main)
    prev_apply = start
    for i in range(K):
        prev_apply = step(batches[i % len(batches)], prev_apply, ev[i])
    stop.record(main)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    pk.check(pk.embbag_status_read(status), "device status")
    total_ms = start.elapsed_time(stop)
    fwd_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / K
    prep_ms = sum(e[2].elapsed_time(e[3]) for e in ev) / K
    apply_ms = sum(e[4].elapsed_time(e[5]) for e in ev) / K
    ms_step = total_ms / K
    # per-step times: consecutive steps partition the timed region
    per_step = [(start if i == 0 else ev[i - 1][5]).elapsed_time(ev[i][5]) for i in range(K)]
    U_avg = sum(batches[i % len(batches)]["U"] for i in range(K)) / K
    fwd_b, bwd_b = bytes_model(cfg, U_avg, split, act_bf16, args.pooling == "weighted")
    step_b = fwd_b + bwd_b
    gbps = step_b / (ms_step * 1e-3) / 1e9
    # B_min: the forward counted with one read per touched row instead of one per look-up
    sw = 2 if split else 4
    step_min_b = step_b - (NS - U_avg) * E * sw
    gbps_min = step_min_b / (ms_step * 1e-3) / 1e9
    # Roofline of the dominant kernel.  The forward call is one launch
    # (fwd_gather_sum); the apply call is segment_sgd plus the short
    # carry_group and segment_fixup, whose events bracket all three.  Algorithmic bytes per launch:
    # forward = NS*E*s_w + 4*NS + 4*(TB+1) + s_y*TB*E (every look-up reads its
    # row); apply = dY once (s_y*TB*E) + the sorted look-ups (8*NS) + one read
    # and one write of every touched row (2*U*E*4).
    TB = T * B
    sy = 2 if act_bf16 else 4
    apply_b = sy * TB * E + 8 * NS + 2 * U_avg * E * 4 + (4 * NS if args.pooling == "weighted" else 0)
    if apply_ms >= fwd_ms:
        roof_call, roof_k, roof_b, roof_ms = ("apply", "segment_sgd+carry_group+segment_fixup",
                                              apply_b, apply_ms)
    else:
        roof_call, roof_k, roof_b, roof_ms = "forward", "fwd_gather_sum", fwd_b, fwd_ms
    achieved = roof_b / (roof_ms * 1e-3) / 1e9
    wtag = workload_tag(cfg, act_bf16, args.pooling)
    roof = {"kernel": roof_k, "bound": "hbm", "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": profiled_traffic(wtag, roof_call),
            "bytes_per_launch": int(roof_b),
            "avg_launch_ms": round(roof_ms, 4)}
    # Measured bytes of the whole step: the counter traffic (L2-to-fabric
    # fetch + write, which MALL hits also count) of the forward, prepare and
    # apply calls, per step, over the step time.
    calls = [profiled_traffic(wtag, c) for c in ("forward", "prepare", "apply")]
    step_traffic = None
    if all(c is not None for c in calls):
        tb = sum(calls)
        step_traffic = {"bytes": int(tb), "gbps": round(tb / (ms_step * 1e-3) / 1e9, 1),
                        "pct_hbm_peak": round(100 * tb / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
                        "forward_bytes": int(calls[0]), "prepare_bytes": int(calls[1]),
                        "apply_bytes": int(calls[2])}
    if roof_call == "apply" and not pooled and not act_bf16:
        # The apply's floor on this GPU: the read and write-back of the same
        # touched rows with nothing summed (no gradient gathers).
        # (the rows of batch 0; its U is within 0.2% of the average)
        if split:
            touch = lambda: pk.embbag_baseline_touch_rows_split(B, NS, td, None, ws)
        else:
            touch = lambda: pk.embbag_baseline_touch_rows(B, NS, td, ws)
        floor_ms = time_floor(pk, torch, touch, batches[0], prep, main, K)
        roof["floor_ms"] = round(floor_ms, 4)
        roof["floor_gbps"] = round(2 * batches[0]["U"] * E * 4 / (floor_ms * 1e-3) / 1e9, 1)
        roof["frac_of_floor"] = round(floor_ms / roof_ms, 4)

    out = {
        "metric": METRIC,
        "value": round(NS / (ms_step * 1e-3), 1),
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": describe(cfg, act_bf16, args.pooling), "tables": T, "dim": E,
                   "batch": B,
                   "pooling": cfg.pooling, "num_indices": NS, "unique_rows": round(U_avg),
                   "lr": cfg.lr, "batches_rotated": args.batches,
                   "table_alloc": args.table_alloc,
                   "streams": 2 if args.overlap_prepare else 1},
        "ms_per_step_median": round(float(np.median(per_step)), 4),
        "ms_per_step_p90": round(float(np.percentile(per_step, 90)), 4),
        "gbps_alg": round(gbps, 1),
        "pct_hbm_peak": round(100 * gbps / HBM_PEAK_GBPS, 2),
        "pct_hbm_peak_model": ("algorithmic bytes, every look-up's whole row read counted as "
                               "Section II frames it (GUPS-like); on Zipf data repeated rows are "
                               "L2/MALL hits, so this exceeds the HBM-delivered share"),
        "bytes_alg_per_step": int(step_b),
        "gbps_min": round(gbps_min, 1),
        "pct_hbm_peak_min": round(100 * gbps_min / HBM_PEAK_GBPS, 2),
        "bytes_min_per_step": int(step_min_b),
        "traffic_step": step_traffic,
        "fwd_ms": round(fwd_ms, 4),
        "bwd_prepare_ms": round(prep_ms, 4),
        "bwd_apply_ms": round(apply_ms, 4),
        "wall_s_timed": round(wall, 3),
        "roofline": roof,
    }
    if cfg.name in PAPER_CONTEXT and not pooled and not act_bf16:
        out["paper_context"] = PAPER_CONTEXT[cfg.name]
    if args.graph:
        out["graph"] = time_graph(torch, batches, prep, fwd, apply, K, args.warmup)
        out["graph_fork"] = time_graph(torch, batches, prep, fwd, apply, K, args.warmup,
                                       fork=True)
    if args.baselines and not split:
        out["baselines"] = time_baselines(pk, torch, cfg, tables, batches, main)
    if not args.no_cpu_baseline:
        host = [(bt["I_host"], bt["G_host"], bt["A_host"]) for bt in batches
                if bt["I_host"] is not None]
        out["cpu_baseline"] = cpu_baseline(pk, cfg, host, args.cpu_sample_bags, act_bf16,
                                           args.pooling)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
