"""Stream and graph use of the boundary.

The training step (backward prepare, forward, backward apply) captured as a
HIP graph and replayed: every replay must give, bit for bit, what the same
calls give when launched directly (the kernels are deterministic).  Eager work
and synchronisations run between the replays, and each replay is checked.
Two steps on two streams at once, each with its own buffers, must both match
the oracle."""
import numpy as np
import pytest
import torch

import paper_2005_04680_amd as pk
from embbag_data import get_config, make_batch, make_grads, scaled, table_values_np
from gpu_util import DEV, bits_equal, log, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _same_bits(x, y):
    if x.dtype == torch.float32:
        x, y = x.view(torch.int32), y.view(torch.int32)
    return torch.equal(x, y)


@pytest.mark.parametrize("split,fork", [(False, False), (True, False), (False, True),
                                        (True, True)])
def test_graph_replays_match_direct_launches(split, fork):
    """With `fork`, the captured prepare is a branch of its own (a second
    stream, joined before the apply) beside the forward, as a training step
    may schedule it; the replays must still equal the direct launches."""
    cfg = scaled(get_config("small"), rows=20000, batch=512)
    T, B, E, NS = cfg.num_tables, cfg.batch, cfg.dim, cfg.num_indices
    log(f"[graph] split={split} fork={fork} T={T} B={B} E={E} NS={NS}")
    host = [table_values_np(cfg.seed, t, np.arange(cfg.rows[t]), E, cfg.value_scale[t])
            for t in range(T)]

    def tables():
        if not split:
            return [torch.from_numpy(w).to(DEV) for w in host], None
        hi, lo = [], []
        for w in host:
            wd = torch.from_numpy(w).to(DEV)
            h = torch.empty(w.shape, dtype=torch.int16, device=DEV)
            l = torch.empty(w.shape, dtype=torch.int16, device=DEV)
            assert pk.embbag_split_fp32(wd, h, l) == 0
            hi.append(h)
            lo.append(l)
        return hi, lo

    batches = []
    for b in range(2):
        I, O = make_batch(cfg, b)
        batches.append(tuple(torch.from_numpy(a).to(DEV) for a in (I, O, make_grads(cfg, b))))

    def step(w, lo, bt, Y, ws, status):
        Id, Od, Gd = bt
        rc = pk.embbag_backward_prepare(cfg.rows, E, B, Id, Od, ws, status)
        if split:
            rc = rc or pk.embbag_forward_split_bf16(w, B, Id, Od, Y, status)
            rc = rc or pk.embbag_backward_apply_sgd_split_bf16(Gd, B, NS, cfg.lr, w, lo, ws)
        else:
            rc = rc or pk.embbag_forward(w, B, Id, Od, Y, status)
            rc = rc or pk.embbag_backward_apply_sgd(Gd, B, NS, cfg.lr, w, ws)
        return rc

    nbytes = pk.embbag_backward_workspace_bytes(T, B, NS, E)
    wa, la = tables()  # replayed by the graph
    wb, lb = tables()  # launched directly
    Ya = torch.empty((T, B, E), dtype=torch.float32, device=DEV)
    Yb = torch.empty_like(Ya)
    wsa = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    wsb = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    sta = torch.zeros(1, dtype=torch.int32, device=DEV)
    stb = torch.zeros(1, dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()

    def step_fork(w, lo, bt, Y, ws, status):
        Id, Od, Gd = bt
        cap = torch.cuda.current_stream()
        side = torch.cuda.Stream(device=DEV)
        side.wait_stream(cap)
        rc = pk.embbag_backward_prepare(cfg.rows, E, B, Id, Od, ws, status, side)
        if split:
            rc = rc or pk.embbag_forward_split_bf16(w, B, Id, Od, Y, status, cap)
        else:
            rc = rc or pk.embbag_forward(w, B, Id, Od, Y, status, cap)
        cap.wait_stream(side)
        if split:
            rc = rc or pk.embbag_backward_apply_sgd_split_bf16(Gd, B, NS, cfg.lr, w, lo, ws, cap)
        else:
            rc = rc or pk.embbag_backward_apply_sgd(Gd, B, NS, cfg.lr, w, ws, cap)
        return rc

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rc = (step_fork if fork else step)(wa, la, batches[0], Ya, wsa, sta)
    assert rc == 0
    torch.cuda.synchronize()
    # capture does not run the work: the tables are still the initial ones
    for x, y in zip(wa, wb):
        assert _same_bits(x, y)

    for it in range(4):
        g.replay()
        torch.cuda.synchronize()
        assert step(wb, lb, batches[0], Yb, wsb, stb) == 0
        # unrelated direct work between replays (the other batch, own buffers)
        scratch_Y = torch.empty_like(Ya)
        I1, O1, _ = batches[1]
        if split:
            assert pk.embbag_forward_split_bf16(wb, B, I1, O1, scratch_Y, stb) == 0
        else:
            assert pk.embbag_forward(wb, B, I1, O1, scratch_Y, stb) == 0
        torch.cuda.synchronize()
        assert pk.embbag_status_read(sta) == 0 and pk.embbag_status_read(stb) == 0
        assert bits_equal(Ya.cpu().numpy(), Yb.cpu().numpy()), f"replay {it}: pooled outputs differ"
        for t in range(T):
            assert _same_bits(wa[t], wb[t]), f"replay {it}: table {t} differs"
            if split:
                assert torch.equal(la[t], lb[t]), f"replay {it}: lo half {t} differs"
        log(f"[graph] replay {it} ok")
    del g


def test_two_streams_at_once():
    """The library keeps no global state: two steps on two streams, each with
    its own tables and workspace, overlap and both match the oracle."""
    import oracle
    from gpu_util import GpuTables, assert_close
    from embbag_data import random_bags

    def inputs(seed):
        rng = np.random.default_rng(seed)
        rows, E, B = (3000, 500, 2000), 64, 300
        W = [rng.uniform(-0.05, 0.05, (m, E)).astype(np.float32) for m in rows]
        I, O = random_bags(rng, rows, B, 20, 0.05, 0.3)
        G = rng.standard_normal((len(rows), B, E)).astype(np.float32)
        return rows, E, B, W, I, O, G

    cases = [inputs(1), inputs(2)]
    gts = [GpuTables(c[3]) for c in cases]
    streams = [torch.cuda.Stream(device=DEV), torch.cuda.Stream(device=DEV)]
    outs = []
    torch.cuda.synchronize()
    for (rows, E, B, W, I, O, G), gt, st in zip(cases, gts, streams):
        with torch.cuda.stream(st):
            Id, Od, Gd = (torch.from_numpy(a).to(DEV, non_blocking=False) for a in (I, O, G))
            Y = torch.empty((len(rows), B, E), dtype=torch.float32, device=DEV)
            ws = torch.empty(pk.embbag_backward_workspace_bytes(len(rows), B, I.size, E),
                             dtype=torch.uint8, device=DEV)
            for _ in range(3):  # several launches in flight on each stream
                assert pk.embbag_forward(gt.w, B, Id, Od, Y, gt.status) == 0
            assert pk.embbag_backward_sgd(Gd, B, Id, Od, 0.1, gt.w, ws, gt.status) == 0
            outs.append((Y, Id, Od, Gd, ws))
    torch.cuda.synchronize()
    for (rows, E, B, W, I, O, G), gt, (Y, *_keep) in zip(cases, gts, outs):
        assert gt.read_status() == 0
        rc, Yref = oracle.forward(W, B, I, O)
        assert rc == 0
        assert_close(Y.cpu().numpy(), Yref, "pooled")
        Wref = [w.copy() for w in W]
        assert oracle.backward_sgd(G, B, I, O, 0.1, Wref) == 0
        for t, (wg, wr) in enumerate(zip(gt.host(), Wref)):
            assert_close(wg, wr, f"table {t}")
