"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare it with the CPU oracle on the same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2005_04680_amd as pk

DEV = "cuda:0"
RTOL, ATOL = 1e-5, 1e-6  # FP32 pooled outputs and updated rows vs the FP64 oracle


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def require_gpu():
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    pk.lib()  # fails loudly if libembbag.so is missing


def within_tol(gpu, ref, rtol=RTOL, atol=ATOL):
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    err = np.abs(g - r)
    ok = err <= atol + rtol * np.abs(r)
    return bool(ok.all()), float(err.max()) if err.size else 0.0


def assert_close(gpu, ref, what, rtol=RTOL, atol=ATOL):
    ok, emax = within_tol(gpu, ref, rtol, atol)
    if not ok:
        g = np.asarray(gpu, np.float64)
        r = np.asarray(ref, np.float64)
        bad = np.argwhere(np.abs(g - r) > atol + rtol * np.abs(r))
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} elements out of tolerance, max err {emax:.3e}; "
                             f"first at {i}: gpu {g[i]!r} oracle {r[i]!r}")


def bf16_bits(t):
    """Host uint16 bit patterns of a GPU bfloat16 (or 16-bit integer) tensor."""
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def to_bf16_bits(x):
    """FP32 host array -> BF16 bit patterns by torch's round-to-nearest-even
    (input preparation: the gradient an upstream BF16 network hands over)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def assert_bf16_bracket(gpu_bits, ref32, what, rtol=RTOL, atol=ATOL):
    """BF16 pooled outputs: the GPU rounds its FP32 sum, which is within the
    FP32 tolerance of the oracle's, to the nearest BF16.  Rounding is monotone,
    so each GPU value must lie between the roundings of ref -/+ tolerance.
    Returns the number of values that differ from the rounding of ref itself."""
    r = np.asarray(ref32, np.float64)
    tol = atol + rtol * np.abs(r)
    lo32 = np.nextafter((r - tol).astype(np.float32), np.float32(-np.inf))
    hi32 = np.nextafter((r + tol).astype(np.float32), np.float32(np.inf))
    lo = oracle.bf16_widen(oracle.bf16_round(lo32))
    hi = oracle.bf16_widen(oracle.bf16_round(hi32))
    g = oracle.bf16_widen(np.ascontiguousarray(gpu_bits, np.uint16))
    bad = ~((g >= lo) & (g <= hi))
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: {int(bad.sum())} BF16 values outside the rounding bracket; "
                             f"first at {i}: gpu {g[i]!r} oracle fp32 {r[i]!r}")
    exact = oracle.bf16_round(np.ascontiguousarray(ref32, np.float32))
    return int((np.ascontiguousarray(gpu_bits, np.uint16) != exact).sum())


def bits_equal(a, b):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    return a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8))


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


class GpuTables:
    """FP32 (or split hi/lo) tables resident on the GPU, driven through the C ABI."""

    def __init__(self, host_tables=None, split=False, dev_tables=None, dev_lo=None):
        self.split = split
        if dev_tables is not None:
            self.w = dev_tables
            self.lo = dev_lo
        elif split:
            self.w, self.lo = [], []
            for h in host_tables:
                hi, lo = oracle.split(h)
                self.w.append(to_dev(hi.view(np.int16)))
                self.lo.append(to_dev(lo.view(np.int16)))
        else:
            self.w = [to_dev(h) for h in host_tables]
            self.lo = None
        self.dim = int(self.w[0].shape[1])
        self.status = torch.zeros(1, dtype=torch.int32, device=DEV)

    def forward(self, batch, I, O, out=None):
        T = len(self.w)
        Id, Od = (to_dev(I) if isinstance(I, np.ndarray) else I), (to_dev(O) if isinstance(O, np.ndarray) else O)
        Y = out if out is not None else torch.empty((T, batch, self.dim), dtype=torch.float32, device=DEV)
        if self.split:
            rc = pk.embbag_forward_split_bf16(self.w, batch, Id, Od, Y, self.status)
        else:
            rc = pk.embbag_forward(self.w, batch, Id, Od, Y, self.status)
        return rc, Y

    def backward(self, G, batch, I, O, lr, ws=None):
        T = len(self.w)
        Id, Od = (to_dev(I) if isinstance(I, np.ndarray) else I), (to_dev(O) if isinstance(O, np.ndarray) else O)
        Gd = to_dev(G) if isinstance(G, np.ndarray) else G
        if ws is None:
            n = pk.embbag_backward_workspace_bytes(T, batch, Id.numel(), self.dim)
            ws = torch.empty(max(n, 1), dtype=torch.uint8, device=DEV)
        if self.split:
            return pk.embbag_backward_sgd_split_bf16(Gd, batch, Id, Od, lr, self.w, self.lo, ws,
                                                     self.status)
        return pk.embbag_backward_sgd(Gd, batch, Id, Od, lr, self.w, ws, self.status)

    def read_status(self):
        return pk.embbag_status_read(self.status)

    def reset_status(self):
        self.status.zero_()

    def host(self):
        """FP32 host copies of the tables (split: recombined on the host by the oracle)."""
        torch.cuda.synchronize()
        if self.split:
            return [oracle.combine(h.cpu().numpy().view(np.uint16), l.cpu().numpy().view(np.uint16))
                    for h, l in zip(self.w, self.lo)]
        return [w.cpu().numpy() for w in self.w]

    def host_split(self):
        torch.cuda.synchronize()
        return ([h.cpu().numpy().view(np.uint16) for h in self.w],
                [l.cpu().numpy().view(np.uint16) for l in self.lo])


def gpu_dedup(rows, batch, I, O):
    NS = int(I.size)
    Id, Od = to_dev(I), to_dev(O)
    n = max(NS, 1)
    sk = torch.empty(n, dtype=torch.int32, device=DEV)
    sb = torch.empty(n, dtype=torch.int32, device=DEV)
    uk = torch.empty(n, dtype=torch.int32, device=DEV)
    so = torch.empty(n + 1, dtype=torch.int32, device=DEV)
    nu = torch.empty(1, dtype=torch.int32, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(max(1, pk.embbag_dedup_workspace_bytes(len(rows), batch, NS)), dtype=torch.uint8,
                     device=DEV)
    rc = pk.embbag_dedup(rows, batch, Id, Od, sk, sb, uk, so, nu, ws, st)
    status = pk.embbag_status_read(st)
    U = int(nu.item())
    return rc, status, dict(sorted_keys=sk[:NS].cpu().numpy().view(np.uint32),
                            sorted_bags=sb[:NS].cpu().numpy().view(np.uint32),
                            unique_keys=uk[:U].cpu().numpy().view(np.uint32),
                            seg_off=so[:U + 1].cpu().numpy(), num_unique=U)
