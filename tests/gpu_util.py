"""Helpers for the GPU parity tests (device upload, error metrics)."""

import sys

import numpy as np

FP32_TOL = 1e-4     # max normwise relative error, fp32 path
BF16_TOL = 2e-2     # bf16-input MFMA path


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def relerr(got, want):
    """max_i |g_i - o_i| / max_i |o_i| (normwise infinity)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    if want.size == 0:
        return 0.0
    den = np.max(np.abs(want))
    num = np.max(np.abs(got - want))
    if den == 0:
        return float(num)
    return float(num / den)


def to_dev(x, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def to_host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def csr_to_dev(csr, transpose=False):
    """Upload an oracle/library CSR dict; returns (gist_csr_dev, keepalive)."""
    from paper_2102_10424_amd import gist as G
    k = "t_" if transpose else ""
    nnz = int(csr["nnz"])
    rp = to_dev(np.asarray(csr[k + "rowptr"], dtype=np.int32))
    col = to_dev(np.asarray(csr[k + "col"], dtype=np.int32)[:max(nnz, 1)] if nnz else
                 np.zeros(1, np.int32))
    val = to_dev(np.asarray(csr[k + "val"], dtype=np.float32)[:max(nnz, 1)] if nnz else
                 np.zeros(1, np.float32))
    rows = csr.get("n_in", csr["n"]) if transpose else csr["n"]   # rectangular: n x n_in
    return G.csr_dev(rows, nnz, rp, col, val), (rp, col, val)


def gpu_orders(kind, s):
    """The association order GIST_ORDER_AUTO takes for each GCN layer of
    slice widths s (include/gist.h: aggregate at min(s_in, s_out),
    aggregation first on a tie), as oracle order names; None for SAGE and
    GAT, which always aggregate first."""
    if kind != "gcn":
        return None
    return ["agg" if s[l] <= s[l + 1] else "xform" for l in range(len(s) - 1)]
