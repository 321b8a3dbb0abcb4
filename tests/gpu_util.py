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


def adam_noise(rel, seed):
    """A gradient perturbation for the oracle's Adam runs
    (``oracle.gist.gist_train(..., grad_noise=...)``): each gradient array g
    becomes g + rel * rms(g) * N(0, 1), seeded.  With ``rel`` of the order of
    fp32 rounding in a gradient (relative to its typical entry), the
    perturbed run shows how far rounding alone moves each trained value."""
    rng = np.random.default_rng(seed)

    def f(g):
        g = np.asarray(g, dtype=np.float64)
        if g.size == 0:
            return g
        return g + rel * np.sqrt(np.mean(g * g)) * rng.standard_normal(g.shape)
    return f


def check_adam(got, want, perturbed, tol=FP32_TOL, c=10.0, good=1e-5):
    """Adam-trained values (weight changes, moments) against the oracle's,
    element by element, scaled by the oracle's own sensitivity.

    Adam divides each gradient by the root of its second moment, so an
    element whose gradients are small or cancel moves by an amount that
    rounding in those gradients changes by orders of magnitude more than it
    changes the gradients.  ``perturbed`` are the oracle's values from the
    same run with ``adam_noise`` on every gradient; S_i = max over them of
    |p_i - want_i|.  Elements with S_i <= good * max|want| (well conditioned)
    must agree to ``tol`` of max|want|; every element to
    |got_i - want_i| <= tol * max|want| + c * S_i.
    Returns (worst error on the well-conditioned elements relative to
    max|want|, their fraction, worst ratio of error to bound).
    """
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return 0.0, 1.0, 0.0
    S = np.max([np.abs(np.asarray(p, dtype=np.float64) - want) for p in perturbed], axis=0)
    scale = float(np.max(np.abs(want)))
    E = np.abs(got - want)
    if scale == 0.0:
        return float(np.max(E)), 1.0, float(np.max(E))
    ok = S <= good * scale
    e_good = float(np.max(E[ok]) / scale) if ok.any() else 0.0
    ratio = float(np.max(E / (tol * scale + c * S)))
    return e_good, float(ok.mean()), ratio


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
