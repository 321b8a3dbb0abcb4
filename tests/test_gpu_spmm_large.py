"""Aggregation on graphs larger than the mini-batches (140,000 nodes, above
2^17 rows) against the fp64 oracle on every row, elementwise per row as
well as normwise: the GCN forward aggregation on a clustered graph at
widths that fill one 64-lane column tile, leave a ragged tile and span
several, and on a cluster-free (Erdos-Renyi) graph; and the SAGE backward
dH = dZ W_self^T + Abar^T (dZ W_neigh^T), whose transposed aggregation adds
the self term (already in dH: the Add operand aliases the output) inside the
kernel."""

import numpy as np
import pytest

from gist_synth.graphs import erdos_renyi, sbm
from oracle import layers as OL
from oracle import minibatch as MB

from gpu_util import FP32_TOL, csr_to_dev, log, relerr, to_dev, to_host

pytestmark = pytest.mark.gpu

_G = {}


def graph(kind):
    if kind not in _G:
        _G[kind] = (sbm(140_000, 1000, 20.0, 0.9, 11) if kind == "sbm"
                    else erdos_renyi(140_000, 700_000, 12))
    return _G[kind]


@pytest.fixture(scope="module")
def G():
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


@pytest.mark.parametrize("gname,width", [("sbm", 64), ("sbm", 130), ("sbm", 384), ("er", 128)])
def test_band_forward_aggregation(G, ctx, gname, width):
    import torch
    g = graph(gname)
    csr = MB.build(g, None, "gcn")
    n = csr["n"]
    assert n >= 1 << 17
    rng = np.random.default_rng(width)
    H = rng.standard_normal((n, width)).astype(np.float32)
    W = (rng.standard_normal((width, width + 8)) / np.sqrt(width)).astype(np.float32)
    log(f"band forward {gname} n={n} nnz={csr['nnz']} width={width}")
    ref = OL.gcn_forward(csr, H, W, True)
    A, keep = csr_to_dev(csr)
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, width, width + 8,
                        G.GIST_DTYPE_F32, G.GIST_ORDER_AGG_FIRST)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    agg = torch.empty(n, width, device="cuda")
    Ho = torch.empty(n, width + 8, device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, to_dev(H), to_dev(W), agg, Ho, ws)
    got = to_host(agg)
    e = relerr(got, ref["AH"])
    # every row, elementwise, not only normwise
    scale = np.max(np.abs(ref["AH"]), axis=1, keepdims=True) + 1e-30
    e_row = float(np.max(np.abs(got - ref["AH"]) / scale))
    log(f"  agg {e:.2e} (worst row {e_row:.2e}), H_out {relerr(to_host(Ho), ref['H_out']):.2e}")
    assert e <= FP32_TOL and e_row <= FP32_TOL
    assert relerr(to_host(Ho), ref["H_out"]) <= FP32_TOL


def test_band_sage_backward_with_add(G, ctx):
    import torch
    g = graph("sbm")
    csr = MB.build(g, None, "sage")
    n, si, so = csr["n"], 130, 96
    rng = np.random.default_rng(3)
    H = rng.standard_normal((n, si)).astype(np.float32)
    Ws = (rng.standard_normal((si, so)) / np.sqrt(si)).astype(np.float32)
    Wn = (rng.standard_normal((si, so)) / np.sqrt(si)).astype(np.float32)
    dHo = rng.standard_normal((n, so)).astype(np.float32)
    log(f"band SAGE backward n={n} nnz={csr['nnz']} {si}->{so}")
    f = OL.sage_forward(csr, H, Ws, Wn, True)
    b = OL.sage_backward(csr, H, f, Ws, Wn, dHo, True)
    A, k1 = csr_to_dev(csr)
    AT, k2 = csr_to_dev(csr, transpose=True)
    desc = G.layer_desc(G.GIST_LAYER_SAGE_MEAN, G.GIST_ACT_RELU, n, si, so)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    dW = torch.empty(2 * si, so, device="cuda")
    dH = torch.empty(n, si, device="cuda")
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, to_dev(H), to_dev(f["AH"].astype(np.float32)),
                         to_dev(f["H_out"].astype(np.float32)), to_dev(np.concatenate([Ws, Wn])),
                         to_dev(dHo), dW, dH, ws)
    e = relerr(to_host(dH), b["dH"])
    ew = relerr(to_host(dW), np.concatenate([b["dW_self"], b["dW_neigh"]]))
    log(f"  dH {e:.2e} dW {ew:.2e}")
    assert e <= FP32_TOL and ew <= FP32_TOL
