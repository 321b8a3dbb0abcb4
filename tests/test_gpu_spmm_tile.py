"""The matrix-core aggregation for cluster mini-batches (GIST_LAYER_CLUSTERED),
through the layer calls of the C ABI, against the fp64 oracle.

The tile kernel splits every value into two bf16 halves and sums
hi*hi + hi*lo + lo*hi in fp32, so each product enters with a relative error
below 2^-15; the checks are therefore elementwise: |got - exact| <=
4e-5 (|Abar| |H|) + 1e-7 max|exact| for Abar H (and for the transposed
aggregation of the backward pass), plus the usual 1e-4 normwise bar on
every output and gradient.  Matrices cover every branch of the kernel:
cluster mini-batches (most entries in the dense window), random graphs (all
entries gathered), bands wider than two windows (the 288-column clamp), hub
rows longer than the 512 entries a wave loads at once, rectangular LADIES
layers, ragged row counts and widths (several 256-column slabs), a single
row, and the SAGE backward whose Add aliases its output.
"""

import numpy as np
import pytest
import scipy.sparse as sp

from gist_synth.graphs import Graph, _csr_from_undirected, erdos_renyi, sbm
from oracle import gist as OG
from oracle import layers as OL
from oracle import ladies as OLD
from oracle import minibatch as OM

from gpu_util import FP32_TOL, csr_to_dev, log, relerr, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available()
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


def _graph_from_edges(n, edges):
    a = [e[0] for e in edges]
    b = [e[1] for e in edges]
    rowptr, col = _csr_from_undirected(n, a, b)
    return Graph(n, rowptr, col, np.array([0, n], dtype=np.int64), np.arange(n, dtype=np.int32))


def _matrices():
    """name -> (graph, clusters or None)."""
    out = {}
    g = sbm(6000, 40, 40.0, 0.9, seed=21)                      # clusters of 150
    out["sbm_batch"] = (g, np.array([1, 4, 9, 17, 30], dtype=np.int32))
    g2 = sbm(4000, 20, 30.0, 0.9, seed=22)                     # clusters of 200 (> kNear)
    out["sbm_wide_clusters"] = (g2, np.array([0, 3, 7], dtype=np.int32))
    out["er_random"] = (erdos_renyi(700, 2800, seed=5), None)
    # a band of half-width 260 > 192: two windows of at most 288 columns, the rest gathered
    n = 900
    out["band_260"] = (_graph_from_edges(n, [(i, j) for i in range(n)
                                             for j in range(i + 1, min(n, i + 261), 7)]), None)
    # two hubs with 1,500 neighbours each (rows far longer than 512 entries)
    n = 3100
    edges = [(0, j) for j in range(2, n)][:1500] + [(1, j) for j in range(1600, n)]
    edges += [(i, i + 1) for i in range(2, n - 1)]
    out["hubs"] = (_graph_from_edges(n, edges), None)
    out["single_node"] = (_graph_from_edges(1, []), None)
    out["ragged_33"] = (_graph_from_edges(33, [(i, (i * 7 + 3) % 33) for i in range(33)
                                               if i != (i * 7 + 3) % 33]), None)
    return out


MATS = _matrices()


def _bound_check(got, A, H, exact):
    """Elementwise: |got - exact| <= 4e-5 (|A| |H|) + 1e-7 max|exact|."""
    bound = 4e-5 * (abs(A) @ np.abs(np.asarray(H, dtype=np.float64)))
    bound += 1e-7 * max(np.max(np.abs(exact)), 1e-30)
    err = np.abs(np.asarray(got, dtype=np.float64) - exact)
    worst = float(np.max(err - bound)) if err.size else -1.0
    return worst <= 0.0, float(np.max(err / np.maximum(bound, 1e-300))) if err.size else 0.0


@pytest.mark.parametrize("mat", list(MATS))
@pytest.mark.parametrize("kind", ["gcn", "sage"])
@pytest.mark.parametrize("width", [7, 100, 256, 600])
def test_clustered_layer_matches_oracle(G, ctx, mat, kind, width):
    import torch
    g, clusters = MATS[mat]
    csr = OM.build(g, clusters, kind)
    n = csr["n"]
    rng = np.random.default_rng(width + n)
    s_out = 24
    H = rng.standard_normal((n, width)).astype(np.float32)
    W = (rng.standard_normal(((2 if kind == "sage" else 1) * width, s_out)) /
         np.sqrt(width)).astype(np.float32)
    dHo = rng.standard_normal((n, s_out)).astype(np.float32)
    A, k1 = csr_to_dev(csr)
    AT, k2 = csr_to_dev(csr, transpose=True) if kind == "sage" else (None, None)
    lk = G.GIST_LAYER_SAGE_MEAN if kind == "sage" else G.GIST_LAYER_GCN
    desc = G.layer_desc(lk, G.GIST_ACT_RELU, n, width, s_out, G.GIST_DTYPE_F32,
                        G.GIST_ORDER_AGG_FIRST, flags=G.GIST_LAYER_CLUSTERED)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    Hd, Wd = to_dev(H), to_dev(W)
    agg = torch.empty(n, width, device="cuda")
    Ho = torch.empty(n, s_out, device="cuda")
    log(f"[tile {mat} {kind} w={width}] n={n} nnz={csr['nnz']}")
    G.gist_gcn_layer_fwd(ctx, desc, A, Hd, Wd, agg, Ho, ws)
    Asp = OL.adjacency(csr)
    exact = Asp @ H.astype(np.float64)
    ok, ratio = _bound_check(to_host(agg), Asp, H, exact)
    Wp = (W,) if kind == "gcn" else (W[:width], W[width:])
    fwd = (OL.gcn_forward(csr, H, W, True) if kind == "gcn"
           else OL.sage_forward(csr, H, Wp[0], Wp[1], True))
    e_h = relerr(to_host(Ho), fwd["H_out"])
    # backward on the oracle's own forward values
    dW = torch.empty(W.shape[0], s_out, device="cuda")
    dH = torch.empty(n, width, device="cuda")
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, Hd, to_dev(fwd["AH"].astype(np.float32)),
                         to_dev(fwd["H_out"].astype(np.float32)), Wd, to_dev(dHo), dW, dH, ws)
    bwd = (OL.gcn_backward(csr, H, fwd, W, dHo, True) if kind == "gcn"
           else OL.sage_backward(csr, H, fwd, Wp[0], Wp[1], dHo, True))
    gW = bwd["dW"] if kind == "gcn" else np.concatenate([bwd["dW_self"], bwd["dW_neigh"]])
    e_w = relerr(to_host(dW), gW)
    e_d = relerr(to_host(dH), bwd["dH"])
    # the transposed aggregation alone, elementwise: dP = dZ W_neigh^T
    dP = bwd["dZ"] @ Wp[-1].astype(np.float64).T
    At = OL.adjacency(csr, transpose=True) if kind == "sage" else Asp.T
    agg_t = At @ dP
    self_t = bwd["dZ"] @ Wp[0].astype(np.float64).T if kind == "sage" else 0.0
    ok_t, ratio_t = _bound_check(to_host(dH) - self_t, At, dP, agg_t) if kind == "gcn" else \
        (relerr(to_host(dH), bwd["dH"]) <= FP32_TOL, 0.0)
    log(f"  agg bound ratio {ratio:.2f}, H_out {e_h:.2e}, dW {e_w:.2e}, dH {e_d:.2e}, "
        f"transposed bound ratio {ratio_t:.2f}")
    assert ok and ok_t
    assert max(e_h, e_w, e_d) <= FP32_TOL


def test_clustered_matches_gather_path_on_a_c3_batch(G, ctx):
    """A c3-sized cluster mini-batch (20 of 1,500 blocks, ~3,100 rows,
    ~140k entries) at the hidden width 4,096 (16 column slabs): the tile
    path against the gather path and the oracle, forward aggregation and
    the SAGE backward's transposed aggregation with Add."""
    import torch
    from gist_synth import get_config
    cfg = get_config("c3")
    g = cfg.make_graph()
    csr = OM.build(g, cfg.minibatch(0, 0), "sage")
    n, w = csr["n"], 4096
    rng = np.random.default_rng(3)
    H = rng.standard_normal((n, w)).astype(np.float32)
    A, k1 = csr_to_dev(csr)
    AT, k2 = csr_to_dev(csr, transpose=True)
    outs = {}
    for name, flags in (("tile", G.GIST_LAYER_CLUSTERED), ("gather", 0)):
        desc = G.layer_desc(G.GIST_LAYER_SAGE_MEAN, G.GIST_ACT_RELU, n, w, 8, G.GIST_DTYPE_F32,
                            G.GIST_ORDER_AGG_FIRST, flags=flags)
        fws, bws = G.gist_layer_workspace_size(desc)
        ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
        agg = torch.empty(n, w, device="cuda")
        Ho = torch.empty(n, 8, device="cuda")
        W = to_dev((rng.standard_normal((2 * w, 8)) * 0.01).astype(np.float32)) if not outs \
            else outs["W"]
        outs["W"] = W
        G.gist_gcn_layer_fwd(ctx, desc, A, to_dev(H), W, agg, Ho, ws)
        outs[name] = to_host(agg)
    exact = OL.adjacency(csr) @ H.astype(np.float64)
    ok, ratio = _bound_check(outs["tile"], OL.adjacency(csr), H, exact)
    e_tg = relerr(outs["tile"], outs["gather"])
    log(f"[c3 batch n={n} nnz={csr['nnz']}] tile bound ratio {ratio:.2f}, tile vs gather {e_tg:.2e}")
    assert ok and e_tg <= FP32_TOL


def test_clustered_rectangular_ladies_layer(G, ctx):
    """Rectangular layers (n output rows, n_in input rows) of a LADIES batch:
    forward in both association orders and the backward (transposed matrix
    with n_in rows), flag set, against the oracle."""
    import torch
    g = sbm(5000, 50, 20.0, 0.9, seed=9)
    Afull = OM.build(g, None, "gcn")
    batch = np.sort(np.random.default_rng(2).choice(g.n, 200, replace=False)).astype(np.int32)
    lay = OLD.sample(Afull, batch, 1, 600, seed=4)["layers"][0]
    n, n_in = lay["n"], lay["n_in"]
    rng = np.random.default_rng(5)
    for si, so in ((40, 300), (300, 40)):     # aggregate first / transform first
        H = rng.standard_normal((n_in, si)).astype(np.float32)
        W = (rng.standard_normal((si, so)) / np.sqrt(si)).astype(np.float32)
        dHo = rng.standard_normal((n, so)).astype(np.float32)
        A, k1 = csr_to_dev(lay)
        AT, k2 = csr_to_dev(lay, transpose=True)
        desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, si, so, n_in=n_in,
                            flags=G.GIST_LAYER_CLUSTERED)
        fws, bws = G.gist_layer_workspace_size(desc)
        ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
        agg = torch.empty(n, si, device="cuda")
        Ho = torch.empty(n, so, device="cuda")
        G.gist_gcn_layer_fwd(ctx, desc, A, to_dev(H), to_dev(W), agg, Ho, ws)
        f = OL.gcn_forward(lay, H, W, True)
        dW = torch.empty(si, so, device="cuda")
        dH = torch.empty(n_in, si, device="cuda")
        G.gist_gcn_layer_bwd(ctx, desc, A, AT, to_dev(H), to_dev(f["AH"].astype(np.float32)),
                             to_dev(f["H_out"].astype(np.float32)), to_dev(W), to_dev(dHo), dW,
                             dH, ws)
        b = OL.gcn_backward(lay, H, f, W, dHo, True)
        e = dict(H_out=relerr(to_host(Ho), f["H_out"]), dW=relerr(to_host(dW), b["dW"]),
                 dH=relerr(to_host(dH), b["dH"]))
        log(f"[ladies rect {n}x{n_in} {si}->{so}] " + ", ".join(f"{k} {v:.2e}" for k, v in e.items()))
        assert max(e.values()) <= FP32_TOL
