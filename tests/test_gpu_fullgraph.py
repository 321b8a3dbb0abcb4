"""Full-graph GCN layer (c5): 2,449,029 nodes, ~126M stored entries, fp32.

Run at full size in the bench's launch configuration and checked on
sampled outputs the oracle computes one by one:

* forward: 1,024 random rows (plus the first and last row and the longest
  row) of Abar H and of H_out = ReLU(Abar H W);
* backward, fed seeded inputs (the backward is a function of H, Abar H,
  H_out, W and dH_out alone, so they need not come from a forward pass):
  dW in full (every entry, the reduction over all 2.45M rows streamed in
  row chunks in fp64), and 1,024 sampled rows of dH, for input widths 100
  and 256 (aggregate first) and 512 (transform first).
"""

import numpy as np
import pytest
import scipy.sparse as sp

from gist_synth import get_config
from gist_synth.tensors import normal_rows
from oracle import minibatch as OM

from gpu_util import FP32_TOL, log, relerr, to_dev, to_host

pytestmark = pytest.mark.gpu

_G = {}


def graph_and_csr():
    if "g" not in _G:
        cfg = get_config("c5")
        log("[c5] generating graph")
        g = cfg.make_graph()
        log("[c5] oracle CSR")
        _G["g"] = g
        _G["csr"] = OM.build(g, None, "gcn")
    return _G["g"], _G["csr"]


def tdot(a32, b, chunk=1 << 18):
    """a^T b in fp64, accumulated over row chunks (keeps fp64 copies small);
    b is an array or a function of a row range giving that chunk of b."""
    get = b if callable(b) else (lambda i, j: b[i:j])
    out = None
    for i in range(0, a32.shape[0], chunk):
        j = min(i + chunk, a32.shape[0])
        part = a32[i:j].astype(np.float64).T @ np.asarray(get(i, j), dtype=np.float64)
        out = part if out is None else out + part
    return out


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available()
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


@pytest.mark.parametrize("d_in", [100, 256, 512])
def test_full_graph_layer(G, ctx, d_in):
    import torch
    g, csr = graph_and_csr()
    n, nnz = csr["n"], csr["nnz"]
    cfg = get_config("c5", widths=[d_in, 2048])
    s_out = 256
    rng = np.random.default_rng(d_in)
    log(f"[c5 d_in={d_in}] inputs")
    X = cfg.features_matrix()
    W = (rng.standard_normal((d_in, s_out)) / np.sqrt(d_in)).astype(np.float32)
    dHo = cfg.upstream(n, s_out)
    Zs = normal_rows((n, s_out), cfg.seed, 91, s_out)
    Hout_in = np.maximum(Zs, 0.0)               # a valid post-ReLU tensor
    del Zs
    A_sp = sp.csr_matrix((csr["val"].astype(np.float64), csr["col"], csr["rowptr"]),
                         shape=(n, n))
    # device side
    rp = to_dev(csr["rowptr"].astype(np.int32))
    col = to_dev(csr["col"])
    val = to_dev(csr["val"])
    A = G.csr_dev(n, nnz, rp, col, val)
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, d_in, s_out)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    Xd, Wd = to_dev(X), to_dev(W)
    agg = torch.empty(n, d_in, device="cuda")
    Ho = torch.empty(n, s_out, device="cuda")
    log(f"[c5 d_in={d_in}] forward")
    G.gist_gcn_layer_fwd(ctx, desc, A, Xd, Wd, agg, Ho, ws)
    deg = np.diff(csr["rowptr"])
    S = np.unique(np.concatenate([rng.choice(n, 1024, replace=False),
                                  [0, n - 1, int(np.argmax(deg))]]))
    AS = A_sp[S]
    cS = np.unique(AS.indices)
    AH_S = AS[:, cS] @ X[cS].astype(np.float64)
    Z_S = AH_S @ W.astype(np.float64)
    e_h = relerr(to_host(Ho)[S], np.maximum(Z_S, 0.0))
    agg_first = d_in <= s_out
    e_a = relerr(to_host(agg)[S], AH_S) if agg_first else 0.0
    log(f"[c5 d_in={d_in}] forward rows: H_out {e_h:.2e} agg {e_a:.2e}")
    assert e_h <= FP32_TOL and e_a <= FP32_TOL
    # backward on seeded inputs
    agg_in = normal_rows((n, d_in), cfg.seed, 92, d_in) if agg_first else None
    dW = torch.empty(d_in, s_out, device="cuda")
    dH = torch.empty(n, d_in, device="cuda")
    log(f"[c5 d_in={d_in}] backward")
    G.gist_gcn_layer_bwd(ctx, desc, A, None, Xd, to_dev(agg_in) if agg_first else agg,
                         to_dev(Hout_in), Wd, to_dev(dHo), dW, dH, ws)
    dW_h = to_host(dW)
    dH_h = to_host(dH)
    dZ_rows = lambda i, j: dHo[i:j].astype(np.float64) * (Hout_in[i:j] > 0)
    log(f"[c5 d_in={d_in}] oracle dW over all rows")
    if agg_first:
        want_dW = tdot(agg_in, dZ_rows)              # (Abar H)^T dZ
    else:                                            # H^T (Abar^T dZ) = (Abar H)^T dZ
        T = np.empty((n, s_out))
        for c in range(0, s_out, 64):
            dZc = dHo[:, c:c + 64].astype(np.float64) * (Hout_in[:, c:c + 64] > 0)
            T[:, c:c + 64] = A_sp.T @ dZc
            del dZc
        want_dW = tdot(X, T)
        del T
    e_w = relerr(dW_h, want_dW)
    # dH rows: Abar^T (dZ W^T) restricted to rows S
    AT_S = A_sp[:, S].T.tocsr()                 # rows S of Abar^T
    nb = np.unique(AT_S.indices)                # the rows of dP they read
    dZ_nb = dHo[nb].astype(np.float64) * (Hout_in[nb] > 0)
    want_dH = AT_S[:, nb] @ (dZ_nb @ W.astype(np.float64).T)
    e_d = relerr(dH_h[S], want_dH)
    log(f"[c5 d_in={d_in}] backward: dW (all entries) {e_w:.2e} dH rows {e_d:.2e}")
    assert e_w <= FP32_TOL and e_d <= FP32_TOL
