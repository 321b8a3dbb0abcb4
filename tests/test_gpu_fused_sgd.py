"""gist_gcn_layer_bwd_sgd: the backward pass with subTrain's SGD step fused
into the weight-gradient GEMM's epilogue.  Its updated weights and input
gradient must be bitwise those of gist_gcn_layer_bwd followed by
gist_sgd_update (the epilogue applies the same fmaf to the same fp32 sum),
for every GEMM path the weight gradient can take: direct tiles and stream-K
partial tiles with their fix-up, node-contiguous copies of the operands
(large fp32 dW), grouped sub-GCNs, rectangular layers, transform-first GCN,
and the bf16-input kernels (packed and in-kernel rounding).  The plain path
is held against the fp64 oracle elsewhere; one case here also checks the
step itself against the oracle's SGD."""

import numpy as np
import pytest

from gist_synth.graphs import chung_lu, sbm
from oracle import layers as OL
from oracle import minibatch as MB

from gpu_util import csr_to_dev, log, relerr, to_dev, to_host

pytestmark = pytest.mark.gpu

LR = 0.05


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


_CSR = {}


def square_csr(name, norm):
    key = (name, norm)
    if key not in _CSR:
        g = sbm(1500, 10, 30.0, 0.9, seed=7) if name == "sbm1500" else \
            sbm(1100, 8, 20.0, 0.9, seed=8) if name == "sbm1100" else \
            chung_lu(2000, 2.5, 5.0, seed=6)
        _CSR[key] = MB.build(g, None, norm)
    return _CSR[key]


def rect_csr(n, n_in, seed):
    """A layer-sampled shape: n output rows over n_in input rows (+ transpose)."""
    rng = np.random.default_rng(seed)
    rows = [np.sort(rng.choice(n_in, size=int(rng.integers(0, 12)), replace=False))
            for _ in range(n)]
    rowptr = np.zeros(n + 1, np.int64)
    rowptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.concatenate(rows).astype(np.int64)
    val = rng.uniform(0.05, 1.0, col.size).astype(np.float32)
    rid = np.repeat(np.arange(n), np.diff(rowptr))
    order = np.lexsort((rid, col))
    t_rowptr = np.zeros(n_in + 1, np.int64)
    np.add.at(t_rowptr, col + 1, 1)
    return dict(n=n, n_in=n_in, nnz=int(col.size), rowptr=rowptr.astype(np.int32),
                col=col.astype(np.int32), val=val, t_rowptr=np.cumsum(t_rowptr).astype(np.int32),
                t_col=rid[order].astype(np.int32), t_val=val[order])


def run_pair(G, ctx, kind, csr, s_in, s_out, order, dtype, groups=1, need_dH=True, seed=0):
    """Backward + SGD and the fused backward on the same inputs; returns
    (W after the separate step, dH, W after the fused step, dH, inputs)."""
    import torch
    n, n_in = csr["n"], csr.get("n_in", csr["n"])
    rng = np.random.default_rng(seed)
    parts = 2 if kind == "sage" else 1
    H = to_dev(rng.standard_normal((n_in, groups * s_in)).astype(np.float32))
    W0 = (rng.standard_normal((groups, parts * s_in, s_out)) / np.sqrt(s_in)).astype(np.float32)
    dHo = to_dev(rng.standard_normal((n, groups * s_out)).astype(np.float32))
    A, k1 = csr_to_dev(csr)
    AT, k2 = csr_to_dev(csr, transpose=True) if "t_rowptr" in csr else (None, None)
    lk = G.GIST_LAYER_SAGE_MEAN if kind == "sage" else G.GIST_LAYER_GCN
    desc = G.layer_desc(lk, G.GIST_ACT_RELU, n, s_in, s_out, dtype, order, groups=groups,
                        n_in=n_in if n_in != n else 0)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    W = to_dev(W0)
    agg = torch.empty(n, groups * s_in, device="cuda")
    Ho = torch.empty(n, groups * s_out, device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, H, W, agg, Ho, ws)
    # separate: gradient, then the SGD step
    dW = torch.empty_like(W)
    dH1 = torch.empty(n_in, groups * s_in, device="cuda") if need_dH else None
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, H, agg, Ho, W, dHo, dW, dH1, ws)
    Wa = W.clone()
    G.gist_sgd_update(ctx, Wa, dW, Wa.numel(), LR)
    # fused
    Wb = W.clone()
    dH2 = torch.empty(n_in, groups * s_in, device="cuda") if need_dH else None
    G.gist_gcn_layer_bwd_sgd(ctx, desc, A, AT, H, agg, Ho, Wb, dHo, LR, dH2, ws)
    out = (to_host(Wa), to_host(dH1) if need_dH else None, to_host(Wb),
           to_host(dH2) if need_dH else None)
    return out, dict(W=W0, dW=to_host(dW))


def same(a, b):
    return np.array_equal(np.asarray(a).view(np.uint32), np.asarray(b).view(np.uint32))


CASES = [
    # kind, graph, s_in, s_out, order, dtype, groups
    ("gcn", "sbm1500", 100, 256, "agg", "f32", 1),     # dW 100 x 256 over K = 1500: stream-K
    ("gcn", "cl2000", 300, 64, "xform", "f32", 1),     # transform-first
    ("sage", "sbm1500", 128, 96, "agg", "f32", 1),
    ("sage", "sbm1100", 1024, 1024, "agg", "f32", 1),  # node-contiguous dW operands
    ("gcn", "sbm1500", 64, 48, "agg", "f32", 3),       # grouped sub-GCNs
    ("sage", "sbm1500", 512, 512, "agg", "bf16", 1),   # packed bf16 kernel
    ("sage", "sbm1500", 1024, 1024, "agg", "bf16", 1),  # 2048 x 1024 dW, rows of 1500 nodes
    ("gcn", "sbm1500", 100, 64, "agg", "bf16", 1),     # bf16 rounding in the fp32 tiles
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[1]}-{c[2]}x{c[3]}-{c[4]}-{c[5]}-g{c[6]}"
                                             for c in CASES])
def test_fused_sgd_is_bitwise(G, ctx, case):
    kind, gname, si, so, order, dt, groups = case
    csr = square_csr(gname, "sage" if kind == "sage" else "gcn")
    o = G.GIST_ORDER_AGG_FIRST if order == "agg" else G.GIST_ORDER_XFORM_FIRST
    d = G.GIST_DTYPE_BF16_IN if dt == "bf16" else G.GIST_DTYPE_F32
    log(f"fused SGD {case} n={csr['n']}")
    (Wa, dHa, Wb, dHb), _ = run_pair(G, ctx, kind, csr, si, so, o, d, groups)
    assert same(Wa, Wb), "W"
    assert same(dHa, dHb), "dH"
    assert not np.array_equal(Wa, _["W"])   # the step moved the weights


def test_fused_sgd_rectangular_and_layer0(G, ctx):
    csr = rect_csr(500, 1300, 4)
    (Wa, dHa, Wb, dHb), _ = run_pair(G, ctx, "gcn", csr, 96, 80, G.GIST_ORDER_AUTO,
                                     G.GIST_DTYPE_F32)
    assert same(Wa, Wb) and same(dHa, dHb)
    (Wa, _n, Wb, _m), _ = run_pair(G, ctx, "gcn", csr, 96, 80, G.GIST_ORDER_AUTO,
                                   G.GIST_DTYPE_F32, need_dH=False)
    assert same(Wa, Wb)


def test_fused_sgd_matches_the_oracle_step(G, ctx):
    csr = square_csr("sbm1500", "gcn")
    (Wa, dHa, Wb, dHb), inp = run_pair(G, ctx, "gcn", csr, 100, 256, G.GIST_ORDER_AGG_FIRST,
                                       G.GIST_DTYPE_F32)
    # the step is exactly fmaf(-lr, dW, W) of the fp32 gradient the GEMM formed
    want = OL.sgd(inp["W"], inp["dW"], np.float32(LR)).astype(np.float32)
    e = relerr(Wb, want)
    log(f"  W vs oracle SGD of the same gradient {e:.2e}")
    assert e <= 1e-6


def test_fused_sgd_empty_batch_and_errors(G, ctx):
    import torch
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, 0, 8, 4)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    rp = torch.zeros(1, dtype=torch.int32, device="cuda")
    A = G.csr_dev(0, 0, rp, rp, rp.float())
    W = torch.randn(8, 4, device="cuda")
    W0 = W.clone()
    G.gist_gcn_layer_bwd_sgd(ctx, desc, A, None, None, None, None, W, None, LR, None, ws)
    assert torch.equal(W, W0)   # no output rows: a zero gradient leaves W unchanged
    with pytest.raises(G.GistError, match="lr"):
        G.gist_gcn_layer_bwd_sgd(ctx, desc, A, None, None, None, None, W, None, float("nan"),
                                 None, ws)
    with pytest.raises(G.GistError, match="NULL"):
        G.gist_gcn_layer_bwd_sgd(ctx, desc, A, None, None, None, None, None, None, LR, None, ws)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", ["sage", "gcn"])
def test_subgcn_step_takes_the_fused_path_bitwise(G, ctx, kind, dtype):
    """SubGCN.step fuses the SGD step into each GCN / SAGE layer's backward
    pass, in fp32 and with bf16-input GEMMs; the weights must equal an
    explicit backward + SGD."""
    import torch
    from paper_2102_10424_amd.step import BatchSlot, SubGCN
    g = sbm(1500, 10, 30.0, 0.9, seed=7)
    widths = [40, 512, 512, 7]
    parts = 2 if kind == "sage" else 1
    rng = np.random.default_rng(11)
    X = to_dev(rng.standard_normal((g.n, widths[0])).astype(np.float32))
    y = rng.integers(0, widths[-1], g.n).astype(np.int32)
    P = [(rng.standard_normal((parts * widths[l], widths[l + 1])) /
          np.sqrt(widths[l])).astype(np.float32) for l in range(3)]
    slot = BatchSlot(ctx, kind, g.n, g.nnz + g.n, widths[0])
    b = slot.load(G.GraphHandle(g), np.array([0, 3, 5, 8], dtype=np.int32), X, y)
    out = []
    for fused in (True, False):
        run = SubGCN(ctx, kind, widths, b.n,
                     dtype=G.GIST_DTYPE_BF16_IN if dtype == "bf16" else G.GIST_DTYPE_F32)
        params = [to_dev(p) for p in P]
        if fused:
            run.step(b, params, LR)
        else:
            run.forward(b, params)
            run.loss_and_grad(b)
            run.backward(b, params)
            run.sgd(params, LR)
        torch.cuda.synchronize()
        out.append([to_host(p) for p in params])
    for l, (a, c) in enumerate(zip(*out)):
        log(f"  {kind} layer {l}: {'bitwise equal' if same(a, c) else 'DIFFERENT'}")
        assert same(a, c), l
        assert not np.array_equal(a, P[l])
