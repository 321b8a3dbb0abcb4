"""The ReLU derivative fused into the producer of the gradient it multiplies
(GIST_LAYER_MASK_DH, GIST_LAYER_DZ_IN), bitwise against the unflagged calls.

* MASK_DH: the backward pass writes dH * 1[H > 0] -- bitwise the plain call's
  dH with every entry whose H <= 0 set to +0 (the select the separate
  ReLU-derivative pass makes) -- through each kernel that can write dH: the
  transposed aggregation (GCN aggregate-first, SAGE with its Add, gather and
  matrix-core paths), the dH product of a transform-first GCN layer (fp32
  stream-K tiles with fix-up, the bf16 kernels), grouped sub-GCNs and
  rectangular layers; also through the fused-SGD entry point.
* DZ_IN: a hidden layer handed dZ = dH_out * 1[H_out > 0] with H_out = NULL
  gives bitwise the dW and dH of the plain call with dH_out and H_out.
* A whole SubGCN step with the fused chain (its default) runs no
  relu_mask launch.
"""

import numpy as np
import pytest

from gist_synth.graphs import sbm

from gpu_util import csr_to_dev, log, to_dev, to_host
from test_gpu_fused_sgd import rect_csr, same, square_csr

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


CASES = [
    # kind, graph, s_in, s_out, order, dtype, groups, extra flags
    ("gcn", "sbm1500", 100, 256, "agg", "f32", 1, 0),
    ("gcn", "cl2000", 300, 64, "xform", "f32", 1, 0),      # dH from the GEMM
    ("gcn", "sbm1500", 700, 96, "xform", "f32", 1, 0),     # stream-K dH product + fix-up
    ("sage", "sbm1500", 128, 96, "agg", "f32", 1, 0),      # Add aliases the output
    ("sage", "sbm1100", 1024, 1024, "agg", "f32", 1, 0),
    ("gcn", "sbm1500", 64, 48, "agg", "f32", 3, 0),        # grouped, aggregate first
    ("gcn", "sbm1500", 96, 32, "xform", "f32", 3, 0),      # grouped, transform first
    ("sage", "sbm1500", 512, 512, "agg", "bf16", 1, 0),
    ("gcn", "cl2000", 1024, 512, "xform", "bf16", 1, 0),   # packed bf16 dH product
    ("gcn", "sbm1500", 100, 64, "agg", "bf16", 1, 0),
    ("sage", "sbm1500", 128, 96, "agg", "f32", 1, 4),      # matrix-core aggregation
    ("gcn", "rect", 80, 40, "xform", "f32", 1, 0),         # rectangular (layer-sampled)
    ("gcn", "rect", 40, 80, "agg", "f32", 1, 0),
]


def _setup(G, kind, graph, s_in, s_out, order, dtype, groups, extra, seed):
    import torch
    csr = rect_csr(300, 700, 5) if graph == "rect" else \
        square_csr(graph, "sage" if kind == "sage" else "gcn")
    n, n_in = csr["n"], csr.get("n_in", csr["n"])
    rng = np.random.default_rng(seed)
    parts = 2 if kind == "sage" else 1
    t = dict(csr=csr, n=n, n_in=n_in)
    # H: a post-ReLU input (about half its entries zero), as the layer below leaves it
    t["H"] = to_dev(np.maximum(rng.standard_normal((n_in, groups * s_in)), 0).astype(np.float32))
    t["W"] = to_dev((rng.standard_normal((groups, parts * s_in, s_out)) /
                     np.sqrt(s_in)).astype(np.float32))
    t["dHo"] = to_dev(rng.standard_normal((n, groups * s_out)).astype(np.float32))
    t["A"], t["k1"] = csr_to_dev(csr)
    t["AT"], t["k2"] = csr_to_dev(csr, transpose=True) if "t_rowptr" in csr else (None, None)
    lk = G.GIST_LAYER_SAGE_MEAN if kind == "sage" else G.GIST_LAYER_GCN
    o = G.GIST_ORDER_AGG_FIRST if order == "agg" else G.GIST_ORDER_XFORM_FIRST
    dt = G.GIST_DTYPE_BF16_IN if dtype == "bf16" else G.GIST_DTYPE_F32
    t["desc"] = lambda flags: G.layer_desc(lk, G.GIST_ACT_RELU, n, s_in, s_out, dt, o,
                                           groups=groups, flags=flags | extra,
                                           n_in=n_in if n_in != n else 0)
    fws, bws = G.gist_layer_workspace_size(t["desc"](0))
    t["ws"] = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    t["agg"] = torch.empty(n, groups * s_in, device="cuda")
    t["Ho"] = torch.empty(n, groups * s_out, device="cuda")
    G.gist_gcn_layer_fwd(ctx_of(G), t["desc"](0), t["A"], t["H"], t["W"], t["agg"], t["Ho"],
                         t["ws"])
    return t


_CTX = {}


def ctx_of(G):
    if "c" not in _CTX:
        _CTX["c"] = G.Context(0)
    return _CTX["c"]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[1]}-{c[2]}x{c[3]}-{c[4]}-{c[5]}-g{c[6]}"
                                             f"{'-tiles' if c[7] else ''}" for c in CASES])
def test_mask_dh_and_dz_in_are_bitwise(G, case):
    import torch
    kind, graph, s_in, s_out, order, dtype, groups, extra = case
    ctx = ctx_of(G)
    t = _setup(G, kind, graph, s_in, s_out, order, dtype, groups, extra, seed=s_in + s_out)
    n, n_in = t["n"], t["n_in"]
    mk = lambda r, c: torch.full((r, c), float("nan"), device="cuda")
    # plain
    dW0, dH0 = torch.full_like(t["W"], float("nan")), mk(n_in, groups * s_in)
    G.gist_gcn_layer_bwd(ctx, t["desc"](0), t["A"], t["AT"], t["H"], t["agg"], t["Ho"], t["W"],
                         t["dHo"], dW0, dH0, t["ws"])
    # MASK_DH
    dW1, dH1 = torch.empty_like(dW0), mk(n_in, groups * s_in)
    G.gist_gcn_layer_bwd(ctx, t["desc"](G.GIST_LAYER_MASK_DH), t["A"], t["AT"], t["H"],
                         t["agg"], t["Ho"], t["W"], t["dHo"], dW1, dH1, t["ws"])
    H = to_host(t["H"])
    want = np.where(H > 0, to_host(dH0), np.float32(0.0)).astype(np.float32)
    assert same(to_host(dW1), to_host(dW0))
    assert same(to_host(dH1), want)
    # DZ_IN: the masked upstream gradient, no H_out
    dZ = to_dev(np.where(to_host(t["Ho"]) > 0, to_host(t["dHo"]),
                         np.float32(0.0)).astype(np.float32))
    dW2, dH2 = torch.empty_like(dW0), mk(n_in, groups * s_in)
    G.gist_gcn_layer_bwd(ctx, t["desc"](G.GIST_LAYER_DZ_IN), t["A"], t["AT"], t["H"], t["agg"],
                         None, t["W"], dZ, dW2, dH2, t["ws"])
    assert same(to_host(dW2), to_host(dW0)) and same(to_host(dH2), to_host(dH0))
    # both, through the fused-SGD entry point
    Wa = t["W"].clone()
    G.gist_sgd_update(ctx, Wa, dW0, Wa.numel(), 0.05)
    Wb = t["W"].clone()
    dH3 = mk(n_in, groups * s_in)
    G.gist_gcn_layer_bwd_sgd(ctx, t["desc"](G.GIST_LAYER_DZ_IN | G.GIST_LAYER_MASK_DH), t["A"],
                             t["AT"], t["H"], t["agg"], None, Wb, dZ, 0.05, dH3, t["ws"])
    assert same(to_host(Wb), to_host(Wa)) and same(to_host(dH3), want)
    log(f"{case}: MASK_DH / DZ_IN bitwise; {int((H <= 0).sum())} entries masked")


def test_subgcn_step_runs_no_relu_mask_pass(G):
    """A 4-layer SAGE and a 3-layer GCN sub-GCN step, fp32 and bf16: the
    library's launch record lists no relu_mask kernel, and the fused chain's
    weights after the step equal a chain of unflagged calls with the separate
    derivative pass, bit for bit."""
    import torch
    from paper_2102_10424_amd import step as S
    ctx = ctx_of(G)
    g = sbm(1500, 10, 30.0, 0.9, seed=7)
    for kind, widths in (("sage", [40, 96, 64, 80, 7]), ("gcn", [40, 200, 64, 7])):
        for dt in (G.GIST_DTYPE_F32, G.GIST_DTYPE_BF16_IN):
            rng = np.random.default_rng(1)
            X = rng.standard_normal((g.n, widths[0])).astype(np.float32)
            y = rng.integers(0, widths[-1], g.n).astype(np.int32)
            parts = 2 if kind == "sage" else 1
            theta = [(rng.standard_normal((parts * widths[l], widths[l + 1])) * 0.3)
                     .astype(np.float32) for l in range(len(widths) - 1)]
            slot = S.BatchSlot(ctx, kind if kind == "sage" else "gcn", g.n, g.nnz + g.n,
                               widths[0])
            b = slot.load(G.GraphHandle(g), np.array([0, 3, 5], np.int32), to_dev(X), y)
            run = S.SubGCN(ctx, kind, widths, b.n, dtype=dt)
            p1 = [to_dev(t.copy()) for t in theta]
            G.gist_profile_begin(ctx, 4096)
            run.step(b, p1, 0.05)
            prof, _ = G.gist_profile_read(ctx)
            G.gist_profile_end(ctx)
            assert not any(k.startswith("relu_mask") for k in prof), sorted(prof)
            # the same step with unflagged layer calls (separate derivative pass)
            p2 = [to_dev(t.copy()) for t in theta]
            flags_fn = S.relu_chain_flags
            try:
                S.relu_chain_flags = lambda l, L: 0
                run.step(b, p2, 0.05)
            finally:
                S.relu_chain_flags = flags_fn
            for a, c in zip(p1, p2):
                assert same(to_host(a), to_host(c))
            log(f"{kind} dtype {dt}: no relu_mask launch, weights bitwise")
