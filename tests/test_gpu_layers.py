"""GPU parity of the layer entry points against the fp64 oracle.

Each case runs gist_gcn_layer_fwd / _bwd through the C ABI on seeded inputs
and compares every output (aggregate, activation, dW, dH) with the oracle,
normwise, within 1e-4 (fp32) or 2e-2 (bf16-input GEMMs).  Shapes span
several 128-wide tiles with ragged tails, odd widths that defeat the
vectorised paths, and the split-K regime (tiny outputs, long reductions).
"""

import numpy as np
import pytest

from gist_synth.graphs import chung_lu, erdos_renyi, sbm
from oracle import layers as OL
from oracle import minibatch as MB

from gpu_util import BF16_TOL, FP32_TOL, csr_to_dev, log, relerr, to_dev, to_host

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


def _graphs():
    return {
        "er300": erdos_renyi(300, 900, seed=5, clusters=3),
        "cl2000": chung_lu(2000, 2.5, 5.0, seed=6),
        "sbm1500": sbm(1500, 10, 30.0, 0.9, seed=7),
    }


GRAPHS = _graphs()


def run_layer(G, ctx, kind, g, s_in, s_out, act, order, dtype, need_dH=True, seed=0):
    """Forward on seeded inputs, then backward on the oracle's forward values.

    The backward's ReLU mask is read from H_out.  Feeding both sides the
    oracle's H_out (and Abar H) rounded to fp32 makes them take every ReLU
    decision from the same numbers, so the comparison measures the kernels'
    arithmetic rather than sign flips of pre-activations within rounding
    distance of zero.
    """
    import torch
    norm = "sage" if kind == "sage" else "gcn"
    csr = MB.build(g, None, norm)
    n = csr["n"]
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((n, s_in)).astype(np.float32)
    parts = 2 if kind == "sage" else 1
    W = (rng.standard_normal((parts * s_in, s_out)) / np.sqrt(s_in)).astype(np.float32)
    dHo = rng.standard_normal((n, s_out)).astype(np.float32)
    A, keep = csr_to_dev(csr)
    AT, keep2 = csr_to_dev(csr, transpose=True) if kind == "sage" else (None, None)
    lk = G.GIST_LAYER_SAGE_MEAN if kind == "sage" else G.GIST_LAYER_GCN
    desc = G.layer_desc(lk, act, n, s_in, s_out, dtype, order)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    relu = act == G.GIST_ACT_RELU
    if kind == "sage":
        f = OL.sage_forward(csr, H, W[:s_in], W[s_in:], relu)
        b = OL.sage_backward(csr, H, f, W[:s_in], W[s_in:], dHo, relu, need_dH)
        want = dict(H_out=f["H_out"], dW=np.concatenate([b["dW_self"], b["dW_neigh"]]),
                    agg=f["AH"])
    else:
        f = OL.gcn_forward(csr, H, W, relu)
        b = OL.gcn_backward(csr, H, f, W, dHo, relu, need_dH)
        want = dict(H_out=f["H_out"], dW=b["dW"], agg=f["AH"])
    if need_dH:
        want["dH"] = b["dH"]
    Hd, Wd, dHod = to_dev(H), to_dev(W), to_dev(dHo)
    agg = torch.empty(n, s_in, device="cuda")
    Ho = torch.empty(n, s_out, device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, Hd, Wd, agg, Ho, ws)
    got = dict(H_out=to_host(Ho), agg=to_host(agg))
    agg_in = to_dev(f["AH"].astype(np.float32))
    Ho_in = to_dev(f["H_out"].astype(np.float32))
    dW = torch.empty(parts * s_in, s_out, device="cuda")
    dH = torch.empty(n, s_in, device="cuda") if need_dH else None
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, Hd, agg_in, Ho_in, Wd, dHod, dW, dH, ws)
    got["dW"] = to_host(dW)
    if need_dH:
        got["dH"] = to_host(dH)
    return got, want


CASES = [
    # kind, graph, s_in, s_out, act, order
    ("gcn", "er300", 37, 45, 1, 1),
    ("gcn", "er300", 128, 256, 1, 1),
    ("gcn", "er300", 200, 130, 1, 2),
    ("gcn", "cl2000", 64, 7, 0, 0),
    ("gcn", "cl2000", 500, 512, 1, 0),
    ("gcn", "cl2000", 512, 3, 0, 0),
    ("gcn", "sbm1500", 1433, 128, 1, 0),
    ("sage", "er300", 41, 47, 0, 0),
    ("sage", "sbm1500", 100, 256, 1, 0),
    ("sage", "sbm1500", 602, 260, 1, 0),
    ("sage", "cl2000", 256, 41, 0, 0),
    # weight gradients large enough (M, N >= 1024) for node-contiguous operand copies
    ("sage", "sbm1500", 512, 1024, 1, 0),
    ("gcn", "er300", 1030, 1100, 1, 1),
    ("gcn", "sbm1500", 1100, 1030, 0, 2),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[1]}-{c[2]}x{c[3]}-a{c[4]}-o{c[5]}"
                                             for c in CASES])
def test_layer_fp32(G, ctx, case):
    kind, gname, s_in, s_out, act, order = case
    log(f"layer fp32 {case}")
    got, want = run_layer(G, ctx, kind, GRAPHS[gname], s_in, s_out, act, order,
                          G.GIST_DTYPE_F32)
    for k in want:
        if k == "agg" and kind == "gcn" and order == 2:
            continue  # transform-first does not form Abar H
        if k == "agg" and kind == "gcn" and order == 0 and s_in > s_out:
            continue
        e = relerr(got[k], want[k])
        log(f"  {k}: {e:.3e}")
        assert e <= FP32_TOL, (k, e)


# bf16 cases include products large enough for the 256 x 256-tile MFMA path,
# with ragged M / N / K, K split into several slices (one shorter than the
# others) and the [dH | dP] split output of the SAGE backward; the last three
# have weight gradients of at least 1024 x 1024 over ragged node counts (300,
# 1500, 2000), read row-contiguous (the fp32 path copies such operands
# node-contiguous first; for bf16 inputs that measured slower).
@pytest.mark.parametrize("case", [("sage", "sbm1500", 100, 256, 1, 0),
                                  ("gcn", "cl2000", 500, 512, 1, 0),
                                  ("sage", "sbm1500", 602, 520, 1, 0),
                                  ("gcn", "cl2000", 1433, 600, 1, 0),
                                  ("sage", "sbm1500", 1024, 1024, 1, 0),
                                  ("gcn", "er300", 1030, 1100, 1, 1),
                                  ("gcn", "cl2000", 1100, 1030, 0, 2)])
def test_layer_bf16_inputs(G, ctx, case):
    kind, gname, s_in, s_out, act, order = case
    log(f"layer bf16 {case}")
    got, want = run_layer(G, ctx, kind, GRAPHS[gname], s_in, s_out, act, order,
                          G.GIST_DTYPE_BF16_IN)
    for k in want:
        if k == "agg" and kind == "gcn" and (order == 2 or (order == 0 and s_in > s_out)):
            continue  # transform-first does not form Abar H
        e = relerr(got[k], want[k])
        log(f"  {k}: {e:.3e}")
        assert e <= BF16_TOL, (k, e)


def test_bf16_direct_and_packed_staging_bitwise(G, ctx):
    """The bf16 product kernel stages operands straight from fp32 memory when
    the 16-byte loads allow it, else from a rounded bf16 copy made by a
    conversion pass; both put the same bf16 values in the same tiles.  A
    transform-first GCN layer reads H as the forward product's K-contiguous
    operand: H 16-byte aligned takes the direct staging, the same values at
    a 4-byte offset take the conversion pass.  Forward and backward outputs
    agree bit for bit (the backward's K = n products take the direct path in
    both runs, with a ragged last K step: n = 2000 = 62 * 32 + 16)."""
    import torch
    g = GRAPHS["cl2000"]
    csr = MB.build(g, None, "gcn")
    n, s_in, s_out = csr["n"], 512, 768
    rng = np.random.default_rng(11)
    H = rng.standard_normal((n, s_in)).astype(np.float32)
    W = (rng.standard_normal((s_in, s_out)) / np.sqrt(s_in)).astype(np.float32)
    dHo = rng.standard_normal((n, s_out)).astype(np.float32)
    A, keep = csr_to_dev(csr)
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, s_in, s_out,
                        G.GIST_DTYPE_BF16_IN, G.GIST_ORDER_XFORM_FIRST)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    Wd, dHod = to_dev(W), to_dev(dHo)
    aligned = to_dev(H)
    buf = torch.empty(n * s_in + 1, device="cuda")
    shifted = buf[1:].view(n, s_in)
    shifted.copy_(aligned)
    assert aligned.data_ptr() % 16 == 0 and shifted.data_ptr() % 16 == 4
    outs = []
    for Hd in (aligned, shifted):
        agg = torch.empty(n, s_in, device="cuda")
        Ho = torch.empty(n, s_out, device="cuda")
        G.gist_gcn_layer_fwd(ctx, desc, A, Hd, Wd, agg, Ho, ws)
        dW = torch.empty(s_in, s_out, device="cuda")
        dH = torch.empty(n, s_in, device="cuda")
        G.gist_gcn_layer_bwd(ctx, desc, A, None, Hd, agg, Ho, Wd, dHod, dW, dH, ws)
        outs.append([to_host(Ho), to_host(dW), to_host(dH)])
    for a, b in zip(*outs):
        assert a.tobytes() == b.tobytes()
    f = OL.gcn_forward(csr, H.astype(np.float64), W.astype(np.float64), True)
    e = relerr(outs[0][0], f["H_out"])
    log(f"direct and packed staging bitwise; H_out vs oracle {e:.3e}")
    assert e <= BF16_TOL


def test_layer_zero_batch_no_dH(G, ctx):
    import torch
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, 0, 8, 4)
    A = G.csr_dev(0, 0, torch.zeros(1, dtype=torch.int32, device="cuda"), None, None)
    W = torch.randn(8, 4, device="cuda")
    dW = torch.full((8, 4), 7.0, device="cuda")
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    e = torch.empty(0, device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, e, W, e, e, ws)
    G.gist_gcn_layer_bwd(ctx, desc, A, None, e, e, e, W, e, dW, None, ws)
    assert float(to_host(dW).max()) == 0.0 and float(to_host(dW).min()) == 0.0


def test_layer_bitwise_deterministic(G, ctx):
    log("determinism")
    a, _ = run_layer(G, ctx, "sage", GRAPHS["sbm1500"], 100, 256, 1, 0, G.GIST_DTYPE_F32, seed=3)
    b, _ = run_layer(G, ctx, "sage", GRAPHS["sbm1500"], 100, 256, 1, 0, G.GIST_DTYPE_F32, seed=3)
    for k in a:
        assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), k


def test_layer_errors(G, ctx):
    import torch
    desc = G.layer_desc(G.GIST_LAYER_SAGE_MEAN, 1, 4, 8, 4, order=G.GIST_ORDER_XFORM_FIRST)
    A = G.csr_dev(4, 0, torch.zeros(5, dtype=torch.int32, device="cuda"), None, None)
    t = torch.zeros(64, device="cuda")
    with pytest.raises(G.GistError) as e:
        G.gist_gcn_layer_fwd(ctx, desc, A, t, t, t, t, None)
    assert e.value.status == G.GIST_E_INVAL
    desc = G.layer_desc(G.GIST_LAYER_GCN, 1, 5, 8, 4)   # CSR has 4 rows, desc says 5
    with pytest.raises(G.GistError):
        G.gist_gcn_layer_fwd(ctx, desc, A, t, t, t, t, None)
