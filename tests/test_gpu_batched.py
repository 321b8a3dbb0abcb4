"""GPU parity of batched sub-GCN layers: G sub-GCNs that share one mini-batch,
each with its own weight slice, in one layer call (one full-width
aggregation, grouped GEMMs).  Every group is compared with the oracle's
single-sub-GCN layer on that group's slice (eq. (2) and its backward),
normwise within 1e-4 (fp32) or 2e-2 (bf16-input), for GCN in both
association orders and SAGE-mean, the shared (unpartitioned) input, and
both output layouts.  As in the single-layer tests, the backward is fed the
oracle's forward values so that every ReLU decision comes from the same
numbers.  A batched sub-GCN step is checked against m oracle steps."""

import numpy as np
import pytest

from gist_synth.graphs import erdos_renyi, sbm
from oracle import gist as OG
from oracle import layers as OL
from oracle import minibatch as MB

from gpu_util import BF16_TOL, FP32_TOL, csr_to_dev, log, relerr, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


GRAPHS = {"er300": erdos_renyi(300, 900, seed=5, clusters=3),
          "sbm1500": sbm(1500, 10, 30.0, 0.9, seed=7)}

CASES = [
    # kind, graph, groups, s_in, s_out, act, order, shared input, group-major out, dtype
    ("gcn", "er300", 3, 40, 56, 1, 1, False, False, "f32"),
    ("gcn", "er300", 3, 56, 20, 1, 2, False, False, "f32"),     # transform first
    ("gcn", "er300", 4, 24, 7, 0, 2, False, True, "f32"),       # last layer, logits per group
    ("gcn", "er300", 2, 33, 64, 1, 0, True, False, "f32"),      # unpartitioned input
    ("sage", "sbm1500", 4, 64, 32, 1, 0, False, False, "f32"),
    ("sage", "sbm1500", 3, 20, 48, 1, 0, True, False, "f32"),   # SAGE input layer
    ("sage", "sbm1500", 2, 32, 5, 0, 0, False, True, "f32"),
    ("sage", "sbm1500", 2, 520, 520, 1, 0, False, False, "bf16"),   # packed bf16, per group
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[1]}-G{c[2]}-{c[3]}x{c[4]}-o{c[6]}"
                                             f"{'-shared' if c[7] else ''}{'-gm' if c[8] else ''}"
                                             f"-{c[9]}" for c in CASES])
def test_batched_layer_matches_oracle(G, ctx, case):
    import torch
    kind, gname, Gn, si, so, act, order, shared, gmajor, dt = case
    log(f"batched layer {case}")
    norm = "sage" if kind == "sage" else "gcn"
    csr = MB.build(GRAPHS[gname], None, norm)
    n = csr["n"]
    rng = np.random.default_rng(Gn * 100 + si)
    parts = 2 if kind == "sage" else 1
    Hs = [rng.standard_normal((n, si)).astype(np.float32)]
    if not shared:
        Hs += [rng.standard_normal((n, si)).astype(np.float32) for _ in range(Gn - 1)]
    Hg = lambda g: Hs[0] if shared else Hs[g]
    Ws = [(rng.standard_normal((parts * si, so)) / np.sqrt(si)).astype(np.float32)
          for _ in range(Gn)]
    dHs = [rng.standard_normal((n, so)).astype(np.float32) for _ in range(Gn)]
    relu = act == 1
    ref = []
    for g in range(Gn):
        if kind == "sage":
            f = OL.sage_forward(csr, Hg(g), Ws[g][:si], Ws[g][si:], relu)
            b = OL.sage_backward(csr, Hg(g), f, Ws[g][:si], Ws[g][si:], dHs[g], relu, not shared)
            dW = np.concatenate([b["dW_self"], b["dW_neigh"]])
        else:
            f = OL.gcn_forward(csr, Hg(g), Ws[g], relu)
            b = OL.gcn_backward(csr, Hg(g), f, Ws[g], dHs[g], relu, not shared)
            dW = b["dW"]
        ref.append(dict(f=f, dW=dW, dH=None if shared else b["dH"]))

    def cat_in(mats):     # n x (G s_in)
        return np.ascontiguousarray(np.concatenate(mats, axis=1))

    def cat_out(mats):    # n x (G s_out) or [G][n][s_out]
        return np.ascontiguousarray(np.stack(mats) if gmajor else np.concatenate(mats, axis=1))

    def split_out(arr):
        return [arr[g] for g in range(Gn)] if gmajor else [arr[:, g * so:(g + 1) * so]
                                                            for g in range(Gn)]

    A, keep = csr_to_dev(csr)
    AT, keep2 = csr_to_dev(csr, transpose=True) if kind == "sage" else (None, None)
    lk = G.GIST_LAYER_SAGE_MEAN if kind == "sage" else G.GIST_LAYER_GCN
    flags = (G.GIST_LAYER_SHARED_INPUT if shared else 0) | (G.GIST_LAYER_GROUP_MAJOR_OUT if gmajor else 0)
    dtype = G.GIST_DTYPE_BF16_IN if dt == "bf16" else G.GIST_DTYPE_F32
    tol = BF16_TOL if dt == "bf16" else FP32_TOL
    desc = G.layer_desc(lk, act, n, si, so, dtype, order, groups=Gn, flags=flags)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    w_in = si if shared else Gn * si
    Hd = to_dev(Hs[0] if shared else cat_in(Hs))
    Wd = to_dev(np.stack(Ws))
    agg = torch.empty(n, w_in, device="cuda")
    Ho = torch.empty(Gn, n, so, device="cuda") if gmajor else torch.empty(n, Gn * so, device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, Hd, Wd, agg, Ho, ws)
    got_H = split_out(to_host(Ho))
    forms_agg = kind == "sage" or order == 1 or (order == 0 and si <= so)
    got_agg = to_host(agg)
    for g in range(Gn):
        e = relerr(got_H[g], ref[g]["f"]["H_out"])
        ea = 0.0
        if forms_agg:
            cols = slice(0, si) if shared else slice(g * si, (g + 1) * si)
            ea = relerr(got_agg[:, cols], ref[g]["f"]["AH"])
        log(f"  group {g}: H_out {e:.2e} agg {ea:.2e}")
        assert e <= tol and ea <= tol
    # backward on the oracle's forward values
    agg_in = to_dev(ref[0]["f"]["AH"].astype(np.float32) if shared else
                    cat_in([r["f"]["AH"].astype(np.float32) for r in ref]))
    Ho_in = to_dev(cat_out([r["f"]["H_out"].astype(np.float32) for r in ref]))
    dW = torch.empty(Gn, parts * si, so, device="cuda")
    dH = None if shared else torch.empty(n, Gn * si, device="cuda")
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, Hd, agg_in, Ho_in, Wd, to_dev(cat_out(dHs)), dW, dH, ws)
    gdW = to_host(dW)
    gdH = None if shared else to_host(dH)
    for g in range(Gn):
        e = relerr(gdW[g], ref[g]["dW"])
        ed = 0.0 if shared else relerr(gdH[:, g * si:(g + 1) * si], ref[g]["dH"])
        log(f"  group {g}: dW {e:.2e} dH {ed:.2e}")
        assert e <= tol and ed <= tol


def test_batched_errors(G, ctx):
    import torch
    t = torch.zeros(64, device="cuda")
    A = G.csr_dev(4, 0, torch.zeros(5, dtype=torch.int32, device="cuda"), None, None)
    desc = G.layer_desc(G.GIST_LAYER_GCN, 1, 4, 2, 2, groups=2, flags=G.GIST_LAYER_SHARED_INPUT)
    with pytest.raises(G.GistError) as e:   # a shared input has no per-group dH
        G.gist_gcn_layer_bwd(ctx, desc, A, None, t, t, t, t, t, t, t, t)
    assert e.value.status == G.GIST_E_INVAL
    bad = G.layer_desc(G.GIST_LAYER_GCN, 1, 4, 2, 2, groups=2, flags=64)   # no such flag
    with pytest.raises(G.GistError):
        G.gist_layer_workspace_size(bad)


@pytest.mark.parametrize("kind", ["gcn", "sage"])
def test_batched_step_matches_oracle(G, ctx, kind):
    """m sub-GCNs stepping on one shared mini-batch, batched, against m
    oracle steps (forward values, loss and the last layer's gradients)."""
    import torch
    from paper_2102_10424_amd.step import BatchSlot, SubGCNBatch
    g = GRAPHS["sbm1500"] if kind == "sage" else GRAPHS["er300"]
    widths, m = ([30, 64, 64, 6] if kind == "sage" else [24, 32, 16, 5]), 4
    L = len(widths) - 1
    s = [widths[0]] + [widths[l] // m for l in range(1, L)] + [widths[-1]]
    parts = 2 if kind == "sage" else 1
    rng = np.random.default_rng(3)
    X = rng.standard_normal((g.n, widths[0])).astype(np.float32)
    y = rng.integers(0, widths[-1], g.n).astype(np.int32)
    P = [[(rng.standard_normal((parts * s[l], s[l + 1])) * 0.3).astype(np.float32)
          for l in range(L)] for _ in range(m)]
    norm = "sage" if kind == "sage" else "gcn"
    slot = BatchSlot(ctx, norm, g.n, g.nnz + g.n, widths[0])
    clusters = np.array([1, 4, 7], dtype=np.int32) if kind == "sage" else None
    b = slot.load(G.GraphHandle(g), clusters, to_dev(X), y)
    runner = SubGCNBatch(ctx, kind, s, m, b.n)
    params = [to_dev(np.stack([P[i][l] for i in range(m)])) for l in range(L)]   # [m][rows][cols]
    # the gradients (a full SGD step fuses its update into the backward pass
    # and keeps none), then the full step on a second copy of the weights
    runner.forward(b, params)
    runner.loss_and_grad(b)
    runner.backward(b, params)
    stepped = [p.clone() for p in params]
    torch.cuda.synchronize()
    losses = to_host(runner.loss)
    logits = [to_host(runner.logits(i)) for i in range(m)]
    grads = [to_host(runner.dW[L - 1][i]) for i in range(m)]
    runner.step(b, stepped, 0.05)
    torch.cuda.synchronize()
    csr = MB.build(g, clusters, norm)
    nm = csr["node_map"]
    for i in range(m):
        pi = [p if kind == "gcn" else (p[:s[l]], p[s[l]:]) for l, p in enumerate(P[i])]
        ref = OG.sub_gcn_step(kind, csr, X[nm], y[nm], pi, 0.05)
        assert abs(losses[i] - ref["loss"]) <= FP32_TOL * abs(ref["loss"])
        assert relerr(logits[i], ref["H"][L]) <= FP32_TOL
        gl = ref["grads"][L - 1]
        want = gl if kind == "gcn" else np.concatenate(gl)
        assert relerr(grads[i], want) <= FP32_TOL
        pl = ref["params"][L - 1]
        assert relerr(to_host(stepped[L - 1][i]), pl if kind == "gcn" else np.concatenate(pl)) \
            <= FP32_TOL
        log(f"  sub-GCN {i}: loss {losses[i]:.6f} (oracle {ref['loss']:.6f})")
