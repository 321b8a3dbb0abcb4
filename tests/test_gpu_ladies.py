"""GPU parity of GIST with LADIES layer sampling (Section 5.4, Appendix A.6)
through the C ABI.

* Rectangular GCN layers (n output rows aggregating n_in input rows, the
  matrices LADIES produces) against the fp64 oracle: aggregate, activation,
  dW and dH within 1e-4 (fp32) or 2e-2 (bf16-input GEMMs), both orders,
  batched groups (column-interleaved, shared input, group-major output),
  and an empty output set (dW and dH zeroed).
* One sub-GCN step on a LADIES mini-batch sampled by the library
  (gist_ladies_sample, bit-exact to the oracle's sampler on the CPU) and
  loaded by LadiesSlot: logits, loss, gradients and updated weights against
  the oracle's step on the oracle's batch.
* GIST training with SGD and Adam on LADIES mini-batches (m = 4, fused
  subAgg and gather) against the oracle's loop run through the GPU's ReLU
  decisions: Theta within 1e-4 normwise, its change within 1e-4 (SGD) or
  element by element within the oracle's rounding sensitivity (Adam), every
  loss within 1e-4; small sizes and those of the 232,965-node workload (512
  output nodes, 512 draws per layer, 602 -> 256/4 -> 41).
"""

import numpy as np
import pytest

from gist_synth.graphs import chung_lu, sbm
from oracle import gist as OG
from oracle import ladies as LD
from oracle import layers as OL
from oracle import minibatch as MB
from oracle import partition as OP

from gpu_util import (BF16_TOL, FP32_TOL, adam_noise, check_adam, csr_to_dev, gpu_orders, log,
                      relerr, to_dev, to_host)

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


_SAMPLES = {}


def _sampled(name):
    """Oracle LADIES layers of a fixed batch on one of two graphs (cached)."""
    if name not in _SAMPLES:
        if name == "cl3000":
            g, b, s = chung_lu(3000, 2.2, 6.0, seed=6), 40, 300
        else:
            g, b, s = sbm(5000, 40, 25.0, 0.9, seed=7), 150, 700
        A = MB.build(g, None, "gcn")
        batch = np.sort(np.random.default_rng(len(name)).choice(g.n, b, replace=False))
        _SAMPLES[name] = LD.sample(A, batch, 2, s, seed=99)
    return _SAMPLES[name]


def _upload(lay):
    A, k1 = csr_to_dev(lay)
    AT, k2 = csr_to_dev(lay, transpose=True)
    return A, AT, (k1, k2)


def _run_rect(G, ctx, lay, s_in, s_out, act, order, dtype, seed=0):
    """Forward, then backward on the oracle's forward values (as the square
    layer tests do, so both sides take every ReLU decision from the same
    numbers)."""
    import torch
    n, n_in = lay["n"], lay["n_in"]
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((n_in, s_in)).astype(np.float32)
    W = (rng.standard_normal((s_in, s_out)) / np.sqrt(s_in)).astype(np.float32)
    dHo = rng.standard_normal((n, s_out)).astype(np.float32)
    relu = act == G.GIST_ACT_RELU
    f = OL.gcn_forward(lay, H, W, relu)
    b = OL.gcn_backward(lay, H, f, W, dHo, relu, True)
    A, AT, keep = _upload(lay)
    desc = G.layer_desc(G.GIST_LAYER_GCN, act, n, s_in, s_out, dtype, order, n_in=n_in)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    Hd, Wd = to_dev(H), to_dev(W)
    agg = torch.full((n, s_in), float("nan"), device="cuda")
    out = torch.empty(n, s_out, device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, Hd, Wd, agg, out, ws)
    tol = FP32_TOL if dtype == G.GIST_DTYPE_F32 else BF16_TOL
    errs = dict(H_out=relerr(to_host(out), f["H_out"]))
    agg_first = order == G.GIST_ORDER_AGG_FIRST or (order == G.GIST_ORDER_AUTO and s_in <= s_out)
    if agg_first:
        errs["agg"] = relerr(to_host(agg), f["AH"])
    # backward from the oracle's forward values
    agg_in = to_dev(f["AH"].astype(np.float32))
    Ho = to_dev(f["H_out"].astype(np.float32))
    dW = torch.empty(s_in, s_out, device="cuda")
    dH = torch.full((n_in, s_in), float("nan"), device="cuda")
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, Hd, agg_in, Ho, Wd, to_dev(dHo), dW, dH, ws)
    errs["dW"] = relerr(to_host(dW), b["dW"])
    errs["dH"] = relerr(to_host(dH), b["dH"])
    return errs, tol


RECT = [
    # sample, layer, s_in, s_out, act, order
    ("cl3000", 0, 602, 64, 1, 0),      # input layer: transform first (s_in > s_out)
    ("cl3000", 1, 64, 41, 0, 0),       # output layer
    ("sbm5000", 0, 100, 256, 1, 0),    # aggregate first
    ("sbm5000", 0, 130, 97, 1, 1),     # forced orders, ragged widths
    ("sbm5000", 1, 33, 7, 0, 2),
    ("sbm5000", 0, 256, 256, 1, 2),
    ("cl3000", 0, 5, 300, 1, 1),
    ("sbm5000", 0, 1030, 1024, 1, 2),  # dW from node-contiguous copies (K = n_in)
]


@pytest.mark.parametrize("case", RECT, ids=[f"{c[0]}-l{c[1]}-{c[2]}x{c[3]}-a{c[4]}-o{c[5]}"
                                            for c in RECT])
@pytest.mark.parametrize("dtype", [0, 1])
def test_rect_layer(G, ctx, case, dtype):
    name, l, s_in, s_out, act, order = case
    lay = _sampled(name)["layers"][l]
    log(f"rect layer {case} dtype {dtype}: n={lay['n']} n_in={lay['n_in']} nnz={lay['nnz']}")
    assert lay["n_in"] > lay["n"]
    errs, tol = _run_rect(G, ctx, lay, s_in, s_out, act, order, dtype, seed=l + s_in)
    log("  " + ", ".join(f"{k} {v:.2e}" for k, v in errs.items()))
    assert max(errs.values()) <= tol, errs


@pytest.mark.parametrize("flags,order", [(0, 1), (0, 2), (1, 1), (1, 2), (2, 1), (2, 2), (3, 2)])
def test_rect_layer_batched(G, ctx, flags, order):
    """G = 3 sub-GCNs on one sampled layer: each group equals its own oracle layer."""
    import torch
    lay = _sampled("sbm5000")["layers"][0]
    n, n_in, Gn, si, so = lay["n"], lay["n_in"], 3, 48, 40
    shared = bool(flags & G.GIST_LAYER_SHARED_INPUT)
    gmajor = bool(flags & G.GIST_LAYER_GROUP_MAJOR_OUT)
    log(f"rect batched flags {flags} order {order}: n={n} n_in={n_in}")
    rng = np.random.default_rng(flags * 7 + order)
    Hs = [rng.standard_normal((n_in, si)).astype(np.float32) for _ in range(1 if shared else Gn)]
    Ws = [(rng.standard_normal((si, so)) / np.sqrt(si)).astype(np.float32) for _ in range(Gn)]
    dHs = [rng.standard_normal((n, so)).astype(np.float32) for _ in range(Gn)]
    ref = []
    for g in range(Gn):
        H = Hs[0 if shared else g]
        f = OL.gcn_forward(lay, H, Ws[g], True)
        ref.append((f, OL.gcn_backward(lay, H, f, Ws[g], dHs[g], True, True)))
    H_all = Hs[0] if shared else np.concatenate(Hs, axis=1)
    cat_out = (lambda xs: np.stack(xs)) if gmajor else (lambda xs: np.concatenate(xs, axis=1))
    A, AT, keep = _upload(lay)
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, si, so, 0, order, groups=Gn,
                        flags=flags, n_in=n_in)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    Hd, Wd = to_dev(H_all), to_dev(np.stack(Ws))
    agg = torch.empty(n, si if shared else Gn * si, device="cuda")
    out = torch.empty(*((Gn, n, so) if gmajor else (n, Gn * so)), device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, Hd, Wd, agg, out, ws)
    e_f = relerr(to_host(out), cat_out([r[0]["H_out"] for r in ref]))
    Ho = to_dev(cat_out([r[0]["H_out"] for r in ref]).astype(np.float32))
    agg_in = to_dev((ref[0][0]["AH"] if shared else
                     np.concatenate([r[0]["AH"] for r in ref], axis=1)).astype(np.float32))
    dW = torch.empty(Gn, si, so, device="cuda")
    dH = None if shared else torch.empty(n_in, Gn * si, device="cuda")
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, Hd, agg_in, Ho, Wd, to_dev(cat_out(dHs)), dW, dH, ws)
    e_w = relerr(to_host(dW), np.stack([r[1]["dW"] for r in ref]))
    e_h = 0.0 if shared else relerr(to_host(dH), np.concatenate([r[1]["dH"] for r in ref], 1))
    log(f"  forward {e_f:.2e} dW {e_w:.2e} dH {e_h:.2e}")
    assert max(e_f, e_w, e_h) <= FP32_TOL


def test_rect_layer_no_output_rows_and_errors(G, ctx):
    import torch
    n_in, si, so = 9, 16, 8
    empty = dict(n=0, n_in=n_in, nnz=0, rowptr=np.zeros(1, np.int32), col=np.zeros(0, np.int32),
                 val=np.zeros(0, np.float32), t_rowptr=np.zeros(n_in + 1, np.int32),
                 t_col=np.zeros(0, np.int32), t_val=np.zeros(0, np.float32))
    A, AT, keep = _upload(empty)
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, 0, si, so, n_in=n_in)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    H = torch.randn(n_in, si, device="cuda")
    W = torch.randn(si, so, device="cuda")
    dW = torch.full((si, so), float("nan"), device="cuda")
    dH = torch.full((n_in, si), float("nan"), device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, A, H, W, torch.empty(1, si, device="cuda"),
                         torch.empty(1, so, device="cuda"), ws)
    G.gist_gcn_layer_bwd(ctx, desc, A, AT, H, torch.empty(1, si, device="cuda"),
                         torch.empty(1, so, device="cuda"), W, torch.empty(1, so, device="cuda"),
                         dW, dH, ws)
    assert np.all(to_host(dW) == 0) and np.all(to_host(dH) == 0)
    # rectangular needs the transpose; SAGE may not be rectangular
    lay = _sampled("cl3000")["layers"][1]
    A, AT, keep = _upload(lay)
    d2 = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_NONE, lay["n"], 8, 8, n_in=lay["n_in"])
    f2, b2 = G.gist_layer_workspace_size(d2)
    ws2 = torch.empty(max(f2, b2, 1), dtype=torch.uint8, device="cuda")
    x = lambda r, c: torch.zeros(r, c, device="cuda")
    with pytest.raises(G.GistError) as e:
        G.gist_gcn_layer_bwd(ctx, d2, A, None, x(lay["n_in"], 8), x(lay["n"], 8), x(lay["n"], 8),
                             x(8, 8), x(lay["n"], 8), x(8, 8), x(lay["n_in"], 8), ws2)
    assert e.value.status == G.GIST_E_INVAL
    with pytest.raises(G.GistError) as e:    # the transpose must have n_in rows
        G.gist_gcn_layer_bwd(ctx, d2, A, A, x(lay["n_in"], 8), x(lay["n"], 8), x(lay["n"], 8),
                             x(8, 8), x(lay["n"], 8), x(8, 8), x(lay["n_in"], 8), ws2)
    assert e.value.status == G.GIST_E_INVAL
    with pytest.raises(G.GistError) as e:
        G.gist_layer_workspace_size(G.layer_desc(G.GIST_LAYER_SAGE_MEAN, 0, 10, 4, 4, n_in=12))
    assert e.value.status == G.GIST_E_INVAL


# ---- sub-GCN steps and GIST training on LADIES mini-batches ---------------------------

class _Workload:
    """Graph, full matrix, features, labels and weights of a LADIES workload."""

    def __init__(self, n, blocks, widths, b, s, seed=3, degree=20.0):
        self.g = sbm(n, blocks, degree, 0.9, seed=seed)
        self.A = MB.build(self.g, None, "gcn")
        rng = np.random.default_rng(seed)
        self.X = rng.standard_normal((n, widths[0])).astype(np.float32)
        self.y = rng.integers(0, widths[-1], n).astype(np.int32)
        self.widths, self.b, self.s, self.L = list(widths), b, s, len(widths) - 1
        self.theta = [(rng.standard_normal((widths[l], widths[l + 1])) *
                       np.sqrt(2.0 / widths[l])).astype(np.float32) for l in range(self.L)]
        self.max_degree = int(np.max(np.diff(self.g.rowptr)))

    def batch_nodes(self, key):
        r = np.random.default_rng(key)
        return np.sort(r.choice(self.g.n, self.b, replace=False)).astype(np.int32)

    def oracle_batch(self, key):
        out = LD.sample(self.A, self.batch_nodes(key), self.L, self.s, seed=key)
        return out["layers"], self.X[out["nodes"][0]], self.y[out["nodes"][self.L]]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("widths,b,s", [((50, 96, 12), 64, 256), ((50, 96, 64, 12), 64, 256),
                                        ((70, 130, 100, 9), 300, 900)])
def test_ladies_step_matches_oracle(G, ctx, widths, b, s, dtype):
    """A sub-GCN step on a library-sampled LADIES batch against the oracle's
    step on the oracle's batch, every tensor: logits, loss, every dW and
    every updated weight.  The oracle's backward runs through the GPU's own
    ReLU decisions (H_out > 0), which may differ from its own only where a
    pre-activation lies within rounding distance of zero; with bf16-input
    GEMMs the oracle rounds every dense product's operands to bf16, in the
    association order the GPU takes."""
    import torch
    from oracle import layers as OLr
    from paper_2102_10424_amd.step import LadiesSlot, SubGCN
    dt = G.GIST_DTYPE_BF16_IN if dtype == "bf16" else G.GIST_DTYPE_F32
    w = _Workload(4000, 40, widths, b, s)
    log(f"ladies step {dtype} widths {widths} b={b} s={s}")
    key = 31
    slot = LadiesSlot(ctx, w.L, w.b, w.s, w.max_degree, widths[0])
    b = slot.load(G.CsrHandle(w.A), w.batch_nodes(key), key, to_dev(w.X), w.y)
    layers, Xo, yo = w.oracle_batch(key)
    for l in range(w.L):
        assert b.rows(l) == layers[l]["n_in"] and b.rows(l + 1) == layers[l]["n"]
    assert b.rows(0) > b.rows(w.L)
    lr = 0.05
    params = [to_dev(t.copy()) for t in w.theta]
    run = SubGCN(ctx, "gcn", widths, 1, dtype=dt)
    logits = run.forward(b, params)
    run.loss_and_grad(b)
    run.backward(b, params)
    run.sgd(params, lr)
    torch.cuda.synchronize()
    masks = [to_host(run.H[l + 1][:b.rows(l + 1)]) > 0 for l in range(w.L - 1)] + [None]
    ref = OG.sub_gcn_step("gcn", layers, Xo, yo, w.theta, lr, masks=masks,
                          rnd=OLr.round_bf16 if dtype == "bf16" else None,
                          orders=gpu_orders("gcn", widths))
    tol = BF16_TOL if dtype == "bf16" else FP32_TOL
    band = 1e-2 if dtype == "bf16" else 1e-5
    flips = 0
    for l in range(w.L - 1):
        Z = ref["recs"][l]["Z"]
        diff = masks[l] != (Z > 0)
        assert np.all(np.abs(Z[diff]) <= band * np.max(np.abs(Z)))
        flips += int(diff.sum())
    e = dict(logits=relerr(to_host(logits), ref["H"][-1]),
             loss=abs(float(to_host(run.loss)[0]) - ref["loss"]) / abs(ref["loss"]),
             dlogits=relerr(to_host(run.dlogits[:b.rows(w.L)]), ref["dlogits"]))
    for l in range(w.L):
        if l < w.L - 1:
            e[f"H{l + 1}"] = relerr(to_host(run.H[l + 1][:b.rows(l + 1)]), ref["H"][l + 1])
        if l > 0:
            # the layer above hands this one dH times its ReLU derivative
            e[f"dH{l}"] = relerr(to_host(run.dH[l][:b.rows(l)]), ref["dH"][l] * masks[l - 1])
        e[f"dW{l}"] = relerr(to_host(run.dW[l]), ref["grads"][l])
        e[f"W{l}"] = relerr(to_host(params[l]), ref["params"][l])
    log(f"  {flips} decisions differ within the band; " +
        ", ".join(f"{k} {v:.2e}" for k, v in e.items()))
    assert max(e.values()) <= tol, e


@pytest.mark.parametrize("policy,size", [("carry", "small"), ("reset", "small"),
                                         ("sgd", "reddit"), ("carry", "reddit")])
def test_gist_train_on_ladies_batches(G, ctx, policy, size):
    """GIST training on LADIES mini-batches against the oracle's, with the
    oracle's backward run through the ReLU decisions the GPU took at each
    local step (H_out > 0): they may differ from the oracle's own only where
    a pre-activation lies within rounding distance of zero, which is
    checked.  SGD: the weights within 1e-4, their change within 1e-4 plus
    the fp32 rounding of the stored weights at each update (half an ulp of
    |Theta| per update, which at the workload's sizes is about as large as
    1e-4 of the first layer's small change).  Adam: the
    weight changes held element by element to the oracle's own sensitivity
    to rounding-sized gradient noise (``check_adam``: 1e-4 where that noise
    does not move them; Theta_0 is exact in fp32, so this holds Theta
    itself).  Small sizes, and the workload's sizes (a
    Reddit-sized graph, 512 outputs, 512 draws per layer, 602-256-41,
    m = 4)."""
    import torch
    from paper_2102_10424_amd.step import GistModel, LadiesSlot, SubGCN, gist_train
    if size == "reddit":
        w = _Workload(232_965, 1500, (602, 256, 41), 512, 512, seed=5, degree=50.0)
        rounds, zeta = 1, 2
    else:
        w = _Workload(3000, 30, (40, 64, 48, 9), 48, 160)
        rounds, zeta = 2, 2
    m, lr, L = 4, 0.01, w.L
    log(f"ladies train {policy} {size}: widths {w.widths} m={m} T={rounds} zeta={zeta}")
    seeds = lambda t: {l: 11 + 10 * t + l for l in range(1, L)}
    key = lambda t, i, z: 1000 * t + 100 * i + z + 1
    th = [[to_dev(t.copy())] for t in w.theta]
    model = GistModel(ctx, "gcn", w.widths, m, th, adam=None if policy == "sgd" else policy)
    slot = LadiesSlot(ctx, L, w.b, w.s, w.max_degree, w.widths[0])
    Ah, Xd = G.CsrHandle(w.A), to_dev(w.X)
    runner = SubGCN(ctx, "gcn", model.slice_widths, 1)
    masks = {}

    def decisions(t, i, z, b):
        torch.cuda.synchronize()
        masks[(t, i, z)] = [to_host(runner.H[l + 1][:b.rows(l + 1)]) > 0
                            for l in range(L - 1)] + [None]

    losses = gist_train(model, runner, rounds, zeta, lr, seeds,
                        lambda t, i, z: slot.load(Ah, w.batch_nodes(key(t, i, z)), key(t, i, z),
                                                  Xd, w.y),
                        after_step=decisions)
    torch.cuda.synchronize()
    losses = to_host(losses)
    parts = lambda t: [None] + [OP.partition(w.widths[l], m, seeds(t)[l])
                                for l in range(1, L)] + [None]
    cache = {}

    def batch(t, i, z):
        if (t, i, z) not in cache:
            cache[(t, i, z)] = w.oracle_batch(key(t, i, z))
        return cache[(t, i, z)]

    steps = []
    if policy == "sgd":
        th_o, lo = [t for t in w.theta], []
        for t in range(rounds):
            th_o, _, lt = OG.gist_round("gcn", th_o, parts(t), lambda i, z: batch(t, i, z), lr,
                                        zeta, masks=lambda i, z: masks[(t, i, z)], steps=steps)
            lo.append(lt)
    else:
        train = lambda noise, st=None: OG.gist_train(
            "gcn", [t for t in w.theta], rounds, zeta, lr, parts, batch, policy=policy,
            grad_noise=noise, masks=lambda t, i, z: masks[(t, i, z)], steps=st)
        th_o, _, _, lo = train(None, steps)
        pert = [train(adam_noise(3e-6, s))[0] for s in (1, 2, 3)]
    flips = 0
    for k, st in zip(sorted(masks), steps):
        for l in range(L - 1):
            Z = st["recs"][l]["Z"]
            diff = masks[k][l] != (Z > 0)
            assert np.all(np.abs(Z[diff]) <= 1e-5 * np.max(np.abs(Z))), (k, l)
            flips += int(diff.sum())
    assert len(steps) == rounds * m * zeta
    log(f"  {flips} decisions differ within the band")
    for l in range(L):
        got = to_host(model.theta[l][0])
        e = relerr(got, th_o[l])
        if policy == "sgd":
            d = relerr(got.astype(np.float64) - w.theta[l], th_o[l] - w.theta[l])
            # each of the rounds * zeta updates stores Theta in fp32 (the
            # oracle keeps fp64): up to half an ulp of |Theta| per update on
            # top of the arithmetic's 1e-4 of the change
            store = rounds * zeta * 2.0 ** -24 * np.max(np.abs(got)) / np.max(
                np.abs(th_o[l] - w.theta[l]))
            log(f"  layer {l}: theta {e:.2e}, change {d:.2e} (fp32 storage: {store:.2e})")
            assert e <= FP32_TOL and d <= FP32_TOL + store
        else:
            # Theta = Theta_0 (exact in fp32) + change, so the element-wise
            # check of the change is the check of Theta; a normwise bar on
            # Theta would ignore that sign-like Adam steps on gradients near
            # zero move by the rounding of those gradients
            d = check_adam(got.astype(np.float64) - w.theta[l], th_o[l] - w.theta[l],
                           [q[l] - w.theta[l] for q in pert])
            log(f"  layer {l}: theta {e:.2e}; change: {d[0]:.2e} on the {100 * d[1]:.0f}% "
                f"well-conditioned entries, worst {d[2]:.2f} of the bound")
            assert d[0] <= FP32_TOL and d[2] <= 1.0
    want_l = np.array([[li for li in lt] for lt in lo])
    assert np.max(np.abs(losses - want_l) / np.abs(want_l)) <= FP32_TOL


def test_graph_runner_replays_match_eager_and_oracle(G, ctx):
    """Sub-GCN steps replayed from HIP graphs (fixed, padded shapes) against
    eager steps on the same batches and against the oracle's chained SGD
    steps; two parameter sets alternate (two graphs), and eager library work
    and synchronisations run between the replays."""
    import torch
    from paper_2102_10424_amd.step import LadiesGraphRunner, LadiesSlot, SubGCN
    widths = (50, 96, 64, 12)
    w = _Workload(4000, 40, widths, 64, 256, seed=9)
    L, lr = w.L, 0.05
    Ah, Xd = G.CsrHandle(w.A), to_dev(w.X)
    fixed = LadiesSlot(ctx, L, w.b, w.s, w.max_degree, widths[0], fixed=True)
    plain = LadiesSlot(ctx, L, w.b, w.s, w.max_degree, widths[0])
    gr = LadiesGraphRunner(ctx, widths, L, w.b, w.s, widths[0], Xd)
    eager = SubGCN(ctx, "gcn", widths, 1)
    sets = 2
    pg = [[to_dev(t.copy()) for t in w.theta] for _ in range(sets)]
    pe = [[to_dev(t.copy()) for t in w.theta] for _ in range(sets)]
    po = [[t.astype(np.float64) for t in w.theta] for _ in range(sets)]
    for k in range(6):
        j = k % sets
        key = 500 + k
        log(f"graph replay {k}: parameter set {j}")
        fixed.build(Ah, w.batch_nodes(key), key, w.y)
        assert fixed.fits_fixed()
        gr.step(fixed, pg[j], lr)
        b = plain.load(Ah, w.batch_nodes(key), key, Xd, w.y)
        eager.step(b, pe[j], lr)
        torch.cuda.synchronize()
        layers, Xo, yo = w.oracle_batch(key)
        po[j] = OG.sub_gcn_step("gcn", layers, Xo, yo, po[j], lr)["params"]
        for l in range(L):
            g_, e_ = to_host(pg[j][l]), to_host(pe[j][l])
            assert relerr(g_, e_) <= 1e-5, (k, l)
            assert relerr(g_, po[j][l]) <= FP32_TOL, (k, l)
        assert abs(float(to_host(gr.loss)[0]) - float(to_host(eager.loss)[0])) <= 1e-5
    assert len(gr.graphs) == sets
    # an eager step through the fixed layout's own upload agrees as well
    fixed.build(Ah, w.batch_nodes(900), 900, w.y)
    b = fixed.upload(Xd)
    assert [b.rows(l) for l in range(L + 1)] == [plain.load(Ah, w.batch_nodes(900), 900, Xd,
                                                            w.y).rows(l) for l in range(L + 1)]


def test_graph_runner_falls_back_when_the_layout_is_full(G, ctx):
    """A batch with more entries than the fixed layout holds is packed
    compactly and stepped eagerly by the runner, with the same result."""
    import torch
    from paper_2102_10424_amd.step import LadiesGraphRunner, LadiesSlot, SubGCN
    widths = (30, 40, 7)
    w = _Workload(3000, 30, widths, 32, 128, seed=12)
    Ah, Xd = G.CsrHandle(w.A), to_dev(w.X)
    slot = LadiesSlot(ctx, w.L, w.b, w.s, w.max_degree, widths[0], fixed=True,
                      fixed_nnz_per_row=1)
    gr = LadiesGraphRunner(ctx, widths, w.L, w.b, w.s, widths[0], Xd, fixed_nnz_per_row=1)
    eager = SubGCN(ctx, "gcn", widths, 1)
    pg = [to_dev(t.copy()) for t in w.theta]
    pe = [to_dev(t.copy()) for t in w.theta]
    plain = LadiesSlot(ctx, w.L, w.b, w.s, w.max_degree, widths[0])
    slot.build(Ah, w.batch_nodes(3), 3, w.y)
    assert not slot.fits_fixed()
    gr.step(slot, pg, 0.05)
    eager.step(plain.load(Ah, w.batch_nodes(3), 3, Xd, w.y), pe, 0.05)
    torch.cuda.synchronize()
    for a, b in zip(pg, pe):
        assert torch.equal(a, b)
    assert not gr.graphs


def test_graph_runner_adam_replays_match_eager(G, ctx):
    """LADIES steps replayed with Adam (the coefficients of steps 1..4 carried
    by the batches, the 'reset' policy's fresh first step included): weights
    and moments match eager gist_adam_update steps on the same batches."""
    import torch
    from paper_2102_10424_amd.step import LadiesGraphRunner, LadiesSlot, SubGCN
    widths = (40, 64, 9)
    w = _Workload(3000, 30, widths, 48, 160, seed=21)
    Ah, Xd = G.CsrHandle(w.A), to_dev(w.X)
    fixed = LadiesSlot(ctx, w.L, w.b, w.s, w.max_degree, widths[0], fixed=True)
    plain = LadiesSlot(ctx, w.L, w.b, w.s, w.max_degree, widths[0])
    gr = LadiesGraphRunner(ctx, widths, w.L, w.b, w.s, widths[0], Xd)
    eager = SubGCN(ctx, "gcn", widths, 1)
    pg = [to_dev(t.copy()) for t in w.theta]
    pe = [to_dev(t.copy()) for t in w.theta]
    Mg, Vg = [torch.full_like(t, 7.0) for t in pg], [torch.full_like(t, 7.0) for t in pg]
    Me, Ve = [torch.full_like(t, 7.0) for t in pg], [torch.full_like(t, 7.0) for t in pg]
    lr = 0.01
    for k, (step, fresh) in enumerate([(1, True), (2, False), (3, False), (1, True)]):
        key = 70 + k
        log(f"ladies adam replay {k}: step {step} fresh {fresh}")
        flags = G.GIST_ADAM_FRESH if fresh else 0
        fixed.build(Ah, w.batch_nodes(key), key, w.y,
                    coef=G.gist_adam_coefficients(lr, step, flags=flags))
        gr.step(fixed, pg, lr, adam=(Mg, Vg))
        eager.step(plain.load(Ah, w.batch_nodes(key), key, Xd, w.y), pe, lr,
                   adam=(Me, Ve, step, fresh))
        torch.cuda.synchronize()
        for l in range(w.L):
            assert relerr(to_host(pg[l]), to_host(pe[l])) <= 1e-5, (k, l)
            assert relerr(to_host(Mg[l]), to_host(Me[l])) <= 1e-5, (k, l)
            assert relerr(to_host(Vg[l]), to_host(Ve[l])) <= 1e-5, (k, l)
    assert len(gr.graphs) == 1
