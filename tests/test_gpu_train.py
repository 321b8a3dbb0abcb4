"""GPU parity of Adam and of the GIST training loop (Algorithm 1 with the
optimizer of the paper's experiments), through the C ABI.

* gist_adam_update against the fp64 oracle (Kingma & Ba's Algorithm 1), both
  with the fp32 hyper-parameters the ABI carries: weights and moments within
  1e-6 normwise, every weight within 1e-4 of its update plus two fp32 ulps;
  FRESH restarts the moments; bad arguments are rejected on the host.
* gist_train (T rounds x m sub-GCNs x zeta local steps, fused subAgg/gather,
  moments carried with the weights or reset per round) against
  oracle.gist.gist_train on the same seeded inputs: Theta within 1e-4
  normwise, every loss within 1e-4; the change of Theta over training and
  the carried first moments element by element against the oracle's own
  sensitivity (tests/gpu_util.check_adam: 1e-4 on the entries that rounding
  noise in the oracle's gradients does not move, a multiple of that
  movement on the rest).
* m = 1: the loop equals plain Adam training of the full model on the GPU,
  bit for bit (Section 2.1: one sub-GCN is the whole GCN).
* GAT models in the same loop (the output layer's attention vectors, which
  every sub-GCN trains in full, aggregated as the mean of the m copies), and
  gist_subagg_mean bit for bit against the fp64 mean rounded to fp32.
"""

import numpy as np
import pytest

from gist_synth.graphs import erdos_renyi, sbm
from oracle import gist as OG
from oracle import minibatch as OM
from oracle import optim as OO
from oracle import partition as OP

from gpu_util import FP32_TOL, adam_noise, check_adam, log, relerr, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


@pytest.mark.parametrize("n", [1, 1001, 4 * 1024 * 1024 + 3])
@pytest.mark.parametrize("step,fresh", [(1, False), (7, False), (3, True)])
def test_adam_update_matches_oracle(G, ctx, n, step, fresh):
    import torch
    log(f"adam n={n} step={step} fresh={fresh}")
    rng = np.random.default_rng(n + step)
    W = rng.standard_normal(n).astype(np.float32)
    g = (rng.standard_normal(n) * np.exp(rng.uniform(-8, 2, n))).astype(np.float32)
    m = (rng.standard_normal(n) * 0.1).astype(np.float32)
    v = (rng.uniform(0, 1, n) * 0.01).astype(np.float32)
    Wd, gd, md, vd = to_dev(W), to_dev(g), to_dev(m), to_dev(v)
    lr = 1e-3
    G.gist_adam_update(ctx, Wd, gd, md, vd, n, lr, step,
                       flags=G.GIST_ADAM_FRESH if fresh else 0)
    m0, v0 = (np.zeros(n), np.zeros(n)) if fresh else (m, v)
    # the ABI takes beta and eps in fp32: the oracle gets the values the kernel receives
    f32 = lambda x: float(np.float32(x))
    Wr, mr, vr = OO.adam(W, g, m0, v0, step, f32(lr), f32(OO.BETA1), f32(OO.BETA2), f32(OO.EPS))
    Wg, mg, vg = to_host(Wd), to_host(md), to_host(vd)
    assert relerr(Wg, Wr) <= 1e-6
    assert relerr(mg, mr) <= 1e-6 and relerr(vg, vr) <= 1e-6
    # every element: within 1e-4 of its update plus two ulps of the stored fp32 result
    bound = 1e-4 * np.abs(W - Wr) + 2 * np.spacing(np.abs(Wr).astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(Wg.astype(np.float64) - Wr) <= bound)
    torch.cuda.synchronize()


def test_adam_update_errors(G, ctx):
    import torch
    t = torch.zeros(8, device="cuda")
    for kw in (dict(step=0), dict(beta1=1.0), dict(beta2=-0.1), dict(eps=-1.0),
               dict(lr=float("nan")), dict(flags=2)):
        args = dict(lr=0.1, step=1)
        args.update(kw)
        with pytest.raises(G.GistError) as e:
            G.gist_adam_update(ctx, t, t, t, t, 8, **args)
        assert e.value.status == G.GIST_E_INVAL
    G.gist_adam_update(ctx, None, None, None, None, 0, 0.1, 1)   # n = 0: no-op


# ---- the loop --------------------------------------------------------------

def test_subagg_mean_matches_oracle(G, ctx):
    import torch
    rng = np.random.default_rng(5)
    for m, rows, cols, lds, ldg in ((3, 2, 47, 53, 50), (8, 5, 1000, 1000, 1000), (1, 1, 7, 7, 7)):
        log(f"subagg_mean m={m} {rows}x{cols}")
        copies = (rng.standard_normal((m, rows, lds)) * np.exp(rng.uniform(-3, 3, (m, rows, lds)))
                  ).astype(np.float32)
        dev = [to_dev(c) for c in copies]
        table = torch.tensor([d.data_ptr() for d in dev], dtype=torch.int64, device="cuda")
        Wg = torch.full((rows, ldg), 7.0, device="cuda")
        G.gist_subagg_mean(ctx, Wg, rows, cols, ldg, m, table, lds)
        got = to_host(Wg)
        want = np.mean(copies[:, :, :cols].astype(np.float64), axis=0).astype(np.float32)
        assert np.array_equal(got[:, :cols], want)
        assert np.all(got[:, cols:] == 7.0)          # padding untouched
    with pytest.raises(G.GistError) as e:
        G.gist_subagg_mean(ctx, Wg, 1, 7, 7, 0, table, 7)
    assert e.value.status == G.GIST_E_INVAL
    G.gist_subagg_mean(ctx, None, 0, 7, 7, 2, None, 7)   # empty: no-op


def _setup(kind):
    """A small seeded problem: (graph, widths, m, theta (fp32), X, labels, batches)."""
    rng = np.random.default_rng(11)
    if kind == "gcn":
        g = erdos_renyi(300, 900, 5)
        widths, m = [24, 32, 16, 5], 2
        clusters = lambda t, i, z: None                 # full graph
    else:
        g = sbm(600, 12, 10.0, 0.9, 6)
        widths, m = [20, 32, 32, 7], 4
        clusters = lambda t, i, z: np.array(sorted(
            np.random.default_rng(1000 * t + 10 * i + z).choice(12, 3, replace=False)),
            dtype=np.int32)
    X = rng.standard_normal((g.n, widths[0])).astype(np.float32)
    y = rng.integers(0, widths[-1], g.n).astype(np.int32)
    L = len(widths) - 1
    if kind == "gat":     # [Theta_l, A_l] with A_l = [a_src; a_dst]
        theta = [[(rng.standard_normal((widths[l], widths[l + 1])) * 0.3).astype(np.float32),
                  (rng.standard_normal((2, widths[l + 1])) * 0.3).astype(np.float32)]
                 for l in range(L)]
    else:
        parts = 1 if kind == "gcn" else 2
        theta = [[(rng.standard_normal((widths[l], widths[l + 1])) * 0.3).astype(np.float32)
                  for _ in range(parts)] for l in range(L)]
    return g, widths, m, theta, X, y, clusters


def _oracle_theta(kind, theta):
    if kind == "gat":
        return [(W, A[0], A[1]) for W, A in theta]
    return [ps[0] for ps in theta] if kind == "gcn" else [(a, b) for a, b in theta]


def _oracle_part(kind, params, p):
    """Part p of an oracle layer in the device layout (GAT: [a_src; a_dst])."""
    if kind == "gcn":
        return params
    if kind == "gat":
        return params[0] if p == 0 else np.stack([params[1], params[2]])
    return params[p]


def _gpu_train(G, ctx, kind, g, widths, m, theta, X, y, clusters, rounds, zeta, lr, policy,
               seeds):
    import torch
    from paper_2102_10424_amd.step import BatchSlot, GistModel, SubGCN, gist_train
    norm = "sage" if kind == "sage" else "gcn"       # GAT: the pattern of A + I
    th = [[to_dev(t.copy()) for t in ps] for ps in theta]
    model = GistModel(ctx, kind, widths, m, th, adam=policy)
    gh = G.GraphHandle(g)
    Xd = to_dev(X)
    slot = BatchSlot(ctx, norm, g.n, g.nnz + g.n, widths[0])
    runner = SubGCN(ctx, kind, model.slice_widths, g.n)
    losses = gist_train(model, runner, rounds, zeta, lr, seeds,
                        lambda t, i, z: slot.load(gh, clusters(t, i, z), Xd, y))
    torch.cuda.synchronize()
    return model, to_host(losses)


@pytest.mark.parametrize("kind,policy", [("gcn", "carry"), ("gcn", "reset"), ("sage", "carry"),
                                         ("sage", "reset"), ("gat", "carry"), ("gat", "reset")])
def test_gist_train_matches_oracle(G, ctx, kind, policy):
    g, widths, m, theta, X, y, clusters = _setup(kind)
    rounds, zeta, lr = 2, 2, 0.01
    L = len(widths) - 1
    seeds = lambda t: {l: 77 + 10 * t + l for l in range(1, L)}
    log(f"train {kind} {policy}: widths {widths} m={m} T={rounds} zeta={zeta}")
    model, losses = _gpu_train(G, ctx, kind, g, widths, m, theta, X, y, clusters, rounds, zeta,
                               lr, policy, seeds)
    norm = "sage" if kind == "sage" else "gcn"

    def batches(t, i, z):
        csr = OM.build(g, clusters(t, i, z), norm)
        nm = csr["node_map"]
        return csr, X[nm], y[nm]

    parts = lambda t: [None] + [OP.partition(widths[l], m, seeds(t)[l]) for l in range(1, L)] + [None]
    train = lambda noise: OG.gist_train(kind, _oracle_theta(kind, theta), rounds, zeta, lr,
                                        parts, batches, policy=policy, grad_noise=noise)
    th_o, Mo, Vo, lo = train(None)
    # the oracle again with rounding-sized noise on its gradients: how far each
    # trained value moves for reasons the path cannot control
    pert = [train(adam_noise(3e-6, s)) for s in (1, 2, 3)]
    for l in range(L):
        for p in range(model.parts):
            want = _oracle_part(kind, th_o[l], p)
            got = to_host(model.theta[l][p])
            e = relerr(got, want)
            d = check_adam(got.astype(np.float64) - theta[l][p], want - theta[l][p],
                           [_oracle_part(kind, q[0][l], p) - theta[l][p] for q in pert])
            msg = f"  layer {l} part {p}: theta {e:.2e}; change: {d[0]:.2e} on the " \
                  f"{100 * d[1]:.0f}% well-conditioned entries, worst {d[2]:.2f} of the bound"
            if policy == "carry":
                mo = check_adam(to_host(model.Mg[l][p]), _oracle_part(kind, Mo[l], p),
                                [_oracle_part(kind, q[1][l], p) for q in pert])
                msg += f"; first moment {mo[0]:.2e} ({100 * mo[1]:.0f}%), {mo[2]:.2f}"
                assert mo[0] <= FP32_TOL and mo[2] <= 1.0
            log(msg)
            assert e <= FP32_TOL and d[0] <= FP32_TOL and d[2] <= 1.0
    want_l = np.array([[li for li in lt] for lt in lo])
    assert np.max(np.abs(losses - want_l) / np.abs(want_l)) <= FP32_TOL
    if kind != "gat":     # four Adam steps on changing batches need not lower a GAT's loss
        assert losses[-1].mean() < losses[0].mean()


def test_gist_train_m1_is_full_model_training(G, ctx):
    """One sub-GCN is the whole GCN: the loop equals Adam on the full model."""
    import torch
    from paper_2102_10424_amd.step import BatchSlot, SubGCN
    g, widths, _, theta, X, y, clusters = _setup("gcn")
    rounds, zeta, lr = 2, 3, 0.01
    L = len(widths) - 1
    seeds = lambda t: {l: 5 + t + l for l in range(1, L)}
    model, losses = _gpu_train(G, ctx, "gcn", g, widths, 1, theta, X, y, clusters, rounds, zeta,
                               lr, "carry", seeds)
    # plain training: the full parameters with one set of moments
    W = [to_dev(ps[0].copy()) for ps in theta]
    M = [torch.zeros_like(w) for w in W]
    V = [torch.zeros_like(w) for w in W]
    slot = BatchSlot(ctx, "gcn", g.n, g.nnz + g.n, widths[0])
    runner = SubGCN(ctx, "gcn", widths, g.n)
    b = slot.load(G.GraphHandle(g), None, to_dev(X), y)
    plain = torch.empty(rounds * zeta, device="cuda")
    for k in range(rounds * zeta):
        runner.step(b, W, lr, adam=(M, V, k + 1, False), loss_out=plain[k:k + 1])
    torch.cuda.synchronize()
    for l in range(L):
        assert torch.equal(model.theta[l][0], W[l]), f"layer {l}"
        assert torch.equal(model.Mg[l][0], M[l]) and torch.equal(model.Vg[l][0], V[l])
    assert np.array_equal(losses.reshape(-1), to_host(plain))
